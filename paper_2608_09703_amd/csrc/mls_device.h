// Device-side building blocks shared by the gfx950 kernels of libmls.
//
// Every dense contraction in the library has the same shape: an "NT" tile
// product C[m][n] = sum_k A[m][k] * B[n][k] where both operands are
// row-major with the contraction index contiguous. The logits l = W h^T of
// the LM head (paper section 2, "Modeling") are computed this way with
// A = W_i (vocabulary rows) and B = h_i (token rows); the two backward
// products use pre-transposed operands so that they take the same form.
//
// Tiles are staged through LDS in rows of 128 bytes of K (64 bf16 or 32 fp32
// values). Each row holds eight 16-byte chunks, stored at a position XOR-ed
// with the row index so that the 32 lanes of a fragment read (32 different
// rows, one chunk each) spread over all LDS banks.
//
// MFMA: v_mfma_f32_32x32x16_bf16 (bf16) or four v_mfma_f32_32x32x2_f32
// (fp32). Lane l supplies row (l % 32) of A and of B and one 16-byte chunk
// of K (chunk 2*kk + l/32 of the 128-byte row); A and B use the same
// assignment, so each MFMA contracts the same K values for both operands.
// Output element r (0..15) of lane l holds
//   row    8*(r/4) + 4*(l/32) + r%4   of the 32-row block (A side)
//   column l % 32                     of the 32-column block (B side).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mls {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;   // 4 waves of 64
constexpr int kRowBytes = 128;  // bytes of K per LDS tile row
constexpr float kLog2e = 1.4426950408889634f;

struct Bf16 {
  typedef uint16_t storage;
  static constexpr int kBytes = 2;
};
struct F32 {
  typedef float storage;
  static constexpr int kBytes = 4;
};

template <typename E>
__device__ __forceinline__ void mma_step(f32x16_t& acc, uint4 a, uint4 b);

template <>
__device__ __forceinline__ void mma_step<Bf16>(f32x16_t& acc, uint4 a, uint4 b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
}

template <>
__device__ __forceinline__ void mma_step<F32>(f32x16_t& acc, uint4 a, uint4 b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
}

// Position of 16-byte chunk c of LDS tile row `row`. Rows r..r+7 get distinct
// chunks, and rows r and r+8 differ as well, so 8- and 16-lane read phases are
// both free of bank conflicts.
__device__ __forceinline__ int lds_off(int row, int c) {
  return row * kRowBytes + ((c ^ (row & 7) ^ ((row >> 3) & 1)) << 4);
}

__device__ __forceinline__ uint4 lds_read16(const char* base, int row, int c) {
  return *reinterpret_cast<const uint4*>(base + lds_off(row, c));
}

// Rows [row0, row0 + ROWS) x K bytes [kb0, kb0 + 128) of a row-major matrix
// with `nrows` rows and `kbytes` bytes per row (stride ld_bytes). Each of the
// 256 threads moves ROWS*8/256 chunks of 16 bytes; out-of-range chunks are 0.
template <int ROWS>
struct TileLoader {
  static constexpr int kChunks = ROWS * 8 / kThreads;
  static_assert(ROWS * 8 % kThreads == 0, "tile rows must be a multiple of 32");
  uint4 r[kChunks];

  __device__ __forceinline__ void load(const char* __restrict__ base, int64_t ld_bytes,
                                       int64_t row0, int64_t nrows, int64_t kb0,
                                       int64_t kbytes, int tid) {
#pragma unroll
    for (int j = 0; j < kChunks; ++j) {
      const int ci = tid + kThreads * j;
      const int row = ci >> 3;
      const int c = ci & 7;
      const int64_t gr = row0 + row;
      const int64_t kb = kb0 + (c << 4);
      if (gr < nrows && kb < kbytes) {
        r[j] = *reinterpret_cast<const uint4*>(base + gr * ld_bytes + kb);
      } else {
        r[j] = make_uint4(0u, 0u, 0u, 0u);
      }
    }
  }

  __device__ __forceinline__ void store(char* lds, int tid) const {
#pragma unroll
    for (int j = 0; j < kChunks; ++j) {
      const int ci = tid + kThreads * j;
      *reinterpret_cast<uint4*>(lds + lds_off(ci >> 3, ci & 7)) = r[j];
    }
  }
};

// Block tile BM x BN computed by 4 waves arranged WGM x WGN; wave (wm, wn)
// owns rows [wm*BM/WGM, ...) and columns [wn*BN/WGN, ...) as FM x FN blocks
// of 32x32.
template <typename E, int BM, int BN, int WGM, int WGN>
struct TileMma {
  static_assert(WGM * WGN == 4, "four waves per block");
  static constexpr int kBM = BM;
  static constexpr int kBN = BN;
  static constexpr int kWGM = WGM;
  static constexpr int kWGN = WGN;
  static constexpr int NT = kThreads;
  static constexpr int WTM = BM / WGM;
  static constexpr int WTN = BN / WGN;
  static constexpr int FM = WTM / 32;
  static constexpr int FN = WTN / 32;
  static constexpr int kStageBytes = (BM + BN) * kRowBytes;
  static constexpr int kSmemBytes = 2 * kStageBytes;

  f32x16_t acc[FM][FN];

  __device__ __forceinline__ void compute_stage(const char* sA, const char* sB, int lane,
                                                int wm, int wn) {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int c = 2 * kk + (lane >> 5);
      uint4 a[FM], b[FN];
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) a[fm] = lds_read16(sA, wm * WTM + fm * 32 + (lane & 31), c);
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) b[fn] = lds_read16(sB, wn * WTN + fn * 32 + (lane & 31), c);
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) mma_step<E>(acc[fm][fn], a[fm], b[fn]);
    }
  }

  // acc = A[a_row0 : a_row0+BM, :K] * B[b_row0 : b_row0+BN, :K]^T.
  // Leaves the block synchronised (the LDS stages may be reused afterwards).
  __device__ __forceinline__ void run(const char* __restrict__ A, int64_t lda_bytes,
                                      int64_t a_row0, int64_t a_rows,
                                      const char* __restrict__ B, int64_t ldb_bytes,
                                      int64_t b_row0, int64_t b_rows, int64_t kbytes,
                                      char* smem, int tid) {
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave % WGM;
    const int wn = wave / WGM;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[fm][fn][r] = 0.0f;

    TileLoader<BM> la;
    TileLoader<BN> lb;
    const int64_t nk = (kbytes + kRowBytes - 1) / kRowBytes;
    la.load(A, lda_bytes, a_row0, a_rows, 0, kbytes, tid);
    lb.load(B, ldb_bytes, b_row0, b_rows, 0, kbytes, tid);
    la.store(smem, tid);
    lb.store(smem + BM * kRowBytes, tid);
    __syncthreads();
    for (int64_t kt = 0; kt < nk; ++kt) {
      const bool more = kt + 1 < nk;
      if (more) {
        la.load(A, lda_bytes, a_row0, a_rows, (kt + 1) * kRowBytes, kbytes, tid);
        lb.load(B, ldb_bytes, b_row0, b_rows, (kt + 1) * kRowBytes, kbytes, tid);
      }
      const char* stage = smem + (kt & 1) * kStageBytes;
      compute_stage(stage, stage + BM * kRowBytes, lane, wm, wn);
      if (more) {
        char* next = smem + ((kt + 1) & 1) * kStageBytes;
        la.store(next, tid);
        lb.store(next + BM * kRowBytes, tid);
      }
      __syncthreads();
    }
  }

  // Row (A side) and column (B side) of output element r of block (fm, fn),
  // relative to the block tile origin.
  __device__ __forceinline__ static int row_of(int wm, int fm, int r, int lane) {
    return wm * WTM + fm * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
  }
  __device__ __forceinline__ static int col_of(int wn, int fn, int lane) {
    return wn * WTN + fn * 32 + (lane & 31);
  }
};

__device__ __forceinline__ float shfl_xor32(float v) { return __shfl_xor(v, 32, 64); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// 16-byte accesses with the non-temporal ("nt") cache policy, for streaming
// passes that read or write each byte once.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 load16_nt(const void* p) {
  const u32x4_t v = __builtin_nontemporal_load(static_cast<const u32x4_t*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void store16_nt(void* p, uint4 v) {
  __builtin_nontemporal_store(u32x4_t{v.x, v.y, v.z, v.w}, static_cast<u32x4_t*>(p));
}

template <typename E>
__device__ __forceinline__ typename E::storage to_storage(float x);
template <>
__device__ __forceinline__ uint16_t to_storage<Bf16>(float x) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(x));
}
template <>
__device__ __forceinline__ float to_storage<F32>(float x) {
  return x;
}

}  // namespace mls
