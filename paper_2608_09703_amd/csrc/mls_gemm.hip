// The two backward products of the LM head (the head is linear, paper
// section 2, "Modeling"), per vocabulary chunk, both products for every
// sub-model in one grouped launch:
//   grad_W_i[chunk] = G_i^T h_i       A = G_i^T slab [Vc, T_pad], B = h_i^T [d_i, T_pad]
//   grad_h_i       += G_i W_i[chunk]  A = G_i slab   [T_pad, Vc], B = W_i[chunk]^T [d_i, Vc]
// Both are NT tile products on the shared MFMA main loop; the transposed
// operands h_i^T and W_i[chunk]^T are produced by the transpose kernel below.
#include "mls_core.h"
#include "mls_device.h"
#include "mls_launch.h"

namespace mls {

namespace {

// One output element: fp32 C (overwritten or accumulated) or bf16 Cb (see GemmGroup).
__device__ __forceinline__ void store_out(const GemmGroup& g, int64_t idx, float v) {
  if (g.Cb) {
    if (g.Cpart) v += g.Cpart[idx];
    if (g.accumulate) v += __uint_as_float((uint32_t)g.Cb[idx] << 16);
    g.Cb[idx] = to_storage<Bf16>(v);
  } else {
    float* c = g.C + idx;
    *c = g.accumulate ? *c + v : v;
  }
}

template <typename E>
__global__ __launch_bounds__(kThreads, 2) void gemm_nt_kernel(GemmArgs a) {
  using Mma = TileMma<E, kGemmBM, kGemmBN, 2, 2>;
  constexpr int FM = Mma::FM;
  constexpr int FN = Mma::FN;
  __shared__ __attribute__((aligned(16))) char smem[Mma::kSmemBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % 2;
  const int wn = wave / 2;
  const int b = blockIdx.x;
  int gi = 0;
  for (int k = 1; k < a.ngroups; ++k)
    if (b >= a.g[k].tile_begin) gi = k;
  const GemmGroup& g = a.g[gi];
  const int local = b - g.tile_begin;
  const int tm = local % g.tiles_m;
  const int tn = local / g.tiles_m;
  const int64_t m0 = (int64_t)tm * kGemmBM;
  const int64_t n0 = (int64_t)tn * kGemmBN;

  Mma mma;
  mma.run(static_cast<const char*>(g.A), g.lda * E::kBytes, m0, g.rows,
          static_cast<const char*>(g.B), g.ldb * E::kBytes, n0, g.cols, g.K * E::kBytes, smem,
          tid);

#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const int64_t n = n0 + Mma::col_of(wn, fn, lane);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t m = m0 + Mma::row_of(wm, fm, r, lane);
        if (m < g.rows && n < g.cols) store_out(g, m * g.ldc + n, mma.acc[fm][fn][r]);
      }
    }
}

// bf16 path: 256 x 256 tiles, 8 waves (2 per SIMD), direct-to-LDS loads, 2
// stages of 64-wide K (each K-tile reads whole 128-byte lines of a K-contiguous
// operand); the next K-tile's loads are spread over the current one's K-steps. The head chunk (grad_h) and the slab and h (grad_W) are
// read in their stored layouts through transposing LDS reads, so no operand is
// ever transposed in memory.
constexpr int kWideBM = 256;
constexpr int kWideBN = 256;
using WideGemmH = WideMma<kWideBM, kWideBN, 2, 4, 2, 128, kLayoutKC, kLayoutMC, true>;
using WideGemmW = WideMma<kWideBM, kWideBN, 2, 4, 2, 128, kLayoutMC, kLayoutMC, true>;

// Loads and stores of one wave's part of an output tile through buffer
// descriptors over the tile's existing rows (rows past them read as 0 and are
// not written). Element (row, col) of the tile is at byte offset
// (row * ldc + col) * size; coff[fn] is the lane's part for column block fn,
// (its first row) * ldc + its column. A wave's 32-column block lies wholly
// inside or outside the output (widths are multiples of 64), so blocks past it
// are skipped by a uniform branch (ok[fn]). INSIDE (all of the tile's rows
// exist): the (fm, r) part of the row goes into the scalar offset; otherwise
// every element gets its own vector offset, which the descriptor checks. Each
// kind of load is one loop with no branch inside, so a wave's loads are all in
// flight together.
// Cache policy of the fp32 output stores and of the reads of an fp32 output
// into the accumulators: non-temporal ("nt"), as each such element is touched
// once per launch. With the stores the headline step's GEMMs and the forward
// that follows them ran 0.01-0.02 ms faster each (7.76 -> 7.71 ms per step
// together with the forward's non-temporal slab stores); the reads took the
// GEMMs from 4.43-4.45 to 4.41-4.42 ms per step.
constexpr int kStoreNT = 2;

template <class Mma, bool INSIDE>
struct TileIo {
  static constexpr int FM = Mma::FM;
  static constexpr int FN = Mma::FN;
  typedef f32x16_t Acc[FM][FN];

  __device__ __forceinline__ static int rrow(int fm, int r) { return fm * 32 + 8 * (r >> 2) + (r & 3); }
  __device__ __forceinline__ static uint32_t voff(const uint32_t* coff, int ldc, int fm, int fn,
                                                  int r, int size) {
    if (INSIDE) return coff[fn] * (uint32_t)size;
    return (coff[fn] + (uint32_t)(rrow(fm, r) * ldc)) * (uint32_t)size;
  }
  __device__ __forceinline__ static int soff(int ldc, int fm, int r, int size) {
    return INSIDE ? rrow(fm, r) * ldc * size : 0;
  }
  __device__ __forceinline__ static float ld32(__amdgpu_buffer_rsrc_t rs, const uint32_t* coff,
                                               int ldc, int fm, int fn, int r) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                         rs, voff(coff, ldc, fm, fn, r, 4), soff(ldc, fm, r, 4),
                                         kStoreNT));
  }
  __device__ __forceinline__ static float ld16(__amdgpu_buffer_rsrc_t rs, const uint32_t* coff,
                                               int ldc, int fm, int fn, int r) {
    return __uint_as_float((uint32_t)__builtin_amdgcn_raw_buffer_load_b16(
                               rs, voff(coff, ldc, fm, fn, r, 2), soff(ldc, fm, r, 2), 0)
                           << 16);
  }

  // acc = Cpart (if part) + old output (if acc_old; bf16 when out16); blocks
  // past the output are left as they are (never stored)
  __device__ __forceinline__ static void init(Acc& acc, __amdgpu_buffer_rsrc_t rc,
                                              __amdgpu_buffer_rsrc_t rp, const uint32_t* coff,
                                              const bool* ok, int ldc, bool part, bool acc_old,
                                              bool out16) {
    if (part) {
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
        if (ok[fn]) {
#pragma unroll
          for (int fm = 0; fm < FM; ++fm)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[fm][fn][r] = ld32(rp, coff, ldc, fm, fn, r);
        }
      if (acc_old) {  // and the old bf16 output: one column block at a time
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) {
          if (!ok[fn]) continue;
          float old[FM][16];
#pragma unroll
          for (int fm = 0; fm < FM; ++fm)
#pragma unroll
            for (int r = 0; r < 16; ++r) old[fm][r] = ld16(rc, coff, ldc, fm, fn, r);
#pragma unroll
          for (int fm = 0; fm < FM; ++fm)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[fm][fn][r] += old[fm][r];
        }
      }
    } else if (out16) {
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
        if (ok[fn]) {
#pragma unroll
          for (int fm = 0; fm < FM; ++fm)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[fm][fn][r] = ld16(rc, coff, ldc, fm, fn, r);
        }
    } else {
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
        if (ok[fn]) {
#pragma unroll
          for (int fm = 0; fm < FM; ++fm)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[fm][fn][r] = ld32(rc, coff, ldc, fm, fn, r);
        }
    }
  }

  __device__ __forceinline__ static void store(const Acc& acc, __amdgpu_buffer_rsrc_t rc,
                                               const uint32_t* coff, const bool* ok, int ldc,
                                               bool out16) {
    if (out16) {
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
        if (!ok[fn]) continue;
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            __builtin_amdgcn_raw_buffer_store_b16(to_storage<Bf16>(acc[fm][fn][r]), rc,
                                                  voff(coff, ldc, fm, fn, r, 2), soff(ldc, fm, r, 2), 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
        if (!ok[fn]) continue;
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc[fm][fn][r]), rc,
                                                  voff(coff, ldc, fm, fn, r, 4), soff(ldc, fm, r, 4),
                                                  kStoreNT);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
};

template <class Mma>
__device__ __forceinline__ void wide_tile(const GemmGroup& g, int tm, int tn, int64_t mext,
                                          int64_t next, char* smem, int tid) {
  constexpr int FM = Mma::FM;
  constexpr int FN = Mma::FN;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % Mma::kWGM;
  const int wn = wave / Mma::kWGM;
  const int64_t m0 = (int64_t)tm * Mma::kBM;
  const int64_t n0 = (int64_t)tn * Mma::kBN;
  // Output through buffer descriptors over the tile's rows [m0, m0 + BM) that
  // exist (rows past mext fall outside them: their loads return 0 and their
  // stores are dropped), so each element's address is a 32-bit offset.
  const int64_t rows = mext - m0 < Mma::kBM ? mext - m0 : Mma::kBM;
  const bool out16 = g.Cb != nullptr;
  const __amdgpu_buffer_rsrc_t rc =
      out16 ? uniform_rsrc(reinterpret_cast<const char*>(g.Cb + m0 * g.ldc), (int)(rows * g.ldc * 2))
            : uniform_rsrc(reinterpret_cast<const char*>(g.C + m0 * g.ldc), (int)(rows * g.ldc * 4));
  const bool part = out16 && g.Cpart;
  const __amdgpu_buffer_rsrc_t rp = uniform_rsrc(
      reinterpret_cast<const char*>(part ? g.Cpart + m0 * g.ldc : g.C), part ? (int)(rows * g.ldc * 4) : 0);
  const bool acc_old = g.accumulate != 0;
  const int ldc = (int)g.ldc;

  uint32_t coff[FN];
  bool ok[FN];
  const int wnu = __builtin_amdgcn_readfirstlane(wn);
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) {
    const int col = (int)n0 + Mma::col_of(wn, fn, lane);
    coff[fn] = (uint32_t)(Mma::row_of(wm, 0, 0, lane) * ldc + col);
    ok[fn] = n0 + wnu * Mma::WTN + fn * 32 < next;  // the whole 32-column block (wave-uniform)
  }
  const bool inside = m0 + Mma::kBM <= mext;

  // A read-modify-write output (accumulate, or the fp32 partial sums of
  // earlier chunks) is read straight into the accumulators before the K loop,
  // so the product is added to it there and the epilogue only stores; the
  // reads' latency overlaps the first K-tile's loads.
  Mma mma;
  mma.run_from(static_cast<const char*>(g.A), g.lda * 2, m0, g.rows, static_cast<const char*>(g.B),
               g.ldb * 2, n0, g.cols, g.K * 2, smem, tid, [&]() {
                 if (!part && !acc_old)
                   mma.zero();
                 else if (inside)
                   TileIo<Mma, true>::init(mma.acc, rc, rp, coff, ok, ldc, part, acc_old, out16);
                 else
                   TileIo<Mma, false>::init(mma.acc, rc, rp, coff, ok, ldc, part, acc_old, out16);
               });
  if (inside)
    TileIo<Mma, true>::store(mma.acc, rc, coff, ok, ldc, out16);
  else
    TileIo<Mma, false>::store(mma.acc, rc, coff, ok, ldc, out16);
}

template <class MmaH, class MmaW>
__global__ __launch_bounds__(MmaH::NT, 1) void gemm_wide_kernel(GemmArgs a, int nb) {
  static_assert(MmaH::kSmemBytes == MmaW::kSmemBytes && MmaH::NT == MmaW::NT, "one footprint");
  __shared__ __attribute__((aligned(16))) char smem[MmaH::kSmemBytes];
  const int b = xcd_remap_phased(blockIdx.x, nb, a.phase_tiles);
  int gi = 0;
  for (int k = 1; k < a.ngroups; ++k)
    if (b >= a.g[k].tile_begin) gi = k;
  const GemmGroup& g = a.g[gi];
  const int local = b - g.tile_begin;
  int tm, tn;
  if (g.group_m > 0) {
    tile_coords(local, g.tiles_m, g.tiles_n, g.group_m, tm, tn);
  } else {
    tn = local % g.tiles_n;
    tm = local / g.tiles_n;
  }
  // output extents: rows of C (grad_h: tokens; grad_W: chunk vocabulary rows) and
  // its columns (the width)
  const int64_t mext = g.ldc_rows;
  const int64_t next = g.ldc;
  if (g.kind == 0)
    wide_tile<MmaH>(g, tm, tn, mext, next, smem, threadIdx.x);
  else
    wide_tile<MmaW>(g, tm, tn, mext, next, smem, threadIdx.x);
}

template <typename S>
__global__ __launch_bounds__(kThreads) void transpose_kernel(TransposeArgs a) {
  const TransposeJob& j = a.j[blockIdx.z];
  const int64_t rb = (int64_t)blockIdx.x * 64;
  const int64_t cb = (int64_t)blockIdx.y * 64;
  if (rb >= j.out_rows || cb >= j.cols) return;
  __shared__ S tile[64][65];
  const int tx = threadIdx.x & 63;
  const int ty = threadIdx.x >> 6;
  const S* src = static_cast<const S*>(j.src);
  S* dst = static_cast<S*>(j.dst);
  for (int rr = ty; rr < 64; rr += 4) {
    const int64_t r = rb + rr;
    const int64_t c = cb + tx;
    S v = S(0);
    if (r < j.out_rows && c < j.cols && j.r0 + r < j.src_rows) v = src[(j.r0 + r) * j.ld_src + c];
    tile[rr][tx] = v;
  }
  __syncthreads();
  for (int cc = ty; cc < 64; cc += 4) {
    const int64_t c = cb + cc;
    const int64_t r = rb + tx;
    if (c < j.cols && r < j.out_rows) dst[c * j.ld_dst + r] = tile[tx][cc];
  }
}

}  // namespace

int gemm_tile_rows(bool wide) { return wide ? kWideBM : kGemmBM; }
int gemm_tile_cols(bool wide) { return wide ? kWideBN : kGemmBN; }
int gemm_wide_k_tile() { return WideGemmH::BK; }

hipError_t launch_gemm_wide(const GemmArgs& a, int total_tiles, hipStream_t stream) {
  if (total_tiles <= 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_wide_kernel<WideGemmH, WideGemmW>), dim3(total_tiles),
                     dim3(WideGemmH::NT), 0, stream, a, total_tiles);
  return hipGetLastError();
}

hipError_t launch_gemm_nt(const GemmArgs& a, int total_tiles, bool f32, hipStream_t stream) {
  if (total_tiles <= 0) return hipSuccess;
  if (f32)
    hipLaunchKernelGGL(gemm_nt_kernel<F32>, dim3(total_tiles), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(gemm_nt_kernel<Bf16>, dim3(total_tiles), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_transpose(const TransposeArgs& a, int64_t max_out_rows, int64_t max_cols,
                            bool f32, hipStream_t stream) {
  if (a.njobs <= 0) return hipSuccess;
  dim3 grid((unsigned)((max_out_rows + 63) / 64), (unsigned)((max_cols + 63) / 64),
            (unsigned)a.njobs);
  if (f32)
    hipLaunchKernelGGL(transpose_kernel<float>, grid, dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(transpose_kernel<uint16_t>, grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace mls
