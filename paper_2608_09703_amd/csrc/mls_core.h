// Wide-tile bf16 MFMA main loop with direct global->LDS loads (gfx950).
//
// Same product as TileMma (C[m][n] = sum_k A[m][k] B[n][k], both operands
// row-major with K contiguous, output layout of v_mfma_f32_32x32x16_bf16) for
// tiles of up to 256 x 256 and any number of waves. Differences:
//  - operands are moved from global memory straight into LDS with
//    buffer_load_dwordx4 ... lds (16 bytes per lane, no register staging);
//    each lane fetches the global chunk that belongs in its LDS slot under the
//    XOR swizzle of lds_off(), so fragment reads stay conflict-free. A buffer
//    descriptor covers the block's operand panel, so per-lane offsets are
//    32-bit, fixed for the whole K loop (the K position is a scalar offset),
//    and rows past the end of the operand read as zero;
//  - STAGES K-tiles of 64 bf16 are in flight; a K-tile is consumed after an
//    explicit vmcnt wait and a plain s_barrier (no memory fence, so younger
//    loads stay in flight across the barrier);
//  - K must be a multiple of 64 and the operand row stride at least K; a
//    panel must be below 4 GiB.
#pragma once

#include "mls_device.h"

namespace mls {

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glb_void_t;

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

__device__ __forceinline__ void block_barrier() { __builtin_amdgcn_s_barrier(); }

// Blocks are dispatched round-robin over the 8 XCDs of the chip; this gives
// each XCD a contiguous range of logical tile indices (a bijection on
// [0, nb)), so tiles that share operand panels share one L2.
__device__ __forceinline__ int xcd_remap(int b, int nb) {
  const int q = nb / 8;
  const int r = nb % 8;
  const int x = b % 8;
  return x * q + (x < r ? x : r) + b / 8;
}

// Like xcd_remap for a launch whose first n1 tiles cost more than the rest:
// every XCD gets an even share of each phase, as one contiguous range per
// phase. Requires every XCD's share of phase 1 to fit in its block count
// (the host passes n1 = 0, i.e. plain xcd_remap, otherwise).
__device__ __forceinline__ int xcd_remap_phased(int b, int nb, int n1) {
  if (n1 <= 0 || n1 >= nb) return xcd_remap(b, nb);
  const int x = b % 8;
  const int i = b / 8;
  const int q = n1 / 8;
  const int r = n1 % 8;
  const int q1 = q + (x < r ? 1 : 0);
  if (i < q1) return x * q + (x < r ? x : r) + i;
  int start2 = 0;
  for (int y = 0; y < x; ++y) start2 += (nb - y + 7) / 8 - (q + (y < r ? 1 : 0));
  return n1 + start2 + (i - q1);
}

// Logical tile index -> (vocabulary tile, token tile). Tiles are taken in
// groups of `group_v` vocabulary tiles; inside a group the vocabulary tile
// varies fastest, so the blocks resident on one XCD at a time cover a
// rectangle of about group_v vocabulary tiles x (32 / group_v) token tiles
// and both operand panels are re-read from L2 rather than from memory.
__device__ __forceinline__ void tile_coords(int bl, int n_vt, int n_tt, int group_v, int& vt,
                                            int& tt) {
  const int per_group = group_v * n_tt;
  const int g = bl / per_group;
  const int first = g * group_v;
  const int gsz = (n_vt - first) < group_v ? (n_vt - first) : group_v;
  const int in = bl - g * per_group;
  vt = first + in % gsz;
  tt = in / gsz;
}

template <int BM, int BN, int WGM, int WGN, int STAGES>
struct WideMma {
  static constexpr int kBM = BM;
  static constexpr int kBN = BN;
  static constexpr int kWGM = WGM;
  static constexpr int kWGN = WGN;
  static constexpr int NW = WGM * WGN;
  static constexpr int NT = NW * 64;
  static constexpr int WTM = BM / WGM;
  static constexpr int WTN = BN / WGN;
  static constexpr int FM = WTM / 32;
  static constexpr int FN = WTN / 32;
  static constexpr int kStageBytes = (BM + BN) * kRowBytes;
  static constexpr int kSmemBytes = STAGES * kStageBytes;
  static constexpr int LA = BM * 8 / NT;  // load instructions per thread per K-tile, A
  static constexpr int LB = BN * 8 / NT;
  static constexpr int kLoadsPerTile = LA + LB;
  static_assert(BM * 8 % NT == 0 && BN * 8 % NT == 0, "tile must split evenly over the waves");
  static_assert(STAGES >= 2 && STAGES <= 4, "2..4 stages");
  static_assert(kLoadsPerTile * (STAGES - 1) < 64, "vmcnt range");

  f32x16_t acc[FM][FN];

  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[fm][fn][r] = 0.0f;
  }

  // Per-lane byte offsets (inside the operand panel) of the L chunks this lane
  // moves for a ROWS x 128-byte tile; fixed for the whole K loop.
  template <int L>
  __device__ __forceinline__ static void panel_offsets(int64_t ld_bytes, int wave, int lane,
                                                       uint32_t* off) {
#pragma unroll
    for (int j = 0; j < L; ++j) {
      const int slot = (j * NW + wave) * 64 + lane;
      const int row = slot >> 3;
      const int c = (slot & 7) ^ (row & 7) ^ ((row >> 3) & 1);
      off[j] = (uint32_t)(row * ld_bytes) + (uint32_t)(c << 4);
    }
  }

  __device__ __forceinline__ static __amdgpu_buffer_rsrc_t panel_rsrc(const char* base,
                                                                      int64_t ld_bytes,
                                                                      int64_t row0, int64_t nrows,
                                                                      int rows) {
    int64_t avail = nrows - row0;
    avail = avail < rows ? avail : rows;
    avail = avail > 0 ? avail : 0;
    return __builtin_amdgcn_make_buffer_rsrc((void*)(base + row0 * ld_bytes), (short)0,
                                             (int)(avail * ld_bytes), 0x00020000);
  }

  // Enqueue the direct loads of one operand tile (the panel's 128 bytes at kb0).
  template <int L>
  __device__ __forceinline__ static void issue_operand(__amdgpu_buffer_rsrc_t rsrc,
                                                       const uint32_t* off, int kb0, char* lds,
                                                       int wave) {
#pragma unroll
    for (int j = 0; j < L; ++j) {
      char* dst = lds + (j * NW + wave) * 64 * 16;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void_t*)dst, 16, off[j], kb0, 0, 0);
    }
  }

  // Fragment reads of sub-step kk+1 are interleaved with the MFMAs of
  // sub-step kk (two register sets), so LDS latency hides behind the MFMA
  // chain while at most FM+FN reads are outstanding.
  __device__ __forceinline__ void load_frags(const char* pa, const char* pb, int kk, int lane,
                                             uint4* a, uint4* b) {
    const int c = 2 * kk + (lane >> 5);
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) a[fm] = lds_read16(pa, fm * 32 + (lane & 31), c);
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) b[fn] = lds_read16(pb, fn * 32 + (lane & 31), c);
  }

  __device__ __forceinline__ void compute_stage(const char* sA, const char* sB, int lane, int wm,
                                                int wn) {
    constexpr int kMfma = FM * FN;
    constexpr int kReads = FM + FN;
    constexpr int kPer = kMfma / kReads > 0 ? kMfma / kReads : 1;  // MFMAs per read
    const char* pa = sA + wm * WTM * kRowBytes;
    const char* pb = sB + wn * WTN * kRowBytes;
    uint4 a[2][FM], b[2][FN];
    load_frags(pa, pb, 0, lane, a[0], b[0]);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      __builtin_amdgcn_sched_barrier(0);
      if (kk < 3) load_frags(pa, pb, kk + 1, lane, a[(kk + 1) & 1], b[(kk + 1) & 1]);
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) mma_step<Bf16>(acc[fm][fn], a[kk & 1][fm], b[kk & 1][fn]);
      if (kk < 3) {
#pragma unroll
        for (int q = 0; q < kReads; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, kPer, 0);  // MFMA
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);     // DS read
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // acc = A[a_row0 : +BM, :K] * B[b_row0 : +BN, :K]^T with K = kbytes / 2.
  // On return every wave has passed a barrier after its last LDS read, so the
  // LDS stages may be reused.
  __device__ __forceinline__ void run(const char* __restrict__ A, int64_t lda_bytes,
                                      int64_t a_row0, int64_t a_rows,
                                      const char* __restrict__ B, int64_t ldb_bytes,
                                      int64_t b_row0, int64_t b_rows, int64_t kbytes,
                                      char* smem, int tid) {
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave % WGM;
    const int wn = wave / WGM;
    zero();
    const int nk = (int)(kbytes / kRowBytes);
    const __amdgpu_buffer_rsrc_t ra = panel_rsrc(A, lda_bytes, a_row0, a_rows, BM);
    const __amdgpu_buffer_rsrc_t rb = panel_rsrc(B, ldb_bytes, b_row0, b_rows, BN);
    uint32_t offa[LA], offb[LB];
    panel_offsets<LA>(lda_bytes, wave, lane, offa);
    panel_offsets<LB>(ldb_bytes, wave, lane, offb);
#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s) {
      if (s < nk) {
        char* st = smem + s * kStageBytes;
        issue_operand<LA>(ra, offa, s * kRowBytes, st, wave);
        issue_operand<LB>(rb, offb, s * kRowBytes, st + BM * kRowBytes, wave);
      }
    }
    for (int kt = 0; kt < nk; ++kt) {
      // tiles issued after kt that may stay in flight
      const int ahead = (nk - 1 - kt) < (STAGES - 2) ? (nk - 1 - kt) : (STAGES - 2);
      if (STAGES >= 4 && ahead >= 2) {
        wait_vmcnt<(STAGES >= 4 ? 2 : 0) * kLoadsPerTile>();
      } else if (STAGES >= 3 && ahead >= 1) {
        wait_vmcnt<(STAGES >= 3 ? 1 : 0) * kLoadsPerTile>();
      } else {
        wait_vmcnt<0>();
      }
      block_barrier();
      const int nt = kt + STAGES - 1;
      if (nt < nk) {
        char* st = smem + (nt % STAGES) * kStageBytes;
        issue_operand<LA>(ra, offa, nt * kRowBytes, st, wave);
        issue_operand<LB>(rb, offb, nt * kRowBytes, st + BM * kRowBytes, wave);
      }
      const char* stage = smem + (kt % STAGES) * kStageBytes;
      compute_stage(stage, stage + BM * kRowBytes, lane, wm, wn);
    }
    block_barrier();
  }

  __device__ __forceinline__ static int row_of(int wm, int fm, int r, int lane) {
    return wm * WTM + fm * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
  }
  __device__ __forceinline__ static int col_of(int wn, int fn, int lane) {
    return wn * WTN + fn * 32 + (lane & 31);
  }
};

}  // namespace mls
