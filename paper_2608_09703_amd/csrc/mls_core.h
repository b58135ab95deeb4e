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
//  - STAGES K-tiles of RB bytes (64 or 32 bf16) are in flight; a K-tile is consumed after an
//    explicit vmcnt wait and a plain s_barrier (no memory fence, so younger
//    loads stay in flight across the barrier);
//  - K must be a multiple of 64 (RB = 128) or 32 (RB = 64) and the operand
//    row stride at least K; a
//    panel must be below 4 GiB.
#pragma once

#include "mls_device.h"

namespace mls {

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glb_void_t;

// Buffer descriptor of a block-uniform base and byte count. The inputs pass
// through readfirstlane so the descriptor lives in scalar registers: values
// the compiler derived with vector instructions (tile coordinates from integer
// division) would otherwise leave it in vector registers, and every buffer
// load through it would then be wrapped in a loop over distinct descriptors.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t uniform_rsrc(const char* base, int bytes) {
  const uint64_t v = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  void* p = reinterpret_cast<void*>(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(p, (short)0, __builtin_amdgcn_readfirstlane(bytes),
                                           0x00020000);
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

__device__ __forceinline__ void block_barrier() { __builtin_amdgcn_s_barrier(); }

// Barrier after which other waves may overwrite LDS this wave has read: the
// wave's own LDS reads are drained first (s_barrier itself waits for nothing,
// and direct-to-LDS loads issued by other waves after the barrier reach LDS
// through the vector memory path, unordered with respect to reads still queued).
__device__ __forceinline__ void stage_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
}

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

// LDS placement for tiles whose rows hold RB bytes of K (RB = 128 or 64):
// 16-byte chunk c of row `row` lives at chunk position c ^ swz(row). For
// 128-byte rows, rows r..r+7 and r, r+8 differ; for 64-byte rows (4 chunks)
// the XOR is ((row >> 1) & 3) ^ (3 * bit3(row)), which is a bijection over 16
// aligned rows sharing row % 4 and over 8 aligned rows sharing row % 2, so
// fragment reads are conflict-free for 8- and 16-lane read phases alike.
template <int RB>
__device__ __forceinline__ int swz_chunk(int row, int c) {
  if (RB == 128) return c ^ (row & 7) ^ ((row >> 3) & 1);
  return c ^ ((row >> 1) & 3) ^ (((row >> 3) & 1) * 3);
}

template <int RB>
__device__ __forceinline__ uint4 lds_read16_rb(const char* base, int row, int c) {
  return *reinterpret_cast<const uint4*>(base + row * RB + (swz_chunk<RB>(row, c) << 4));
}

// Operand layouts: KC = row-major [m][k] (K contiguous, the MFMA's natural
// operand order); MC = row-major [k][m] (M contiguous). An MC tile is staged
// in LDS as stored (K-tile rows of BM*2 bytes) and its fragments are read with
// ds_read_b64_tr_b16, which hands lane i of each 16-lane group column m0+i of
// four consecutive rows. Two such reads give the 8 consecutive K values of
// one MFMA operand. Chunks of a staged row are XOR-swizzled with 4*(k % 4):
// the 32 lanes served together read 64 contiguous bytes from each of four
// rows, and the swizzle puts those four 64-byte pieces in distinct banks.
enum { kLayoutKC = 0, kLayoutMC = 1 };

typedef short v4s_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int mc_chunk(int krow, int c) { return c ^ ((krow & 3) << 2); }

__device__ __forceinline__ uint2 lds_read_tr8(const char* p) {
  const v4s_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4s_t*)((__attribute__((address_space(3))) char*)p));
  return __builtin_bit_cast(uint2, v);
}

// SPREAD: the next K-tile's loads are issued a few at a time over the first two
// K-steps of the current one instead of in one burst after the barrier, so their
// LDS writes interleave with the fragment reads while the last of them still
// has half a K-tile of lead. It pays where a K-tile lasts long (the 256 x 256
// GEMM tile), and costs where it does not (the 128 x 128 fused tiles).
template <int BM, int BN, int WGM, int WGN, int STAGES, int RB = 128, int ALAY = kLayoutKC,
          int BLAY = kLayoutKC, bool SPREAD = false>
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
  static constexpr int CPR = RB / 16;     // 16-byte chunks per LDS row (KC layout)
  static constexpr int KSTEPS = RB / 32;  // MFMA K-steps (16 bf16) per K-tile
  static constexpr int BK = RB / 2;       // K values per K-tile
  static constexpr int kStageBytes = (BM + BN) * RB;
  static constexpr int kSmemBytes = STAGES * kStageBytes;
  static constexpr int LA = BM * CPR / NT;  // load instructions per thread per K-tile, A
  static constexpr int LB = BN * CPR / NT;
  static constexpr int kLoadsPerTile = LA + LB;
  static_assert(RB == 128 || RB == 64, "LDS rows of 64 or 128 bytes");
  static_assert(BM * CPR % NT == 0 && BN * CPR % NT == 0, "tile must split evenly over the waves");
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
      const int row = slot / CPR;
      const int c = swz_chunk<RB>(row, slot % CPR);  // the XOR is an involution
      off[j] = (uint32_t)(row * ld_bytes) + (uint32_t)(c << 4);
    }
  }

  // MC operand: per-lane offsets of its chunks inside a K-tile of BK rows of
  // ROWS*2 bytes (relative to the tile's first row and the block's column m0).
  template <int ROWS, int L>
  __device__ __forceinline__ static void panel_offsets_mc(int64_t ld_bytes, int wave, int lane,
                                                          uint32_t* off) {
    constexpr int CPM = ROWS / 8;  // chunks per staged row
#pragma unroll
    for (int j = 0; j < L; ++j) {
      const int slot = (j * NW + wave) * 64 + lane;
      const int krow = slot / CPM;
      const int c = mc_chunk(krow, slot % CPM);
      off[j] = (uint32_t)(krow * ld_bytes) + (uint32_t)(c << 4);
    }
  }

  // MC operand panel: columns from m0 on, over the `nrows` stored rows (the
  // K extent that exists in memory); reads past the end return 0, so K-tiles
  // beyond nrows contribute nothing.
  __device__ __forceinline__ static __amdgpu_buffer_rsrc_t panel_rsrc_mc(const char* base,
                                                                         int64_t ld_bytes,
                                                                         int64_t m0, int64_t nrows) {
    const int64_t bytes = nrows * ld_bytes - m0 * 2;
    return uniform_rsrc(base + m0 * 2, (int)(bytes > 0 ? bytes : 0));
  }

  __device__ __forceinline__ static __amdgpu_buffer_rsrc_t panel_rsrc(const char* base,
                                                                      int64_t ld_bytes,
                                                                      int64_t row0, int64_t nrows,
                                                                      int rows) {
    int64_t avail = nrows - row0;
    avail = avail < rows ? avail : rows;
    avail = avail > 0 ? avail : 0;
    return uniform_rsrc(base + row0 * ld_bytes, (int)(avail * ld_bytes));
  }

  // Enqueue the direct loads of one operand tile. `vofs` is added to every
  // lane's offset (it takes part in the descriptor's range check); `sofs` is
  // the scalar offset (not range-checked, so only used where every lane's
  // address stays inside its row: the K position of a KC operand).
  template <int L>
  __device__ __forceinline__ static void issue_operand(__amdgpu_buffer_rsrc_t rsrc,
                                                       const uint32_t* off, uint32_t vofs,
                                                       int sofs, char* lds, int wave) {
#pragma unroll
    for (int j = 0; j < L; ++j) {
      char* dst = lds + (j * NW + wave) * 64 * 16;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void_t*)dst, 16, off[j] + vofs, sofs, 0,
                                               0);
    }
  }

  // Issues load j (0 .. LA + LB - 1) of one K-tile into stage `st`; ka / kb
  // are the tile's K positions as issue_operand takes them.
  __device__ __forceinline__ static void issue_one(int j, __amdgpu_buffer_rsrc_t ra,
                                                   __amdgpu_buffer_rsrc_t rb, const uint32_t* offa,
                                                   const uint32_t* offb, uint32_t ka, uint32_t kb,
                                                   char* st, int wave) {
    if (j < LA) {
      char* dst = st + (j * NW + wave) * 64 * 16;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void_t*)dst, 16,
                                               offa[j] + (ALAY == kLayoutKC ? 0u : ka),
                                               ALAY == kLayoutKC ? (int)ka : 0, 0, 0);
    } else {
      const int jb = j - LA;
      char* dst = st + BM * RB + (jb * NW + wave) * 64 * 16;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void_t*)dst, 16,
                                               offb[jb] + (BLAY == kLayoutKC ? 0u : kb),
                                               BLAY == kLayoutKC ? (int)kb : 0, 0, 0);
    }
  }

  // One MFMA operand fragment of an MC tile: row block `r0` (32 rows), K-step kk.
  template <int ROWS>
  __device__ __forceinline__ static uint4 mc_frag(const char* base, int r0, int kk, int lane) {
    constexpr int RBYTES = ROWS * 2;
    const int g = lane >> 4;
    const int j = lane & 15;
    const int m = r0 + (g & 1) * 16 + 4 * (j & 3);
    const int k = kk * 16 + (g >> 1) * 8 + (j >> 2);
    const int c = m >> 3;
    const int in = (m & 7) * 2;
    const uint2 lo = lds_read_tr8(base + k * RBYTES + (mc_chunk(k, c) << 4) + in);
    const uint2 hi = lds_read_tr8(base + (k + 4) * RBYTES + (mc_chunk(k + 4, c) << 4) + in);
    return make_uint4(lo.x, lo.y, hi.x, hi.y);
  }

  __device__ __forceinline__ void load_frags(const char* sA, const char* sB, int kk, int lane,
                                             int wm, int wn, uint4* a, uint4* b) {
    const int c = 2 * kk + (lane >> 5);
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      if (ALAY == kLayoutKC)
        a[fm] = lds_read16_rb<RB>(sA + wm * WTM * RB, fm * 32 + (lane & 31), c);
      else
        a[fm] = mc_frag<BM>(sA, wm * WTM + fm * 32, kk, lane);
    }
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      if (BLAY == kLayoutKC)
        b[fn] = lds_read16_rb<RB>(sB + wn * WTN * RB, fn * 32 + (lane & 31), c);
      else
        b[fn] = mc_frag<BN>(sB, wn * WTN + fn * 32, kk, lane);
    }
  }

  // `hook(kk)` runs at the start of K-step kk (the spread loads of the next K-tile).
  template <class Hook>
  __device__ __forceinline__ void compute_stage(const char* sA, const char* sB, int lane, int wm,
                                                int wn, Hook&& hook) {
    constexpr int kMfma = FM * FN;
    constexpr int kReads = (FM + FN) * ((ALAY == kLayoutMC || BLAY == kLayoutMC) ? 2 : 1);
    constexpr int kPer = kMfma / kReads > 0 ? kMfma / kReads : 1;  // MFMAs per read
    uint4 a[2][FM], b[2][FN];
    load_frags(sA, sB, 0, lane, wm, wn, a[0], b[0]);
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) {
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (SPREAD) {
        hook(kk);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (kk < KSTEPS - 1) load_frags(sA, sB, kk + 1, lane, wm, wn, a[(kk + 1) & 1], b[(kk + 1) & 1]);
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) mma_step<Bf16>(acc[fm][fn], a[kk & 1][fm], b[kk & 1][fn]);
      if (kk < KSTEPS - 1) {
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
  // a_rows / b_rows: rows of the stored operand matrix (M extent for a KC
  // operand, K extent for an MC operand; rows beyond it read as zero).
  // For an MC operand, a_row0 / b_row0 is the first column.
  // On return every wave has passed a barrier after its last LDS read, so the
  // LDS stages may be reused.
  __device__ __forceinline__ void run(const char* __restrict__ A, int64_t lda_bytes,
                                      int64_t a_row0, int64_t a_rows,
                                      const char* __restrict__ B, int64_t ldb_bytes,
                                      int64_t b_row0, int64_t b_rows, int64_t kbytes,
                                      char* smem, int tid) {
    run_from(A, lda_bytes, a_row0, a_rows, B, ldb_bytes, b_row0, b_rows, kbytes, smem, tid,
             [this]() { zero(); });
  }

  // As run(), with the accumulators set by init() instead of zeroed. init()
  // runs before any K-tile load is issued, so loads it issues are older than
  // the first K-tile's and are complete once that K-tile is (loads return in
  // order): their latency hides behind the pipeline's prologue.
  template <class Init>
  __device__ __forceinline__ void run_from(const char* __restrict__ A, int64_t lda_bytes,
                                           int64_t a_row0, int64_t a_rows,
                                           const char* __restrict__ B, int64_t ldb_bytes,
                                           int64_t b_row0, int64_t b_rows, int64_t kbytes,
                                           char* smem, int tid, Init&& init) {
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave % WGM;
    const int wn = wave / WGM;
    init();
    const int nk = (int)(kbytes / RB);
    // KC operands: panel of BM (BN) rows, K position as scalar byte offset.
    // MC operands: panel of BM (BN) columns, K position as scalar row offset.
    const __amdgpu_buffer_rsrc_t ra = ALAY == kLayoutKC
                                          ? panel_rsrc(A, lda_bytes, a_row0, a_rows, BM)
                                          : panel_rsrc_mc(A, lda_bytes, a_row0, a_rows);
    const __amdgpu_buffer_rsrc_t rb = BLAY == kLayoutKC
                                          ? panel_rsrc(B, ldb_bytes, b_row0, b_rows, BN)
                                          : panel_rsrc_mc(B, ldb_bytes, b_row0, b_rows);
    uint32_t offa[LA], offb[LB];
    if (ALAY == kLayoutKC)
      panel_offsets<LA>(lda_bytes, wave, lane, offa);
    else
      panel_offsets_mc<BM, LA>(lda_bytes, wave, lane, offa);
    if (BLAY == kLayoutKC)
      panel_offsets<LB>(ldb_bytes, wave, lane, offb);
    else
      panel_offsets_mc<BN, LB>(ldb_bytes, wave, lane, offb);
    // K position of tile t: KC operands move along the row (scalar offset);
    // MC operands move down BK rows (per-lane offset, range-checked).
    const uint32_t stepa = ALAY == kLayoutKC ? (uint32_t)RB : (uint32_t)(BK * lda_bytes);
    const uint32_t stepb = BLAY == kLayoutKC ? (uint32_t)RB : (uint32_t)(BK * ldb_bytes);
#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s) {
      if (s < nk) {
        char* st = smem + s * kStageBytes;
        const uint32_t ka = s * stepa, kb = s * stepb;
        issue_operand<LA>(ra, offa, ALAY == kLayoutKC ? 0u : ka, ALAY == kLayoutKC ? (int)ka : 0, st,
                          wave);
        issue_operand<LB>(rb, offb, BLAY == kLayoutKC ? 0u : kb, BLAY == kLayoutKC ? (int)kb : 0,
                          st + BM * RB, wave);
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
      // stage (kt - 1) % STAGES is refilled below: every wave's reads of it must
      // have completed
      stage_barrier();
      const int nt = kt + STAGES - 1;
      const char* stage = smem + (kt % STAGES) * kStageBytes;
      if constexpr (!SPREAD) {
        if (nt < nk) {
          char* st = smem + (nt % STAGES) * kStageBytes;
          const uint32_t ka = nt * stepa, kb = nt * stepb;
          issue_operand<LA>(ra, offa, ALAY == kLayoutKC ? 0u : ka, ALAY == kLayoutKC ? (int)ka : 0,
                            st, wave);
          issue_operand<LB>(rb, offb, BLAY == kLayoutKC ? 0u : kb, BLAY == kLayoutKC ? (int)kb : 0,
                            st + BM * RB, wave);
        }
        compute_stage(stage, stage + BM * RB, lane, wm, wn, [](int) {});
      } else {
        char* st = smem + (nt % STAGES) * kStageBytes;
        const uint32_t ka = nt * stepa, kb = nt * stepb;
        const bool more = nt < nk;
        compute_stage(stage, stage + BM * RB, lane, wm, wn, [&](int kk) {
          if (!more) return;
          // the tile's loads in the first two K-steps, the B panel's first (on the
          // 256 x 256 GEMM tile: B's four, then A's four; B, the head or the
          // hidden states, is re-read from L2 less often than the slab, so its
          // loads take longer): spread enough that their LDS writes do not land
          // in one burst, early enough that the last ones still have half a
          // K-tile to arrive before the next barrier
          constexpr int kSpreadSteps = KSTEPS < 2 ? KSTEPS : 2;
          constexpr int kPerStep = (kLoadsPerTile + kSpreadSteps - 1) / kSpreadSteps;
#pragma unroll
          for (int q = 0; q < kPerStep; ++q) {
            const int j = kk * kPerStep + q;
            if (j < kLoadsPerTile) issue_one((j + LA) % kLoadsPerTile, ra, rb, offa, offb, ka, kb, st, wave);
          }
        });
      }
    }
    stage_barrier();
  }

  __device__ __forceinline__ static int row_of(int wm, int fm, int r, int lane) {
    return wm * WTM + fm * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
  }
  __device__ __forceinline__ static int col_of(int wn, int fn, int lane) {
    return wn * WTN + fn * 32 + (lane & 31);
  }
};

}  // namespace mls
