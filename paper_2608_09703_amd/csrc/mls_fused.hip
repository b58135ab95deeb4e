// Fused LM-head logits kernels: one block owns a 128 (vocabulary) x 128 (token)
// tile and computes it for every sub-model, teacher first.
//
// Forward (per tile, per sub-model i, per token t): the online log-sum-exp
// statistics of paper section 2 ("Modeling": logits of every head;
// "Integrated Distillation": eq. (2) needs the teacher's softmax next to every
// student's). The teacher's tile is computed first and its exponentials
// e_v = exp((l_s,v - max) / tau) stay in registers, laid out exactly like the
// accumulators of the students' tiles, so each student adds its cross term
// sum_v e_v l_i,v with no extra memory traffic. Only partial rows (max, sum
// exp, sum exp / tau, cross term), one per wave row of the tile, leave the
// block.
//
// Backward (per vocabulary chunk): logits are recomputed tile by tile, the
// teacher's q = softmax(l_s / tau) is formed once per tile and reused by every
// student, and the logit gradient
//   G_i = ( g_ce,i (softmax(l_i) - onehot(y)) + g_kl,i / tau (softmax(l_i / tau) - q) ) / N
// (eq. (2) with stop_grad on q, eq. (3) through the coefficients) is written
// to the chunk slab in two layouts for the two backward GEMMs.
#include <math.h>

#include "mls_core.h"
#include "mls_device.h"
#include "mls_launch.h"

namespace mls {

namespace {

// Tile cores: the general one (any width, fp32 or bf16) and the wide bf16 one
// (widths multiples of 64).
using GenMmaBf16 = TileMma<Bf16, kFusedBM, kFusedBN, 2, 2>;
using GenMmaF32 = TileMma<F32, kFusedBM, kFusedBN, 2, 2>;
using WideFused = WideMma<kFusedWideBM, kFusedBN, 2, 2, 2>;  // 2 blocks per CU

// Per-lane copy of the teacher's tile values (its softmax weights), laid out
// like the accumulators. The bf16 paths keep them as packed fp16 pairs (half
// the registers; probabilities lie in [0, 1], where fp16 rounds to 2^-11
// relative and flushes below 2^-24, an absolute error under 3e-8), the fp32
// path in fp32.
template <int FM, int FN, bool PACK>
struct TeacherTile;

template <int FM, int FN>
struct TeacherTile<FM, FN, false> {
  float v[FM][FN][16];
  __device__ __forceinline__ void set(int fm, int fn, int r, float x) { v[fm][fn][r] = x; }
  __device__ __forceinline__ float get(int fm, int fn, int r) const { return v[fm][fn][r]; }
};

template <int FM, int FN>
struct TeacherTile<FM, FN, true> {
  uint32_t v[FM][FN][8];
  __device__ __forceinline__ void set(int fm, int fn, int r, float x) {
    const uint32_t b = __builtin_bit_cast(uint16_t, (_Float16)x);
    if (r & 1)
      v[fm][fn][r >> 1] = (v[fm][fn][r >> 1] & 0xffffu) | (b << 16);
    else
      v[fm][fn][r >> 1] = b;
  }
  __device__ __forceinline__ float get(int fm, int fn, int r) const {
    const uint32_t w = v[fm][fn][r >> 1];
    return (float)__builtin_bit_cast(_Float16, (uint16_t)((r & 1) ? (w >> 16) : (w & 0xffffu)));
  }
};

// Forward tile kernel: for each sub-model (the teacher first) the logit tile
// of BM vocabulary rows x BN tokens, reduced in registers to one partial record
// (max, sum exp, sum exp at tau, teacher-weighted logit sum) per token and wave
// row. Each wave normalises to the max over its own rows, so the epilogue needs
// no exchange between waves; the row merge rescales the records.
// STORE (fused forward + backward): every logit also goes to the chunk's slab as
// fp16 of its distance to the record's maximum (at most 0; 2^-11 relative, so
// the entries that carry the softmax's mass, near the maximum, are the most
// exact), token-major, for the logit gradient pass.
template <class Mma, typename E, bool TAU1, int MINB = 1, bool STORE = false>
__global__ __launch_bounds__(Mma::NT, MINB) void fused_fwd_kernel(FusedArgs a) {
  constexpr int BM = Mma::kBM;
  constexpr int BN = Mma::kBN;
  constexpr int WGM = Mma::kWGM;
  constexpr int FM = Mma::FM;
  constexpr int FN = Mma::FN;
  static_assert(WGM == kFusedFwdParts, "one partial record per wave row");
  static_assert(BN == kFusedBN, "partial records are grouped by token tile");
  __shared__ __attribute__((aligned(16))) char smem[Mma::kSmemBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % WGM;
  const int wn = wave / WGM;
  const int hi = lane >> 5;
  const int bl = xcd_remap(blockIdx.x, gridDim.x);
  int vt, tt;
  tile_coords(bl, a.n_vt, a.n_tt, a.group_v, vt, tt);
  const int64_t vbase = (int64_t)vt * BM;
  const int64_t tbase = (int64_t)tt * BN;
  const bool full = vbase + BM <= a.V;
  const float ct = kLog2e * a.inv_tau;
  // records of sub-model order[oi] and token tile tt: [n_vt * WGM][BN]
  const int64_t n_rec = (int64_t)a.n_vt * WGM;
  const int64_t rec = (int64_t)vt * WGM + wm;

  // teacher weights exp((l_s - max_s) / tau); 0 outside V
  TeacherTile<FM, FN, false> e_t;
  Mma mma;

  for (int oi = 0; oi < a.M; ++oi) {
    const int i = a.order[oi];
    const int64_t kb = a.d[i] * E::kBytes;
    mma.run(static_cast<const char*>(a.W[i]), kb, vbase, a.V, static_cast<const char*>(a.h[i]),
            kb, tbase, a.T, kb, smem, tid);

#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      // 1. max of the token column over the wave's valid vocabulary rows
      // (-inf when all of them lie beyond V)
      float mb = -INFINITY;
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const bool ok = full || vbase + Mma::row_of(wm, fm, r, lane) < a.V;
          if (ok) mb = fmaxf(mb, mma.acc[fm][fn][r]);
        }
      mb = fmaxf(mb, shfl_xor32(mb));

      if constexpr (STORE && TAU1) {
        // The wave's 64 rows x 32 tokens go through its own 4 KB of LDS, token
        // by token (16-byte chunks XOR-swizzled with the token), and leave as
        // whole 128-byte lines of token-major slab rows: eight lines per store
        // instruction instead of 32 partial ones. The staging area is the
        // second pipeline stage, which is idle here: the product just ended
        // with a barrier after every wave's last read, and the next product
        // fills only the first stage before its first barrier, which no wave
        // passes before every wave's staging reads are done (stage_barrier
        // drains them). Only this wave touches its area and its LDS accesses
        // complete in order, so no barrier is needed here. The slab lines are
        // written with the non-temporal policy (forward 2.82 -> 2.78 ms per
        // step at the headline shape).
        static_assert(Mma::kStageBytes >= Mma::NW * 32 * 128 && Mma::WTM == 64, "staging fits");
        char* stg = smem + Mma::kStageBytes + wave * 32 * 128;
        const int c = lane & 31;  // token inside the 32-token block
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
#pragma unroll
          for (int rg = 0; rg < 4; ++rg) {
            uint32_t w[2];
#pragma unroll
            for (int k = 0; k < 2; ++k) {
              const float x0 = mma.acc[fm][fn][rg * 4 + 2 * k] - mb;
              const float x1 = mma.acc[fm][fn][rg * 4 + 2 * k + 1] - mb;
              w[k] = (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)x0) |
                     ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)x1) << 16);
            }
            const int chunk = (fm * 4 + rg) ^ (c & 7);  // 8 vocabulary rows per chunk
            *reinterpret_cast<uint2*>(stg + c * 128 + chunk * 16 + hi * 8) = make_uint2(w[0], w[1]);
          }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        uint16_t* rows = a.lslab + ((int64_t)i * a.n_tt * BN + tbase + wn * Mma::WTN + fn * 32) *
                                       a.ld_lslab + vbase + wm * Mma::WTM;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int tr = q * 8 + (lane >> 3);
          const int kk = lane & 7;
          const uint4 v = *reinterpret_cast<const uint4*>(stg + tr * 128 + ((kk ^ (tr & 7)) << 4));
          store16_nt(rows + (int64_t)tr * a.ld_lslab + kk * 8, v);
        }
      }
      if constexpr (STORE && !TAU1) {
        // At tau != 1 the staging's registers cost spills (the teacher's fp32
        // weights are live), so four consecutive vocabulary rows of one token
        // go out per 8-byte store instead: the two lane halves fill 16
        // contiguous bytes, a wave's 64 rows one 128-byte line per token. These
        // partial lines keep the default cache policy, under which the L2
        // combines them (non-temporal, the C3 forward took 22.4 ms, not 14.6).
        const int c = Mma::col_of(wn, fn, lane);
        uint16_t* row = a.lslab + ((int64_t)i * a.n_tt * BN + tbase + c) * a.ld_lslab + vbase;
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
#pragma unroll
          for (int rg = 0; rg < 4; ++rg) {
            uint32_t w[2];
#pragma unroll
            for (int k = 0; k < 2; ++k) {
              const float x0 = mma.acc[fm][fn][rg * 4 + 2 * k] - mb;
              const float x1 = mma.acc[fm][fn][rg * 4 + 2 * k + 1] - mb;
              w[k] = (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)x0) |
                     ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)x1) << 16);
            }
            *reinterpret_cast<uint2*>(row + Mma::row_of(wm, fm, rg * 4, lane)) = make_uint2(w[0], w[1]);
          }
      }

      // 2. sums relative to that max (every term is 0 on rows beyond V)
      float s1 = 0.f, st = 0.f, xr = 0.f;
      if (oi == 0) {
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const bool ok = full || vbase + Mma::row_of(wm, fm, r, lane) < a.V;
            const float l = mma.acc[fm][fn][r];
            const float x = l - mb;
            const float e = ok ? fast_exp2(x * ct) : 0.f;
            e_t.set(fm, fn, r, e);
            st += e;
            xr = fmaf(e, l, xr);
            if (!TAU1) s1 += ok ? fast_exp2(x * kLog2e) : 0.f;
          }
        if (TAU1) s1 = st;
      } else {
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const bool ok = full || vbase + Mma::row_of(wm, fm, r, lane) < a.V;
            const float l = mma.acc[fm][fn][r];
            const float x = l - mb;
            s1 += ok ? fast_exp2(x * kLog2e) : 0.f;
            if (!TAU1) st += ok ? fast_exp2(x * ct) : 0.f;
            xr = fmaf(e_t.get(fm, fn, r), l, xr);
          }
        if (TAU1) st = s1;
      }
      s1 += shfl_xor32(s1);
      st += shfl_xor32(st);
      xr += shfl_xor32(xr);

      // 3. the wave's partial record of this token
      const int c = Mma::col_of(wn, fn, lane);
      if (hi == 0 && tbase + c < a.T)
        a.partials[(((int64_t)oi * a.n_tt + tt) * n_rec + rec) * BN + c] = make_float4(mb, s1, st, xr);
    }
  }
}

template <typename E>
__device__ __forceinline__ void store4(typename E::storage* p, float a0, float a1, float a2,
                                       float a3);
template <>
__device__ __forceinline__ void store4<Bf16>(uint16_t* p, float a0, float a1, float a2,
                                             float a3) {
  uint2 v;
  v.x = (uint32_t)to_storage<Bf16>(a0) | ((uint32_t)to_storage<Bf16>(a1) << 16);
  v.y = (uint32_t)to_storage<Bf16>(a2) | ((uint32_t)to_storage<Bf16>(a3) << 16);
  *reinterpret_cast<uint2*>(p) = v;
}
template <>
__device__ __forceinline__ void store4<F32>(float* p, float a0, float a1, float a2, float a3) {
  *reinterpret_cast<float4*>(p) = make_float4(a0, a1, a2, a3);
}

template <class Mma, typename E, bool TAU1>
__global__ __launch_bounds__(Mma::NT, 1) void fused_bwd_kernel(FusedArgs a) {
  constexpr int BM = Mma::kBM;
  constexpr int BN = Mma::kBN;
  constexpr int WGM = Mma::kWGM;
  using S = typename E::storage;
  constexpr int FM = Mma::FM;
  constexpr int FN = Mma::FN;
  __shared__ __attribute__((aligned(16))) char smem[Mma::kSmemBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % WGM;
  const int wn = wave / WGM;
  const int bl = xcd_remap(blockIdx.x, gridDim.x);
  int vt, tt;
  tile_coords(bl, a.n_vt, a.n_tt, a.group_v, vt, tt);
  const int64_t vloc = (int64_t)vt * BM;  // row offset inside the chunk
  const int64_t vbase = a.v0 + vloc;      // absolute vocabulary row
  const int64_t tbase = (int64_t)tt * BN;
  const bool full = vbase + BM <= a.V;
  const int nv = *a.n_valid;
  const float invN = nv > 0 ? 1.0f / (float)nv : 0.0f;

  int64_t tok[FN];
  int ylab[FN];  // label row relative to the tile, or -1
  bool rv[FN];
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) {
    const int64_t t = tbase + Mma::col_of(wn, fn, lane);
    tok[fn] = t;
    const int64_t y = t < a.T ? a.labels[t] : a.ignore_index;
    rv[fn] = t < a.T && y != a.ignore_index && y >= 0 && y < a.V;
    const int64_t rel = y - vbase;
    ylab[fn] = (rv[fn] && rel >= 0 && rel < BM) ? (int)rel : -1;
  }

  // teacher softmax at tau; 0 outside V and on invalid rows
  TeacherTile<FM, FN, E::kBytes == 2> q_t;
  Mma mma;

  for (int oi = 0; oi < a.M; ++oi) {
    const int i = a.order[oi];
    const int64_t kb = a.d[i] * E::kBytes;
    mma.run(static_cast<const char*>(a.W[i]), kb, vbase, a.V, static_cast<const char*>(a.h[i]),
            kb, tbase, a.T, kb, smem, tid);
    const float gce = a.g_ce ? a.g_ce[i] : a.host_gce[i];
    const float gkl = a.g_kl ? a.g_kl[i] : a.host_gkl[i];
    S* slab = static_cast<S*>(a.slab) + (int64_t)i * a.T_pad * a.Vc;
    S* slabT = static_cast<S*>(a.slabT) + (int64_t)i * a.T_pad * a.Vc;

#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const int64_t t = tok[fn];
      // invalid rows: +inf log-normalisers make every probability 0
      const float l1 = rv[fn] ? a.lse1[(int64_t)i * a.T + t] : INFINITY;
      const float lt = rv[fn] ? a.lset[(int64_t)i * a.T + t] : INFINITY;
      const float cg = rv[fn] ? gce * invN : 0.f;
      const float ck = (rv[fn] && oi != 0) ? gkl * invN * a.inv_tau : 0.f;
      const float l1s = l1 * kLog2e;
      const float lts = lt * kLog2e;
      const float ct = kLog2e * a.inv_tau;
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          float g[4];
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            const int r = rg * 4 + rr;
            const int row = Mma::row_of(wm, fm, r, lane);
            const bool ok = full || vbase + row < a.V;
            const float l = mma.acc[fm][fn][r];
            const float oh = row == ylab[fn] ? 1.f : 0.f;
            if (oi == 0) {
              const float q = ok ? fast_exp2(fmaf(l, ct, -lts)) : 0.f;
              q_t.set(fm, fn, r, q);
              const float p1 = TAU1 ? q : (ok ? fast_exp2(fmaf(l, kLog2e, -l1s)) : 0.f);
              g[rr] = cg * (p1 - oh);
            } else {
              const float p1 = ok ? fast_exp2(fmaf(l, kLog2e, -l1s)) : 0.f;
              const float pt = TAU1 ? p1 : (ok ? fast_exp2(fmaf(l, ct, -lts)) : 0.f);
              g[rr] = fmaf(cg, p1 - oh, ck * (pt - q_t.get(fm, fn, r)));
            }
            // a selection, not a product: an ignored row's logits may be NaN
            g[rr] = rv[fn] ? g[rr] : 0.f;
          }
          const int row0 = Mma::row_of(wm, fm, rg * 4, lane);
          store4<E>(slab + t * a.Vc + vloc + row0, g[0], g[1], g[2], g[3]);
#pragma unroll
          for (int rr = 0; rr < 4; ++rr)
            slabT[(vloc + row0 + rr) * a.T_pad + t] = to_storage<E>(g[rr]);
        }
    }
  }
}

// Backward tile kernel of the wide bf16 core. Same arithmetic as
// fused_bwd_kernel; the bf16 logit-gradient tile is staged in LDS as
// [token][vocabulary] (16-byte chunks XOR-swizzled with the token index) and
// leaves the block as 16-byte coalesced stores of token-major slab rows. The
// gradient GEMMs read this one layout for both products.
template <class Mma, bool TAU1, int MINB>
__global__ __launch_bounds__(Mma::NT, MINB) void fused_bwd_wide_kernel(FusedArgs a) {
  constexpr int BM = Mma::kBM;  // vocabulary rows
  constexpr int BN = Mma::kBN;  // tokens
  constexpr int WGM = Mma::kWGM;
  constexpr int FM = Mma::FM;
  constexpr int FN = Mma::FN;
  constexpr int NT = Mma::NT;
  constexpr int kGRow = BM * 2;     // bytes per token row of the staged tile
  constexpr int kChunks = BM / 8;   // 16-byte chunks per token row
  constexpr int kCMask = kChunks - 1;
  static_assert((kChunks & kCMask) == 0 && kChunks <= 32, "row chunk count is a power of two");
  static_assert(BN * kGRow <= Mma::kSmemBytes, "staged tile fits in the stage memory");
  __shared__ __attribute__((aligned(16))) char smem[Mma::kSmemBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % WGM;
  const int wn = wave / WGM;
  const int bl = xcd_remap(blockIdx.x, gridDim.x);
  int vt, tt;
  tile_coords(bl, a.n_vt, a.n_tt, a.group_v, vt, tt);
  const int64_t vloc = (int64_t)vt * BM;
  const int64_t vbase = a.v0 + vloc;
  const int64_t tbase = (int64_t)tt * BN;
  const bool full = vbase + BM <= a.V;
  const int nv = *a.n_valid;
  const float invN = nv > 0 ? 1.0f / (float)nv : 0.0f;
  const float ct = kLog2e * a.inv_tau;

  int tcol[FN];
  int ylab[FN];
  bool rv[FN];
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) {
    tcol[fn] = Mma::col_of(wn, fn, lane);
    const int64_t t = tbase + tcol[fn];
    const int64_t y = t < a.T ? a.labels[t] : a.ignore_index;
    rv[fn] = t < a.T && y != a.ignore_index && y >= 0 && y < a.V;
    const int64_t rel = y - vbase;
    ylab[fn] = (rv[fn] && rel >= 0 && rel < BM) ? (int)rel : -1;
  }

  TeacherTile<FM, FN, true> q_t;
  Mma mma;

  for (int oi = 0; oi < a.M; ++oi) {
    const int i = a.order[oi];
    const int64_t kb = a.d[i] * 2;
    mma.run(static_cast<const char*>(a.W[i]), kb, vbase, a.V, static_cast<const char*>(a.h[i]),
            kb, tbase, a.T, kb, smem, tid);
    const float gce = a.g_ce ? a.g_ce[i] : a.host_gce[i];
    const float gkl = a.g_kl ? a.g_kl[i] : a.host_gkl[i];

    // 1. logit gradient -> bf16 tile in LDS
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const int64_t t = tbase + tcol[fn];
      const float l1 = rv[fn] ? a.lse1[(int64_t)i * a.T + t] : INFINITY;
      const float lt = rv[fn] ? a.lset[(int64_t)i * a.T + t] : INFINITY;
      const float cg = rv[fn] ? gce * invN : 0.f;
      const float ck = (rv[fn] && oi != 0) ? gkl * invN * a.inv_tau : 0.f;
      const float l1s = l1 * kLog2e;
      const float lts = lt * kLog2e;
      const int trow = tcol[fn];
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          float g[4];
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            const int r = rg * 4 + rr;
            const int row = Mma::row_of(wm, fm, r, lane);
            const bool ok = full || vbase + row < a.V;
            const float l = mma.acc[fm][fn][r];
            const float oh = row == ylab[fn] ? 1.f : 0.f;
            if (oi == 0) {
              const float q = ok ? fast_exp2(fmaf(l, ct, -lts)) : 0.f;
              q_t.set(fm, fn, r, q);
              const float p1 = TAU1 ? q : (ok ? fast_exp2(fmaf(l, kLog2e, -l1s)) : 0.f);
              g[rr] = cg * (p1 - oh);
            } else {
              const float p1 = ok ? fast_exp2(fmaf(l, kLog2e, -l1s)) : 0.f;
              const float pt = TAU1 ? p1 : (ok ? fast_exp2(fmaf(l, ct, -lts)) : 0.f);
              g[rr] = fmaf(cg, p1 - oh, ck * (pt - q_t.get(fm, fn, r)));
            }
            // a selection, not a product: an ignored row's logits may be NaN
            g[rr] = rv[fn] ? g[rr] : 0.f;
          }
          const int v0 = Mma::row_of(wm, fm, rg * 4, lane);  // multiple of 4
          uint2 w;
          w.x = (uint32_t)to_storage<Bf16>(g[0]) | ((uint32_t)to_storage<Bf16>(g[1]) << 16);
          w.y = (uint32_t)to_storage<Bf16>(g[2]) | ((uint32_t)to_storage<Bf16>(g[3]) << 16);
          const int off = trow * kGRow + ((((v0 >> 3) ^ (trow & kCMask))) << 4) + ((v0 >> 2) & 1) * 8;
          *reinterpret_cast<uint2*>(smem + off) = w;
          __builtin_amdgcn_sched_barrier(0);  // bound live ranges: one 4-row group at a time
        }
    }
    stage_barrier();  // the staged tile is complete before any wave copies it out

    // 2. token-major slab: BN rows x kChunks chunks of 16 bytes, whole lines with
    // the non-temporal policy (2.93 -> 2.81 ms per step of the recompute plan
    // at the headline shape)
    uint16_t* slab = static_cast<uint16_t*>(a.slab) + (int64_t)i * a.T_pad * a.Vc;
#pragma unroll 4
    for (int j = 0; j < BN * kChunks / NT; ++j) {
      const int idx = tid + NT * j;
      const int t = idx / kChunks;
      const int c = idx & kCMask;
      const uint4 v = *reinterpret_cast<const uint4*>(smem + t * kGRow + ((c ^ (t & kCMask)) << 4));
      store16_nt(slab + (tbase + t) * a.Vc + vloc + c * 8, v);
    }
    stage_barrier();  // the stage memory is refilled by the next tile product
  }
}

template <class Mma, typename E, bool TAU1>
hipError_t launch_fwd_t(const FusedArgs& a, hipStream_t stream) {
  dim3 grid((unsigned)a.n_tt * (unsigned)a.n_vt);
  hipLaunchKernelGGL((fused_fwd_kernel<Mma, E, TAU1>), grid, dim3(Mma::NT), 0, stream, a);
  return hipGetLastError();
}

template <class Mma, typename E, bool TAU1>
hipError_t launch_bwd_t(const FusedArgs& a, hipStream_t stream) {
  dim3 grid((unsigned)a.n_tt * (unsigned)a.n_vt);
  hipLaunchKernelGGL((fused_bwd_kernel<Mma, E, TAU1>), grid, dim3(Mma::NT), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

int fused_tile_rows(bool wide) { return wide ? kFusedWideBM : kFusedBM; }

hipError_t launch_fused_fwd(const FusedArgs& a, bool f32, hipStream_t stream) {
  const bool tau1 = a.tau == 1.0f;
  if (f32)
    return tau1 ? launch_fwd_t<GenMmaF32, F32, true>(a, stream)
                : launch_fwd_t<GenMmaF32, F32, false>(a, stream);
  if (a.wide) {
    dim3 grid((unsigned)a.n_tt * (unsigned)a.n_vt);
    if (a.lslab) {
      if (tau1)
        hipLaunchKernelGGL((fused_fwd_kernel<WideFused, Bf16, true, 2, true>), grid,
                           dim3(WideFused::NT), 0, stream, a);
      else
        hipLaunchKernelGGL((fused_fwd_kernel<WideFused, Bf16, false, 2, true>), grid,
                           dim3(WideFused::NT), 0, stream, a);
    } else if (tau1) {
      hipLaunchKernelGGL((fused_fwd_kernel<WideFused, Bf16, true, 2>), grid, dim3(WideFused::NT), 0,
                         stream, a);
    } else {
      hipLaunchKernelGGL((fused_fwd_kernel<WideFused, Bf16, false, 2>), grid, dim3(WideFused::NT), 0,
                         stream, a);
    }
    return hipGetLastError();
  }
  if (a.lslab) return hipErrorInvalidValue;  // the stored-logit forward is wide-only
  return tau1 ? launch_fwd_t<GenMmaBf16, Bf16, true>(a, stream)
              : launch_fwd_t<GenMmaBf16, Bf16, false>(a, stream);
}

hipError_t launch_fused_bwd(const FusedArgs& a, bool f32, hipStream_t stream) {
  const bool tau1 = a.tau == 1.0f;
  if (f32)
    return tau1 ? launch_bwd_t<GenMmaF32, F32, true>(a, stream)
                : launch_bwd_t<GenMmaF32, F32, false>(a, stream);
  if (a.wide) {
    dim3 grid((unsigned)a.n_tt * (unsigned)a.n_vt);
    if (tau1)
      hipLaunchKernelGGL((fused_bwd_wide_kernel<WideFused, true, 2>), grid, dim3(WideFused::NT), 0,
                         stream, a);
    else
      hipLaunchKernelGGL((fused_bwd_wide_kernel<WideFused, false, 2>), grid, dim3(WideFused::NT), 0,
                         stream, a);
    return hipGetLastError();
  }
  return tau1 ? launch_bwd_t<GenMmaBf16, Bf16, true>(a, stream)
              : launch_bwd_t<GenMmaBf16, Bf16, false>(a, stream);
}

}  // namespace mls
