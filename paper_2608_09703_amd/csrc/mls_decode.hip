// The head step of nested speculative decoding (paper section 2, paragraph
// "Speculative Decoding"; the measured setting of section 3, "Speculative
// Decoding Throughput": greedy or nucleus top-p 0.9 sampling at temperature
// 0.4, a smaller sub-model drafting gamma tokens and a larger one verifying).
//
// 1. head_logits_kernel: logits[t][v] = sum_k o[t][k] W[v][k] in fp32, on the
//    MFMA tile core (128 or 192 vocabulary rows x 128 tokens); the fp32 tile is
//    staged in LDS and leaves the block as 16-byte stores of token-major rows.
//    Decode batches are small, so the [rows, V] logits are cheap next to the
//    head itself.
// 2. sample_kernel: one 1024-thread block per row. The row's sampling
//    distribution is softmax(l / temperature) restricted to the nucleus: the
//    most probable tokens (ties: lower index first) up to and including the
//    first one at which the kept mass reaches top_p. The nucleus threshold is
//    the largest exp-weight value theta whose "weight >= theta" mass still
//    reaches top_p of the total, found by bisection on the fp32 bit pattern
//    (positive floats order like their bits); tokens tied at theta are kept in
//    index order as far as needed. A draw with uniform u returns the smallest
//    index whose cumulative kept weight in index order exceeds u times the
//    kept total.
// 3. verify_kernel: one block per sequence walks its gamma drafts: the draft
//    token x is kept when u * q(x) < p(x); at the first rejection the next
//    token is drawn from max(0, p - q); if all are kept, one more token is drawn
//    from the verifier's distribution after the drafts. Greedy mode compares
//    with the verifier's argmax (lowest index on ties).
//
// All reductions run in a fixed order, so results are bitwise reproducible.
#include <math.h>

#include "mls_core.h"
#include "mls_device.h"
#include "mls_launch.h"
#include "mls_wave.h"

namespace mls {

namespace {

// ---------------------------------------------------------------------------
// 1. head logits
// ---------------------------------------------------------------------------

template <class Mma, typename E>
__global__ __launch_bounds__(Mma::NT, 2) void head_logits_kernel(HeadArgs a) {
  constexpr int BM = Mma::kBM;  // vocabulary rows
  constexpr int BN = Mma::kBN;  // tokens
  constexpr int FM = Mma::FM;
  constexpr int FN = Mma::FN;
  constexpr int NT = Mma::NT;
  constexpr int kChunks = BM / 4;          // 16-byte chunks (4 floats) per token row of the tile
  constexpr int kSw = kChunks & -kChunks;  // chunk swizzle span: XOR stays inside aligned groups
  // the fp32 tile leaves in one pass, or in one pass per wave column when it
  // is larger than the stage memory
  constexpr int kPasses = (BN * BM * 4 + Mma::kSmemBytes - 1) / Mma::kSmemBytes;
  constexpr int kTok = BN / kPasses;  // tokens per pass
  static_assert(kPasses == 1 || kPasses == Mma::kWGN, "one pass, or one per wave column");
  static_assert(kTok * BM * 4 <= Mma::kSmemBytes, "a pass fits in the stage memory");
  __shared__ __attribute__((aligned(16))) char smem[Mma::kSmemBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % Mma::kWGM;
  const int wn = wave / Mma::kWGM;
  const int bl = xcd_remap(blockIdx.x, gridDim.x);
  int vt, tt;
  tile_coords(bl, a.n_vt, a.n_tt, a.group_v, vt, tt);
  const int64_t vbase = (int64_t)vt * BM;
  const int64_t tbase = (int64_t)tt * BN;
  const int64_t kb = a.d * E::kBytes;

  Mma mma;
  mma.run(static_cast<const char*>(a.W), kb, vbase, a.V, static_cast<const char*>(a.o), kb, tbase,
          a.T, kb, smem, tid);

  // stage: token row t of a pass holds kChunks chunks of 4 vocabulary entries,
  // chunk c at c ^ (t % kSw)
  float* st = reinterpret_cast<float*>(smem);
  const bool vec = (a.V & 3) == 0;
#pragma unroll
  for (int ps = 0; ps < kPasses; ++ps) {
    if (ps > 0) __syncthreads();  // every read of the previous pass is done
    if (kPasses == 1 || wn == ps) {
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
        const int t = Mma::col_of(wn, fn, lane) - ps * kTok;
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
#pragma unroll
          for (int rg = 0; rg < 4; ++rg) {
            const int v0 = Mma::row_of(wm, fm, rg * 4, lane);  // multiple of 4
            const float4 w = make_float4(mma.acc[fm][fn][rg * 4], mma.acc[fm][fn][rg * 4 + 1],
                                         mma.acc[fm][fn][rg * 4 + 2], mma.acc[fm][fn][rg * 4 + 3]);
            *reinterpret_cast<float4*>(st + t * BM + (((v0 >> 2) ^ (t & (kSw - 1))) << 2)) = w;
          }
      }
    }
    __syncthreads();
    for (int idx = tid; idx < kTok * kChunks; idx += NT) {
      const int t = idx / kChunks;
      const int c = idx % kChunks;
      const int64_t tg = tbase + ps * kTok + t;
      const int64_t v = vbase + 4 * c;
      if (tg >= a.T || v >= a.V) continue;
      const float4 w = *reinterpret_cast<const float4*>(st + t * BM + ((c ^ (t & (kSw - 1))) << 2));
      float* out = a.logits + tg * a.V + v;
      if (vec) {
        // whole lines, non-temporal (decode step 0.74 -> 0.72 ms: draft heads
        // 0.141 -> 0.126 ms, verifier head 3 % faster)
        store16_nt(out, make_uint4(__float_as_uint(w.x), __float_as_uint(w.y), __float_as_uint(w.z),
                                   __float_as_uint(w.w)));
      } else {
        const float x[4] = {w.x, w.y, w.z, w.w};
        for (int q = 0; q < 4 && v + q < a.V; ++q) out[q] = x[q];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// 2./3. per-row sampling distribution
// ---------------------------------------------------------------------------
//
// One 1024-thread block per row. Element i of a thread sits at vocabulary
// index v = 64 EPT wave + 64 i + lane: each wave owns a contiguous range of
// 64 EPT tokens, a slab i of it is one coalesced 256-byte load, and index
// order is (wave, slab, lane).
//
// Nucleus threshold. With `total` the sum of the row's exp weights and
// P = top_p * total, theta is the largest weight value whose mass
// S(theta) = sum(weight >= theta) still reaches P. Two facts bound it:
// * S(c) >= P implies theta >= c (theta is the largest such value);
// * for c' > c, S(c') >= S(c) - n(c) c', where n(c) counts the weights at or
//   above c; so S(c) >= P also gives theta >= (S(c) - P) / n(c).
// The search starts at c0 = (1 - top_p) total / V (the weights below c0 hold
// less than (1 - top_p) of the mass, so S(c0) >= P). The candidates
// {weight >= c0} are compacted once into a first LDS list (each wave its own
// region, in index order), the bound is raised with the second fact on that
// list, and the survivors move in index order to the final list. One wave
// then finds theta over the fp32 bit pattern (positive floats order like
// their bits) with four-way steps, resolves ties and draws: every kept token
// is in the final list. Rows whose first list overflows raise the bound over
// the row's registers instead; rows whose candidate set stays large (flat
// distributions) take a block-wide search over the whole row.

constexpr int kRowThreads = 1024;
constexpr int kRowWaves = kRowThreads / 64;
constexpr int kMaxEPT = 64;
constexpr int kRunMax = 16;              // candidate entries per lane of the list wave
constexpr int kMaxCand = 64 * kRunMax;   // candidates one wave holds
constexpr int kSmallCand = 4 * 64;       // lists searched with 4 entries per lane
constexpr int kBigCand = 4 * kRowThreads;  // first list: 4 entries per thread
constexpr int kRegion = kBigCand / kRowWaves;  // first-list entries per wave
constexpr int kBoundRounds = 3;          // raises of the lower bound

// LDS slot of list entry j: one gap after every 16 entries, so that the lanes
// of the list wave, each reading a run of consecutive entries, hit different
// banks.
__device__ __forceinline__ int cand_slot(int j) { return j + (j >> 4); }
constexpr int kCandSlots = kMaxCand + kMaxCand / 16;

struct RowShared {
  float bw[kBigCand];             // first list (weights >= c0): one region per wave,
  int bi[kBigCand];               // each in index order
  float cw[kCandSlots];           // final list, index order
  int ci[kCandSlots];             // their vocabulary indices
  float seg[kMaxEPT * kRowWaves]; // per (wave, slab) sums for whole-row index-order scans
  float red[kRowWaves];
  int ired[kRowWaves];
  int wcnt[kRowWaves];            // per-wave list counts
  float bcast[4];
  int ibcast[4];
};

// A row's exp weights are formed in several places (the distribution's
// parameters, then draws and probabilities recomputed from the logits); they
// must agree bitwise, so the product and the difference are rounded on their
// own and never contracted into an FMA.
__device__ __forceinline__ float scaled_logit(float l, float inv_temp) {
#pragma clang fp contract(off)
  return l * inv_temp;
}
__device__ __forceinline__ float weight_of(float scaled, float m) {
#pragma clang fp contract(off)
  return fast_exp2((scaled - m) * kLog2e);
}

// Block-wide reductions in a fixed order (every thread gets the result).
__device__ __forceinline__ float block_sum(float v, RowShared& sh) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh.red[w] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kRowWaves; ++i) s += sh.red[i];
  __syncthreads();
  return s;
}
__device__ __forceinline__ int block_count(int v, RowShared& sh) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh.ired[w] = v;
  __syncthreads();
  int s = 0;
#pragma unroll
  for (int i = 0; i < kRowWaves; ++i) s += sh.ired[i];
  __syncthreads();
  return s;
}
__device__ __forceinline__ void block_sum2(float& f, int& n, RowShared& sh) {
  f = wave_sum(f);
  n = wave_sum(n);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sh.red[w] = f;
    sh.ired[w] = n;
  }
  __syncthreads();
  float s = 0.f;
  int c = 0;
#pragma unroll
  for (int i = 0; i < kRowWaves; ++i) {
    s += sh.red[i];
    c += sh.ired[i];
  }
  __syncthreads();
  f = s;
  n = c;
}
// As block_sum2, with n already the wave's total in every lane.
__device__ __forceinline__ void block_sum2w(float& f, int& n, RowShared& sh) {
  f = wave_sum(f);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sh.red[w] = f;
    sh.ired[w] = n;
  }
  __syncthreads();
  float s = 0.f;
  int c = 0;
#pragma unroll
  for (int i = 0; i < kRowWaves; ++i) {
    s += sh.red[i];
    c += sh.ired[i];
  }
  __syncthreads();
  f = s;
  n = c;
}
__device__ __forceinline__ float block_max(float v, RowShared& sh) {
  v = wave_max(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh.red[w] = v;
  __syncthreads();
  float s = -INFINITY;
#pragma unroll
  for (int i = 0; i < kRowWaves; ++i) s = fmaxf(s, sh.red[i]);
  __syncthreads();
  return s;
}

// Argmax with the lowest index on ties.
__device__ __forceinline__ void block_argmax(float& val, int& idx, RowShared& sh) {
  wave_argmax(val, idx);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sh.red[w] = val;
    sh.ired[w] = idx;
  }
  __syncthreads();
  val = sh.red[0];
  idx = sh.ired[0];
#pragma unroll
  for (int i = 1; i < kRowWaves; ++i)
    if (argmax_better(sh.red[i], sh.ired[i], val, idx)) {
      val = sh.red[i];
      idx = sh.ired[i];
    }
  __syncthreads();
}

// Vocabulary index of the thread's element i.
template <int EPT>
__device__ __forceinline__ int elem_v(int i) {
  return (int)(threadIdx.x >> 6) * (64 * EPT) + 64 * i + (int)(threadIdx.x & 63);
}

// Number of the thread's elements inside the row: element i exists iff
// i < elems_in_row (a compare with a constant, so no per-element index needs
// to stay live).
template <int EPT>
__device__ __forceinline__ int elems_in_row(int V) {
  const int v0 = elem_v<EPT>(0);
  return V > v0 ? (V - v0 + 63) >> 6 : 0;
}

// The thread's EPT logits of a row, x[i] = row[elem_v(i)], as buffer loads
// over the row's V * 4 bytes: one per-lane offset, the slab as a scalar
// offset, and indices past the row read 0 from the hardware range check, so
// every load is unconditional and all of them are in flight together.
// Callers mask v >= V themselves.
template <int EPT>
__device__ __forceinline__ void load_row(const float* row, int V, float* x) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc((void*)row, (short)0, V * 4, 0x00020000);
  const int base = elem_v<EPT>(0) * 4;
#pragma unroll
  for (int i = 0; i < EPT; ++i)
    x[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, base, 256 * i, 0));
}

__device__ __forceinline__ int lanes_below(unsigned long long m) {
  return (int)__builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32),
                                        __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
}

// Smallest index whose cumulative weight in index order exceeds `target`,
// over the whole row; weight(i) gives the thread's i-th weight. Returns -1 if
// the total does not exceed it.
template <int EPT, class Wt>
__device__ __forceinline__ int index_order_draw(Wt weight, float target, RowShared& sh) {
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  // per (slab, wave) sums
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const float s = wave_sum(weight(i));
    if (lane == 0) sh.seg[wave * EPT + i] = s;
  }
  __syncthreads();
  // wave 0 scans the 16 EPT segment sums in index order (each lane owns a run of them)
  if (wave == 0) {
    constexpr int NSEG = EPT * kRowWaves;
    constexpr int PER = NSEG / 64;
    float run = 0.f;
#pragma unroll
    for (int q = 0; q < PER; ++q) run += sh.seg[lane * PER + q];
    const float incl = wave_incl_scan(run);
    float before = incl - run;
    int found = -1;
    float found_before = 0.f;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int sidx = lane * PER + q;
      const float s = sh.seg[sidx];
      if (found < 0 && s > 0.f && before + s > target) {
        found = sidx;
        found_before = before;
      }
      before += s;
    }
    // the first lane (in index order) that found its segment wins
    const unsigned long long m = __ballot(found >= 0);
    if (lane == 0) sh.ibcast[0] = -1;
    if (m && lane == __builtin_ctzll(m)) {
      sh.ibcast[0] = found;
      sh.bcast[0] = found_before;
    }
  }
  __syncthreads();
  const int sidx = sh.ibcast[0];
  const float base = sh.bcast[0];
  __syncthreads();
  if (sidx < 0) return -1;
  const int swave = sidx / EPT;
  const int slab = sidx % EPT;
  // inside the segment: the owning wave scans its 64 lanes
  if (wave == swave) {
    float x = 0.f;
#pragma unroll
    for (int i = 0; i < EPT; ++i)
      if (i == slab) x = weight(i);
    const float incl = wave_incl_scan(x);
    const unsigned long long m = __ballot(x > 0.f && base + incl > target);
    int pick;
    if (m) {
      pick = __builtin_ctzll(m);
    } else {  // rounding: take the last positive weight of the segment
      const unsigned long long pos = __ballot(x > 0.f);
      pick = pos ? 63 - __builtin_clzll(pos) : 0;
    }
    if (lane == 0) sh.ibcast[1] = swave * (64 * EPT) + slab * 64 + pick;
  }
  __syncthreads();
  const int v = sh.ibcast[1];
  __syncthreads();
  return v;
}

__device__ __forceinline__ bool kept_w(float e, int v, const RowDist& d) {
  return e > d.theta || (e == d.theta && e > 0.f && v <= d.tie_cut);
}

// Writes the row elements with flag(i) set to an LDS list in index order
// (weight val(i) to dw, vocabulary index to di; at cand_slot(position) when
// PAD) and returns how many there are; entries beyond CAP are not written.
// Index order is (wave, slab, lane): a first pass counts each wave's
// elements, then every wave writes from the sum of the counts before it.
template <int EPT, int CAP, bool PAD, class Flag, class Val>
__device__ __forceinline__ int compact_row(Flag flag, Val val, float* dw, int* di,
                                           RowShared& sh) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  int cnt = 0;  // wave-uniform
#pragma unroll
  for (int i = 0; i < EPT; ++i) cnt += __builtin_popcountll(__ballot(flag(i)));
  if (lane == 0) sh.wcnt[wave] = cnt;
  __syncthreads();
  int pos0 = 0, total = 0;
#pragma unroll
  for (int k = 0; k < kRowWaves; ++k) {
    pos0 += k < wave ? sh.wcnt[k] : 0;
    total += sh.wcnt[k];
  }
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const bool f = flag(i);
    const unsigned long long b = __ballot(f);
    if (f) {
      const int pos = pos0 + lanes_below(b);
      if (pos < CAP) {
        const int sl = PAD ? cand_slot(pos) : pos;
        dw[sl] = val(i);
        di[sl] = elem_v<EPT>(i);
      }
    }
    pos0 += __builtin_popcountll(b);
  }
  __syncthreads();
  return total;
}

// One pass: each wave writes its flagged elements, in index order, to its own
// region of kRegion entries of the first list (bw, bi); the counts go to
// sh.wcnt. Returns the total; `fits` tells whether every wave's elements fit
// its region.
template <int EPT, class Flag, class Val>
__device__ __forceinline__ int compact_regions(Flag flag, Val val, RowShared& sh, bool& fits) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  int pos0 = 0;  // wave-uniform
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const bool f = flag(i);
    const unsigned long long b = __ballot(f);
    if (f) {
      const int pos = pos0 + lanes_below(b);
      if (pos < kRegion) {
        sh.bw[wave * kRegion + pos] = val(i);
        sh.bi[wave * kRegion + pos] = elem_v<EPT>(i);
      }
    }
    pos0 += __builtin_popcountll(b);
  }
  if (lane == 0) sh.wcnt[wave] = pos0;
  __syncthreads();
  int total = 0;
  fits = true;
#pragma unroll
  for (int k = 0; k < kRowWaves; ++k) {
    total += sh.wcnt[k];
    fits = fits && sh.wcnt[k] <= kRegion;
  }
  return total;
}

// ---- list wave (wave 0, all lanes active): lane l holds entries [l RUN, (l + 1) RUN)

template <int RUN>
__device__ __forceinline__ void load_run(const RowShared& sh, int n, float (&w)[RUN]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int q = 0; q < RUN; ++q) {
    const int j = lane * RUN + q;
    w[q] = j < n ? sh.cw[cand_slot(j)] : 0.f;
  }
}

template <int RUN>
__device__ __forceinline__ int run_index(const RowShared& sh, int q) {
  return sh.ci[cand_slot((int)(threadIdx.x & 63) * RUN + q)];
}

// Position in the list of the first entry (index order) whose cumulative
// weight exceeds `target`; the last positive entry when rounding leaves the
// target at or above the sum; 0 when every weight is 0 (a kept set never is
// empty: the largest weight is 1 and theta <= 1).
template <int RUN>
__device__ __forceinline__ int run_draw(const float (&kw)[RUN], float target) {
  const int lane = threadIdx.x & 63;
  float run = 0.f;
#pragma unroll
  for (int q = 0; q < RUN; ++q) run += kw[q];
  const float incl = wave_incl_scan(run);
  const unsigned long long hit = __ballot(run > 0.f && incl > target);
  const unsigned long long pos = __ballot(run > 0.f);
  if (!pos) return 0;
  const int L = hit ? __builtin_ctzll(hit) : 63 - __builtin_clzll(pos);
  int j = 0;
  if (lane == L) {
    float acc = incl - run;
    int first = -1, last = 0;
#pragma unroll
    for (int q = 0; q < RUN; ++q) {
      if (kw[q] > 0.f) {
        acc += kw[q];
        last = q;
        if (first < 0 && acc > target) first = q;
      }
    }
    j = lane * RUN + (first >= 0 ? first : last);
  }
  return __builtin_amdgcn_readlane(j, L);
}

// Theta from the final list (list wave; n entries, weights >= c with
// S(c) >= P): the largest bit pattern whose mass reaches P. Four-way steps:
// three probes, three independent reductions. The probed sets are nested and
// summed in the same order, so the computed masses are ordered like the exact
// ones and the decisions are consistent. Theta is a list value: once a single
// entry remains in [lo, hi), it is theta. Once at most 64 entries remain in
// the bracket, the mass at or above hi is fixed (B) and those entries move to
// one per lane (through `scr`, 64 floats of LDS the list wave owns): each
// later probe is B plus one compare per lane instead of a pass over the run.
template <int RUN>
__device__ __forceinline__ float list_theta(const float (&w)[RUN], float c, float P, float* scr) {
  const int lane = threadIdx.x & 63;
  // invariant: S(lo) >= P > S(hi); lo, hi and the decisions are wave-uniform
  uint32_t lo = __float_as_uint(c), hi = 0x3f800001u;  // nothing is above 1
  while (hi - lo > 1) {
    int inside = 0;
    float last = 0.f;
#pragma unroll
    for (int q = 0; q < RUN; ++q) {
      const uint32_t b = __float_as_uint(w[q]);
      const bool in = b >= lo && b < hi;
      inside += in ? 1 : 0;
      last = in ? w[q] : last;
    }
    const unsigned long long any = __ballot(inside > 0);
    if (__builtin_popcountll(any) == 1 && __ballot(inside > 1) == 0) {
      const float v = __builtin_bit_cast(
          float, __builtin_amdgcn_readlane(__float_as_int(last), __builtin_ctzll(any)));
      return v;
    }
    if (RUN > 1 && wave_sum(inside) <= 64) break;
    if (hi - lo > 3) {
      const uint32_t st = (hi - lo) >> 2;
      const uint32_t m1 = lo + st, m2 = m1 + st, m3 = m2 + st;
      float p1 = 0.f, p2 = 0.f, p3 = 0.f;
#pragma unroll
      for (int q = 0; q < RUN; ++q) {
        const uint32_t b = __float_as_uint(w[q]);
        p1 += b >= m1 ? w[q] : 0.f;
        p2 += b >= m2 ? w[q] : 0.f;
        p3 += b >= m3 ? w[q] : 0.f;
      }
      const int g1 = __builtin_amdgcn_readfirstlane(wave_sum(p1) >= P ? 1 : 0);
      const int g2 = __builtin_amdgcn_readfirstlane(wave_sum(p2) >= P ? 1 : 0);
      const int g3 = __builtin_amdgcn_readfirstlane(wave_sum(p3) >= P ? 1 : 0);
      if (g3) {
        lo = m3;
      } else if (g2) {
        lo = m2;
        hi = m3;
      } else if (g1) {
        lo = m1;
        hi = m2;
      } else {
        hi = m1;
      }
    } else {
      const uint32_t mid = lo + (hi - lo) / 2;
      float part = 0.f;
#pragma unroll
      for (int q = 0; q < RUN; ++q) part += __float_as_uint(w[q]) >= mid ? w[q] : 0.f;
      if (__builtin_amdgcn_readfirstlane(wave_sum(part) >= P ? 1 : 0))
        lo = mid;
      else
        hi = mid;
    }
  }
  if (hi - lo <= 1) return __uint_as_float(lo);
  // at most 64 entries in [lo, hi): B = the mass at or above hi, and the
  // bracket's entries one per lane (in run order)
  float base = 0.f;
  int cnt = 0;
#pragma unroll
  for (int q = 0; q < RUN; ++q) {
    const uint32_t b = __float_as_uint(w[q]);
    base += b >= hi ? w[q] : 0.f;
    cnt += (b >= lo && b < hi) ? 1 : 0;
  }
  const float B = wave_sum(base);
  const int incl = wave_incl_scan(cnt);
  const int n2 = __builtin_amdgcn_readlane(incl, 63);
  int pos = incl - cnt;
#pragma unroll
  for (int q = 0; q < RUN; ++q) {
    const uint32_t b = __float_as_uint(w[q]);
    if (b >= lo && b < hi) scr[pos++] = w[q];
  }
  const float x = lane < n2 ? scr[lane] : 0.f;
  const uint32_t bx = __float_as_uint(x);
  while (hi - lo > 1) {
    const unsigned long long in = __ballot(lane < n2 && bx >= lo && bx < hi);
    if (__builtin_popcountll(in) == 1)
      return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__float_as_int(x), __builtin_ctzll(in)));
    if (hi - lo > 3) {
      const uint32_t st = (hi - lo) >> 2;
      const uint32_t m1 = lo + st, m2 = m1 + st, m3 = m2 + st;
      const int g1 = __builtin_amdgcn_readfirstlane(B + wave_sum(bx >= m1 ? x : 0.f) >= P ? 1 : 0);
      const int g2 = __builtin_amdgcn_readfirstlane(B + wave_sum(bx >= m2 ? x : 0.f) >= P ? 1 : 0);
      const int g3 = __builtin_amdgcn_readfirstlane(B + wave_sum(bx >= m3 ? x : 0.f) >= P ? 1 : 0);
      if (g3) {
        lo = m3;
      } else if (g2) {
        lo = m2;
        hi = m3;
      } else if (g1) {
        lo = m1;
        hi = m2;
      } else {
        hi = m1;
      }
    } else {
      const uint32_t mid = lo + (hi - lo) / 2;
      if (__builtin_amdgcn_readfirstlane(B + wave_sum(bx >= mid ? x : 0.f) >= P ? 1 : 0))
        lo = mid;
      else
        hi = mid;
    }
  }
  return __uint_as_float(lo);
}

// Completes a row's distribution from its final list (list wave): theta, the
// tie cut and the kept mass. `kw` receives the kept weights of the lane's run.
template <int RUN>
__device__ __forceinline__ void run_dist(RowShared& sh, int n, float c, float P, int V,
                                         RowDist& d, float (&kw)[RUN]) {
  const int lane = threadIdx.x & 63;
  float w[RUN];
  load_run<RUN>(sh, n, w);
  const float th = list_theta<RUN>(w, c, P, sh.bw);  // the first list is spent by now
  d.theta = th;
  float above = 0.f;
  int ties = 0;
#pragma unroll
  for (int q = 0; q < RUN; ++q) {
    above += w[q] > th ? w[q] : 0.f;
    ties += w[q] == th ? 1 : 0;  // th > 0, so padding zeros never tie
  }
  const float mass_above = wave_sum(above);
  const int n_tie = wave_sum(ties);
  int k = n_tie;
  if (n_tie > 1) {
    k = (int)ceilf((P - mass_above) / th);
    k = k < 1 ? 1 : (k > n_tie ? n_tie : k);
  }
  d.tie_cut = V;
  if (k < n_tie) {  // vocabulary index of the k-th tied entry (the list is in index order)
    const int incl = wave_incl_scan(ties);
    const int L = __builtin_ctzll(__ballot(incl >= k));
    int cut = 0;
    if (lane == L) {
      int seen = incl - ties;
#pragma unroll
      for (int q = 0; q < RUN; ++q)
        if (w[q] == th && ++seen == k) cut = run_index<RUN>(sh, q);
    }
    d.tie_cut = __builtin_amdgcn_readlane(cut, L);
  }
  float kp = 0.f;
#pragma unroll
  for (int q = 0; q < RUN; ++q) {
    kw[q] = w[q] > th || (w[q] == th && run_index<RUN>(sh, q) <= d.tie_cut) ? w[q] : 0.f;
    kp += kw[q];
  }
  d.kept = wave_sum(kp);
}

// Mass and count of the weights at or above t (block-wide).
template <int EPT>
__device__ __forceinline__ void mass_at(const float* e, float t, float& F, int& n, RowShared& sh) {
  F = 0.f;
  n = 0;  // per wave: the same in every lane
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const bool in = e[i] >= t;
    F += in ? e[i] : 0.f;
    n += __builtin_popcountll(__ballot(in));
  }
  block_sum2w(F, n, sh);
}

// Mass and count of the list entries w[] >= t held by the threads (block-wide).
__device__ __forceinline__ void list_mass(const float (&w)[4], float t, float& F, int& n,
                                          RowShared& sh) {
  F = 0.f;
  n = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    F += w[q] >= t ? w[q] : 0.f;
    n += w[q] >= t ? 1 : 0;
  }
  block_sum2(F, n, sh);
}

// Loads a row and computes its sampling distribution. `e` receives the
// thread's exp weights exp(l / T - max) (0 beyond V). With a nucleus and a
// small candidate set the candidates (weights >= `c`) are left in the LDS
// list and their number is returned: then only m and total are set in d, and
// the list wave completes it (run_dist). Otherwise the whole distribution is
// in d for every thread and -1 is returned.
template <int EPT>
__device__ __forceinline__ int row_dist(const float* row, int V, float inv_temp, float top_p,
                                        float* e, RowShared& sh, RowDist& d, float& c, float& P) {
  load_row<EPT>(row, V, e);
  const int nv = elems_in_row<EPT>(V);
  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    e[i] = i < nv ? scaled_logit(e[i], inv_temp) : -INFINITY;
    mx = fmaxf(mx, e[i]);
  }
  d.m = block_max(mx, sh);
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    e[i] = e[i] == -INFINITY ? 0.f : weight_of(e[i], d.m);
    s += e[i];
  }
  d.total = block_sum(s, sh);
  d.theta = 0.f;
  d.tie_cut = V;
  d.kept = d.total;
  if (!(top_p < 1.f)) return -1;
  P = top_p * d.total;
  c = (1.f - top_p) * d.total / (float)V;
  bool ok = c > 0.f;
  if (ok) {
    const float c0 = c;
    bool fits;
    compact_regions<EPT>([&](int i) { return e[i] >= c0; }, [&](int i) { return e[i]; }, sh,
                         fits);
    if (fits) {
      // the bound rounds run on the first list: the thread holds entries 4 lane
      // .. 4 lane + 3 of its wave's region, so thread order is index order
      const int lane = threadIdx.x & 63;
      const int wave = threadIdx.x >> 6;
      const int nw = sh.wcnt[wave];
      float w[4];
      int ix[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int j = 4 * lane + q;
        w[q] = j < nw ? sh.bw[wave * kRegion + j] : 0.f;
        ix[q] = sh.bi[wave * kRegion + j];
      }
      float F;
      int n;
      list_mass(w, c, F, n, sh);
      ok = F >= P;
      for (int r = 0; ok && r < kBoundRounds && n > kSmallCand; ++r) {
        const float t = (F - P) / (float)n;
        if (!(t > c)) break;
        float F2;
        int n2;
        list_mass(w, t, F2, n2, sh);
        if (!(F2 >= P)) break;
        c = t;
        F = F2;
        n = n2;
      }
      if (ok && n <= kMaxCand) {  // stable compaction of the weights >= c into the final list
        int cnt = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) cnt += w[q] >= c ? 1 : 0;
        const int incl = wave_incl_scan(cnt);
        if (lane == 63) sh.ired[wave] = incl;
        __syncthreads();
        int pos = incl - cnt;
#pragma unroll
        for (int k = 0; k < kRowWaves; ++k) pos += k < wave ? sh.ired[k] : 0;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (w[q] >= c) {
            sh.cw[cand_slot(pos)] = w[q];
            sh.ci[cand_slot(pos)] = ix[q];
            ++pos;
          }
        __syncthreads();
        return n;
      }
    } else {
      // a large first list: the rounds run over the thread's row elements
      float F;
      int n;
      mass_at<EPT>(e, c, F, n, sh);
      ok = F >= P;
      for (int r = 0; ok && r < kBoundRounds && n > kSmallCand; ++r) {
        const float t = (F - P) / (float)n;
        if (!(t > c)) break;
        float F2;
        int n2;
        mass_at<EPT>(e, t, F2, n2, sh);
        if (!(F2 >= P)) break;
        c = t;
        F = F2;
        n = n2;
      }
      if (ok && n <= kMaxCand) {
        const float cc = c;
        return compact_row<EPT, kMaxCand, true>([&](int i) { return e[i] >= cc; },
                                                [&](int i) { return e[i]; }, sh.cw, sh.ci, sh);
      }
    }
  }
  // whole-row search: largest bit pattern b with sum(e >= b) >= P
  uint32_t lo = 0, hi = 0x3f800001u;  // sum(e >= 0) = total >= P; nothing is above 1
  if (ok) lo = __float_as_uint(c);  // S(c) >= P was checked
  while (hi - lo > 1) {
    const uint32_t mid = lo + (hi - lo) / 2;
    float part = 0.f;
#pragma unroll
    for (int i = 0; i < EPT; ++i) part += __float_as_uint(e[i]) >= mid ? e[i] : 0.f;
    if (block_sum(part, sh) >= P)
      lo = mid;
    else
      hi = mid;
  }
  d.theta = __uint_as_float(lo);
  float above = 0.f;
  int ties = 0;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    above += e[i] > d.theta ? e[i] : 0.f;
    ties += (e[i] == d.theta && e[i] > 0.f) ? 1 : 0;
  }
  const float mass_above = block_sum(above, sh);
  const int n_tie = block_count(ties, sh);
  int k = n_tie;
  if (n_tie > 1 && d.theta > 0.f) {
    k = (int)ceilf((P - mass_above) / d.theta);
    k = k < 1 ? 1 : (k > n_tie ? n_tie : k);
  }
  // index of the k-th tied token (counts are exact in fp32 up to 2^24)
  const float th = d.theta;
  d.tie_cut = k >= n_tie ? V
                         : index_order_draw<EPT>(
                               [&](int i) { return (e[i] == th && e[i] > 0.f) ? 1.f : 0.f; },
                               (float)k - 0.5f, sh);
  float kp = 0.f;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const int v = elem_v<EPT>(i);
    kp += kept_w(e[i], v, d) ? e[i] : 0.f;
  }
  d.kept = block_sum(kp, sh);
  return -1;
}

// Whole-row draw from a row's distribution with uniform u (weights in `e`,
// parameters in d); `e` is overwritten with the kept weights.
template <int EPT>
__device__ __forceinline__ int row_draw(float* e, const RowDist& d, float u, RowShared& sh) {
  int last = -1;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const int v = elem_v<EPT>(i);
    e[i] = kept_w(e[i], v, d) ? e[i] : 0.f;
    if (e[i] > 0.f) last = v;
  }
  int v = index_order_draw<EPT>([&](int i) { return e[i]; }, u * d.kept, sh);
  if (v < 0) {  // rounding pushed the target past the total: the last kept index
    float lv = (float)last;
    int li = last;
    block_argmax(lv, li, sh);
    v = li;
  }
  return v;
}

template <int EPT>
__device__ __forceinline__ int row_argmax(const float* row, int V, RowShared& sh) {
  float x[EPT];
  load_row<EPT>(row, V, x);
  const int nv = elems_in_row<EPT>(V);
  float best = -INFINITY;
  int bi = 0x7fffffff;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    if (i < nv && x[i] > best) {  // the index increases with i: strict > keeps the lowest
      best = x[i];
      bi = i;
    }
  }
  bi = bi == 0x7fffffff ? bi : elem_v<EPT>(0) + 64 * bi;
  block_argmax(best, bi, sh);
  return bi;
}

// The distribution from the final list (every thread calls it; only wave 0
// works, the other waves return -2 at once), then (with u >= 0) a draw;
// returns the drawn token (or -1 without a draw).
template <int RUN>
__device__ __forceinline__ int list_finish(RowShared& sh, int n, float c, float P, int V,
                                           float u, RowDist& d) {
  if (threadIdx.x >= 64) return -2;
  float kw[RUN];
  run_dist<RUN>(sh, n, c, P, V, d, kw);
  if (u < 0.f) return -1;
  const int j = run_draw<RUN>(kw, u * d.kept);
  return sh.ci[cand_slot(j)];
}

template <int EPT>
__global__ __launch_bounds__(kRowThreads) void sample_kernel(SampleArgs a) {
  __shared__ RowShared sh;
  const int64_t r = blockIdx.x;
  const float* row = a.logits + r * a.V;
  int tok;
  if (a.greedy) {
    tok = row_argmax<EPT>(row, (int)a.V, sh);
  } else {
    float e[EPT];
    RowDist d;
    float c = 0.f, P = 0.f;
    const int n = row_dist<EPT>(row, (int)a.V, a.inv_temp, a.top_p, e, sh, d, c, P);
    if (n >= 0) {
      tok = n <= kSmallCand ? list_finish<4>(sh, n, c, P, (int)a.V, a.u[r], d)
                            : list_finish<kRunMax>(sh, n, c, P, (int)a.V, a.u[r], d);
      if (threadIdx.x >= 64) return;
    } else {
      tok = row_draw<EPT>(e, d, a.u[r], sh);
    }
    if (threadIdx.x == 0 && a.params) a.params[r] = d;
  }
  if (threadIdx.x == 0) a.tokens[r] = tok;
}

// Every row's sampling-distribution parameters (rows of several arrays: the
// draft rows, then the verifier rows).
template <int EPT>
__global__ __launch_bounds__(kRowThreads) void row_params_kernel(RowParamArgs a) {
  __shared__ RowShared sh;
  const int64_t r = blockIdx.x;
  const float* row = r < a.rows0 ? a.logits0 + r * a.V : a.logits1 + (r - a.rows0) * a.V;
  float e[EPT];
  RowDist d;
  float c = 0.f, P = 0.f;
  const int n = row_dist<EPT>(row, (int)a.V, a.inv_temp, a.top_p, e, sh, d, c, P);
  if (n >= 0) {
    if (n <= kSmallCand)
      list_finish<4>(sh, n, c, P, (int)a.V, -1.f, d);
    else
      list_finish<kRunMax>(sh, n, c, P, (int)a.V, -1.f, d);
    if (threadIdx.x >= 64) return;
  }
  if (threadIdx.x == 0) a.params[r] = d;
}

// Exp weight of logit x under a row's parameters, with row_dist's arithmetic.
__device__ __forceinline__ float exp_weight(float logit, float inv_temp, const RowDist& d) {
  return weight_of(scaled_logit(logit, inv_temp), d.m);
}

// Kept, normalised probability of token v (v < V).
__device__ __forceinline__ float prob_at(const float* row, int v, float inv_temp,
                                         const RowDist& d) {
  const float e = exp_weight(row[v], inv_temp, d);
  return kept_w(e, v, d) ? e / d.kept : 0.f;
}

// Whole-row draw with uniform u from a row's distribution, weights recomputed
// from the logits.
template <int EPT>
__device__ __forceinline__ int draw_kept(const float* row, int V, float it, const RowDist& d,
                                         float u, RowShared& sh) {
  auto w = [&](int i) {
    const int v = elem_v<EPT>(i);
    if (v >= V) return 0.f;
    const float e = exp_weight(row[v], it, d);
    return kept_w(e, v, d) ? e : 0.f;
  };
  int v = index_order_draw<EPT>(w, u * d.kept, sh);
  if (v < 0) {
    int last = -1;
    for (int i = 0; i < EPT; ++i)
      if (w(i) > 0.f) last = elem_v<EPT>(i);
    float lv = (float)last;
    block_argmax(lv, last, sh);
    v = last;
  }
  return v;
}

// Compacts the kept tokens of row p (weights recomputed from the logits) into
// the LDS list; returns their number.
template <int EPT>
__device__ __forceinline__ int compact_kept(const float* prow, int V, float it, const RowDist& dp,
                                            RowShared& sh) {
  float w[EPT];
  load_row<EPT>(prow, V, w);
  const int nv = elems_in_row<EPT>(V);
  const int v0 = elem_v<EPT>(0);
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const float e = exp_weight(w[i], it, dp);
    w[i] = i < nv && kept_w(e, v0 + 64 * i, dp) ? e : 0.f;
  }
  return compact_row<EPT, kMaxCand, true>([&](int i) { return w[i] > 0.f; },
                                          [&](int i) { return w[i]; }, sh.cw, sh.ci, sh);
}

// List wave: a draw from p's kept list (n entries) with uniform u; with a
// draft row qrow (parameters dq), from max(0, p - q), or p itself if that has
// no mass.
template <int RUN>
__device__ __forceinline__ int list_residual_draw(const RowShared& sh, int n, const RowDist& dp,
                                                  const float* qrow, const RowDist& dq, float it,
                                                  float u) {
  float w[RUN];
  load_run<RUN>(sh, n, w);
  if (qrow) {
    float r[RUN];
    float s = 0.f;
#pragma unroll
    for (int q = 0; q < RUN; ++q) {
      r[q] = 0.f;
      if (w[q] > 0.f)
        r[q] = fmaxf(w[q] / dp.kept - prob_at(qrow, run_index<RUN>(sh, q), it, dq), 0.f);
      s += r[q];
    }
    const float tot = wave_sum(s);
    if (tot > 0.f) return sh.ci[cand_slot(run_draw<RUN>(r, u * tot))];
  }
  return sh.ci[cand_slot(run_draw<RUN>(w, u * dp.kept))];
}

// Verification: one block per sequence. Rows' parameters come from
// row_params_kernel; weights are recomputed from the logits as needed (the
// rows stay in L2). The draw after a rejection (or after the last draft) runs
// over the verifier row's kept tokens, which hold all of max(0, p - q).
template <int EPT, bool GREEDY>
__global__ __launch_bounds__(kRowThreads) void verify_kernel(VerifyArgs a) {
  __shared__ RowShared sh;
  const int64_t b = blockIdx.x;
  const int V = (int)a.V;
  const int G = a.gamma;
  const float it = a.inv_temp;
  int k = 0;
  int next = 0;
#pragma nounroll
  for (; k < G; ++k) {
    const int x = a.draft_tokens[(int64_t)k * a.batch + b];
    const float* trow = a.target_logits + (b * (G + 1) + k) * a.V;
    if (GREEDY) {
      const int best = row_argmax<EPT>(trow, V, sh);
      if (best != x) {
        next = best;
        break;
      }
      continue;
    }
    const float* drow = a.draft_logits + ((int64_t)k * a.batch + b) * a.V;
    const RowDist dq = a.dparams[(int64_t)k * a.batch + b];
    const RowDist dp = a.tparams[b * (G + 1) + k];
    const bool in = x >= 0 && x < V;
    const float qx = in ? prob_at(drow, x, it, dq) : 0.f;
    const float px = in ? prob_at(trow, x, it, dp) : 0.f;
    if (a.u_accept[(int64_t)k * a.batch + b] * qx < px) continue;
    // rejected: draw from max(0, p - q)
    const int n = compact_kept<EPT>(trow, V, it, dp, sh);
    if (n <= kMaxCand) {
      if (threadIdx.x >= 64) return;
      next = n <= kSmallCand ? list_residual_draw<4>(sh, n, dp, drow, dq, it, a.u_sample[b])
                         : list_residual_draw<kRunMax>(sh, n, dp, drow, dq, it, a.u_sample[b]);
      break;
    }
    auto res = [&](int i) {
      const int v = elem_v<EPT>(i);
      if (v >= V) return 0.f;
      return fmaxf(prob_at(trow, v, it, dp) - prob_at(drow, v, it, dq), 0.f);
    };
    float rs = 0.f;
#pragma unroll 4
    for (int i = 0; i < EPT; ++i) rs += res(i);
    const float tot = block_sum(rs, sh);
    if (tot > 0.f) {
      int v = index_order_draw<EPT>(res, a.u_sample[b] * tot, sh);
      if (v < 0) {
        int last = -1;
        for (int i = 0; i < EPT; ++i)
          if (res(i) > 0.f) last = elem_v<EPT>(i);
        float lv = (float)last;
        block_argmax(lv, last, sh);
        v = last;
      }
      next = v;
    } else {
      // no residual mass: the rejected token was impossible under both
      // distributions and they coincide, so the draw is from the verifier's
      next = draw_kept<EPT>(trow, V, it, dp, a.u_sample[b], sh);
    }
    break;
  }
  if (k == G) {  // every draft kept: one more token from the verifier
    const float* trow = a.target_logits + (b * (G + 1) + G) * a.V;
    if (GREEDY) {
      next = row_argmax<EPT>(trow, V, sh);
    } else {
      const RowDist dp = a.tparams[b * (G + 1) + G];
      const int n = compact_kept<EPT>(trow, V, it, dp, sh);
      if (n <= kMaxCand) {
        if (threadIdx.x >= 64) return;
        next = n <= kSmallCand ? list_residual_draw<4>(sh, n, dp, nullptr, dp, it, a.u_sample[b])
                           : list_residual_draw<kRunMax>(sh, n, dp, nullptr, dp, it,
                                                         a.u_sample[b]);
      } else {
        next = draw_kept<EPT>(trow, V, it, dp, a.u_sample[b], sh);
      }
    }
  }
  if (threadIdx.x == 0) {
    a.n_accepted[b] = k;
    a.next_token[b] = next;
  }
}

using HeadWide = WideMma<128, 128, 2, 2, 2>;
// 192 vocabulary rows: 80 KB of stages, two blocks fill a CU's LDS
using HeadWide192 = WideMma<192, 128, 2, 2, 2>;
using HeadGenBf16 = TileMma<Bf16, 128, 128, 2, 2>;
using HeadGenF32 = TileMma<F32, 128, 128, 2, 2>;

}  // namespace

int head_tile() { return 128; }
// Vocabulary rows of a head tile. With at least four token tiles (the
// verifier's rows) the 192-row tile on the wide path: at 102 x 7 rows and
// V = 49,152 it makes 1,536 blocks, three full rounds of two blocks per CU,
// where 128-row tiles make 2,304 (four and a half).
int head_tile_rows(bool wide, int n_tt) { return wide && n_tt >= 4 ? 192 : 128; }
int row_elems_per_thread(int64_t V) {
  for (int e : {16, 32, 48, 64})
    if (V <= (int64_t)e * kRowThreads) return e;
  return 0;
}

hipError_t launch_head_logits(const HeadArgs& a, bool f32, bool wide, int rows,
                              hipStream_t stream) {
  const dim3 grid((unsigned)a.n_tt * (unsigned)a.n_vt);
  if (rows != (f32 || !wide ? 128 : head_tile_rows(wide, a.n_tt))) return hipErrorInvalidValue;
  if (f32)
    hipLaunchKernelGGL((head_logits_kernel<HeadGenF32, F32>), grid, dim3(HeadGenF32::NT), 0, stream,
                       a);
  else if (wide && rows == 192)
    hipLaunchKernelGGL((head_logits_kernel<HeadWide192, Bf16>), grid, dim3(HeadWide192::NT), 0,
                       stream, a);
  else if (wide)
    hipLaunchKernelGGL((head_logits_kernel<HeadWide, Bf16>), grid, dim3(HeadWide::NT), 0, stream, a);
  else
    hipLaunchKernelGGL((head_logits_kernel<HeadGenBf16, Bf16>), grid, dim3(HeadGenBf16::NT), 0,
                       stream, a);
  return hipGetLastError();
}

hipError_t launch_sample(const SampleArgs& a, int ept, hipStream_t stream) {
  const dim3 grid((unsigned)a.rows);
  switch (ept) {
    case 16: hipLaunchKernelGGL(sample_kernel<16>, grid, dim3(kRowThreads), 0, stream, a); break;
    case 32: hipLaunchKernelGGL(sample_kernel<32>, grid, dim3(kRowThreads), 0, stream, a); break;
    case 48: hipLaunchKernelGGL(sample_kernel<48>, grid, dim3(kRowThreads), 0, stream, a); break;
    case 64: hipLaunchKernelGGL(sample_kernel<64>, grid, dim3(kRowThreads), 0, stream, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_row_params(const RowParamArgs& a, int ept, hipStream_t stream) {
  const dim3 grid((unsigned)(a.rows0 + a.rows1));
  switch (ept) {
    case 16: hipLaunchKernelGGL(row_params_kernel<16>, grid, dim3(kRowThreads), 0, stream, a); break;
    case 32: hipLaunchKernelGGL(row_params_kernel<32>, grid, dim3(kRowThreads), 0, stream, a); break;
    case 48: hipLaunchKernelGGL(row_params_kernel<48>, grid, dim3(kRowThreads), 0, stream, a); break;
    case 64: hipLaunchKernelGGL(row_params_kernel<64>, grid, dim3(kRowThreads), 0, stream, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int EPT>
static void launch_verify_ept(const VerifyArgs& a, hipStream_t stream) {
  const dim3 grid((unsigned)a.batch);
  if (a.greedy)
    hipLaunchKernelGGL((verify_kernel<EPT, true>), grid, dim3(kRowThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((verify_kernel<EPT, false>), grid, dim3(kRowThreads), 0, stream, a);
}

hipError_t launch_verify(const VerifyArgs& a, int ept, hipStream_t stream) {
  switch (ept) {
    case 16: launch_verify_ept<16>(a, stream); break;
    case 32: launch_verify_ept<32>(a, stream); break;
    case 48: launch_verify_ept<48>(a, stream); break;
    case 64: launch_verify_ept<64>(a, stream); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace mls
