// The head step of nested speculative decoding (paper section 2, paragraph
// "Speculative Decoding"; the measured setting of section 3, "Speculative
// Decoding Throughput": greedy or nucleus top-p 0.9 sampling at temperature
// 0.4, a smaller sub-model drafting gamma tokens and a larger one verifying).
//
// 1. head_logits_kernel: logits[t][v] = sum_k o[t][k] W[v][k] in fp32, on the
//    MFMA tile core; the 128x128 fp32 tile is staged in LDS and leaves the
//    block as 16-byte stores of token-major rows. Decode batches are small, so
//    the [rows, V] logits are cheap next to the head itself.
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
  constexpr int kChunks = BM / 4;  // 16-byte chunks (4 floats) per token row of the tile
  static_assert(BN * BM * 4 <= Mma::kSmemBytes, "fp32 tile fits in the stage memory");
  static_assert(kChunks == 32, "swizzle assumes 32 chunks per row");
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

  // stage: token row t holds 32 chunks of 4 vocabulary entries, chunk c at c ^ (t & 31)
  float* st = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) {
    const int t = Mma::col_of(wn, fn, lane);
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const int v0 = Mma::row_of(wm, fm, rg * 4, lane);  // multiple of 4
        const float4 w = make_float4(mma.acc[fm][fn][rg * 4], mma.acc[fm][fn][rg * 4 + 1],
                                     mma.acc[fm][fn][rg * 4 + 2], mma.acc[fm][fn][rg * 4 + 3]);
        *reinterpret_cast<float4*>(st + t * BM + (((v0 >> 2) ^ (t & 31)) << 2)) = w;
      }
  }
  __syncthreads();
  const bool vec = (a.V & 3) == 0;
  for (int idx = tid; idx < BN * kChunks; idx += NT) {
    const int t = idx / kChunks;
    const int c = idx % kChunks;
    const int64_t tg = tbase + t;
    const int64_t v = vbase + 4 * c;
    if (tg >= a.T || v >= a.V) continue;
    const float4 w = *reinterpret_cast<const float4*>(st + t * BM + ((c ^ (t & 31)) << 2));
    float* out = a.logits + tg * a.V + v;
    if (vec) {
      *reinterpret_cast<float4*>(out) = w;
    } else {
      const float x[4] = {w.x, w.y, w.z, w.w};
      for (int q = 0; q < 4 && v + q < a.V; ++q) out[q] = x[q];
    }
  }
}

// ---------------------------------------------------------------------------
// 2./3. per-row sampling distribution
// ---------------------------------------------------------------------------

constexpr int kRowThreads = 1024;
constexpr int kRowWaves = kRowThreads / 64;

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

constexpr int kMaxCand = 2048;  // nucleus candidates searched by one wave

struct RowShared {
  float cand[kMaxCand];       // compacted candidate weights (thread order)
  int woff[kRowWaves];        // per-wave offsets of the compaction
  float red[kRowWaves];
  int ired[kRowWaves];
  float seg[kRowWaves * 64];  // per (slab, wave) partial sums for index-order scans
  float bcast[4];
  int ibcast[4];
};

__device__ __forceinline__ float wave_sum_f(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ int wave_sum_i(int v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max_f(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Block-wide reductions in a fixed order (every thread gets the result).
__device__ __forceinline__ float block_sum(float v, RowShared& sh) {
  v = wave_sum_f(v);
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
  v = wave_sum_i(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh.ired[w] = v;
  __syncthreads();
  int s = 0;
#pragma unroll
  for (int i = 0; i < kRowWaves; ++i) s += sh.ired[i];
  __syncthreads();
  return s;
}
__device__ __forceinline__ float block_max(float v, RowShared& sh) {
  v = wave_max_f(v);
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
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float ov = __shfl_xor(val, o, 64);
    const int oi = __shfl_xor(idx, o, 64);
    if (ov > val || (ov == val && oi < idx)) {
      val = ov;
      idx = oi;
    }
  }
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
    if (sh.red[i] > val || (sh.red[i] == val && sh.ired[i] < idx)) {
      val = sh.red[i];
      idx = sh.ired[i];
    }
  __syncthreads();
}

// The thread's element i sits at vocabulary index v = threadIdx.x + kRowThreads * i
// (slab i), so index order is (slab, wave, lane).

// Smallest index whose cumulative weight in index order exceeds `target`;
// weight(i) gives the thread's i-th weight. Returns -1 if the total does not
// exceed it.
template <int EPT, class Wt>
__device__ __forceinline__ int index_order_draw(Wt weight, float target, RowShared& sh) {
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  // per (slab, wave) sums
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const float s = wave_sum_f(weight(i));
    if (lane == 0) sh.seg[i * kRowWaves + wave] = s;
    __builtin_amdgcn_sched_barrier(0);  // one reduction chain at a time
  }
  __syncthreads();
  // wave 0 scans the EPT * 16 segment sums in order (each lane owns a run of them)
  if (wave == 0) {
    constexpr int NSEG = EPT * kRowWaves;
    constexpr int PER = (NSEG + 63) / 64;
    float run = 0.f;
    for (int q = 0; q < PER; ++q) {
      const int sidx = lane * PER + q;
      run += sidx < NSEG ? sh.seg[sidx] : 0.f;
    }
    // exclusive prefix of the lanes' runs
    float incl = run;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const float up = __shfl_up(incl, o, 64);
      if (lane >= o) incl += up;
    }
    float before = incl - run;
    int found = -1;
    float found_before = 0.f;
    for (int q = 0; q < PER; ++q) {
      const int sidx = lane * PER + q;
      const float s = sidx < NSEG ? sh.seg[sidx] : 0.f;
      if (found < 0 && s > 0.f && before + s > target) {
        found = sidx;
        found_before = before;
      }
      before += s;
    }
    // the first lane (in index order) that found its segment wins
    const unsigned long long m = __ballot(found >= 0);
    const int first = m ? __ffsll((long long)m) - 1 : -1;
    if (lane == 0) {
      sh.ibcast[0] = -1;
    }
    if (first >= 0 && lane == first) {
      sh.ibcast[0] = found;
      sh.bcast[0] = found_before;
    }
  }
  __syncthreads();
  const int sidx = sh.ibcast[0];
  const float base = sh.bcast[0];
  __syncthreads();
  if (sidx < 0) return -1;
  const int slab = sidx / kRowWaves;
  const int swave = sidx % kRowWaves;
  // inside the segment: the owning wave scans its 64 lanes
  if (wave == swave) {
    float x = 0.f;
#pragma unroll
    for (int i = 0; i < EPT; ++i)
      if (i == slab) x = weight(i);
    float incl = x;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const float up = __shfl_up(incl, o, 64);
      if (lane >= o) incl += up;
    }
    const unsigned long long m = __ballot(x > 0.f && base + incl > target);
    int pick = m ? __ffsll((long long)m) - 1 : -1;
    if (pick < 0) {  // rounding: take the last positive weight of the segment
      const unsigned long long pos = __ballot(x > 0.f);
      pick = pos ? 63 - __clzll((long long)pos) : 0;
    }
    if (lane == 0) sh.ibcast[1] = slab * kRowThreads + swave * 64 + pick;
  }
  __syncthreads();
  const int v = sh.ibcast[1];
  __syncthreads();
  return v;
}


__device__ __forceinline__ bool kept_w(float e, int v, const RowDist& d) {
  return e > d.theta || (e == d.theta && e > 0.f && v <= d.tie_cut);
}

// Loads a row and computes its sampling distribution; `e` receives the exp
// weights exp(l / T - max) of the thread's elements (0 beyond V).
template <int EPT>
__device__ __forceinline__ RowDist row_dist(const float* row, int V, float inv_temp, float top_p, float* e,
                            RowShared& sh) {
  RowDist d;
  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const int v = threadIdx.x + kRowThreads * i;
    e[i] = v < V ? scaled_logit(row[v], inv_temp) : -INFINITY;
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
  if (!(top_p < 1.f)) return d;
  const float P = top_p * d.total;
  // largest bit pattern b with sum(e >= b) >= P; weights are in (0, 1]
  uint32_t lo = 0, hi = 0x3f800001u;  // sum(e >= 0) = total >= P; nothing is above 1
  // Weights below c0 = (1 - top_p) total / V cannot decide the threshold: all V
  // of them together hold at most (1 - top_p) of the mass, so sum(e >= c0) >= P
  // and theta >= c0. The few weights at or above c0 are compacted into LDS and
  // one wave bisects over them without block barriers.
  const float c0 = (1.f - top_p) * d.total / (float)V;
  const uint32_t b0 = __float_as_uint(c0);
  int nc = 0;
  float f0 = 0.f;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const bool c = __float_as_uint(e[i]) >= b0 && e[i] > 0.f;
    nc += c ? 1 : 0;
    f0 += c ? e[i] : 0.f;
  }
  // exclusive prefix of the candidate counts in thread order
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  int incl = nc;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int up = __shfl_up(incl, o, 64);
    if (lane >= o) incl += up;
  }
  if (lane == 63) sh.woff[wave] = incl;
  const float F0 = block_sum(f0, sh);  // (also orders the woff writes before the reads)
  int base = 0, n_cand = 0;
#pragma unroll
  for (int w = 0; w < kRowWaves; ++w) {
    base += w < wave ? sh.woff[w] : 0;
    n_cand += sh.woff[w];
  }
  if (F0 >= P && b0 > 0 && n_cand <= kMaxCand) {
    int pos = base + incl - nc;
#pragma unroll
    for (int i = 0; i < EPT; ++i)
      if (__float_as_uint(e[i]) >= b0 && e[i] > 0.f) sh.cand[pos++] = e[i];
    __syncthreads();
    if (wave == 0) {
      constexpr int PER = kMaxCand / 64;
      float cv[PER];
#pragma unroll
      for (int q = 0; q < PER; ++q) {
        const int k = q * 64 + lane;
        cv[q] = k < n_cand ? sh.cand[k] : 0.f;
      }
      uint32_t wlo = b0, whi = hi;  // sum(e >= b0) = F0 >= P
      while (whi - wlo > 1) {
        const uint32_t mid = wlo + (whi - wlo) / 2;
        float part = 0.f;
#pragma unroll
        for (int q = 0; q < PER; ++q) part += __float_as_uint(cv[q]) >= mid ? cv[q] : 0.f;
        if (wave_sum_f(part) >= P)
          wlo = mid;
        else
          whi = mid;
      }
      if (lane == 0) sh.ibcast[2] = (int)wlo;
    }
    __syncthreads();
    lo = (uint32_t)sh.ibcast[2];
    __syncthreads();
  } else {
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
    const float need = P - mass_above;
    k = (int)ceilf(need / d.theta);
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
    const int v = threadIdx.x + kRowThreads * i;
    kp += kept_w(e[i], v, d) ? e[i] : 0.f;
  }
  d.kept = block_sum(kp, sh);
  return d;
}

// Draw from a row's distribution with uniform u (weights in `e`, parameters in
// d); `e` is overwritten with the kept weights.
template <int EPT>
__device__ __forceinline__ int row_draw(float* e, const RowDist& d, float u, RowShared& sh) {
  int last = -1;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const int v = threadIdx.x + kRowThreads * i;
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
  float best = -INFINITY;
  int bi = 0x7fffffff;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const int v = threadIdx.x + kRowThreads * i;
    if (v < V) {
      const float x = row[v];
      if (x > best) {  // v increases with i: strict > keeps the lowest index
        best = x;
        bi = v;
      }
    }
  }
  block_argmax(best, bi, sh);
  return bi;
}

// Normalised probability of token x under a row's distribution (0 outside [0, V)).
template <int EPT>
__device__ __forceinline__ float weight_at(const float* e, const RowDist& d, int x, int V, RowShared& sh) {
  if (x >= 0 && x < V && (x % kRowThreads) == (int)threadIdx.x) {
    const int i = x / kRowThreads;
    float w = 0.f;
#pragma unroll
    for (int j = 0; j < EPT; ++j)
      if (j == i) w = kept_w(e[j], x, d) ? e[j] : 0.f;
    sh.bcast[2] = w / d.kept;
  }
  __syncthreads();
  const float r = (x >= 0 && x < V) ? sh.bcast[2] : 0.f;
  __syncthreads();
  return r;
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
    const RowDist d = row_dist<EPT>(row, (int)a.V, a.inv_temp, a.top_p, e, sh);
    tok = row_draw<EPT>(e, d, a.u[r], sh);
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
  const RowDist d = row_dist<EPT>(row, (int)a.V, a.inv_temp, a.top_p, e, sh);
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

// Draw with uniform u from a row's distribution, weights recomputed from the logits.
template <int EPT>
__device__ __forceinline__ int draw_kept(const float* row, int V, float it, const RowDist& d,
                                         float u, RowShared& sh) {
  auto w = [&](int i) {
    const int v = threadIdx.x + kRowThreads * i;
    if (v >= V) return 0.f;
    const float e = exp_weight(row[v], it, d);
    return kept_w(e, v, d) ? e : 0.f;
  };
  int v = index_order_draw<EPT>(w, u * d.kept, sh);
  if (v < 0) {
    int last = -1;
    for (int i = 0; i < EPT; ++i)
      if (w(i) > 0.f) last = threadIdx.x + kRowThreads * i;
    float lv = (float)last;
    block_argmax(lv, last, sh);
    v = last;
  }
  return v;
}

// Verification: one block per sequence. Rows' parameters come from
// row_params_kernel; weights are recomputed from the logits as needed (the
// rows stay in L2), so no per-thread arrays are held.
template <int EPT>
__global__ __launch_bounds__(kRowThreads) void verify_kernel(VerifyArgs a) {
  __shared__ RowShared sh;
  const int64_t b = blockIdx.x;
  const int V = (int)a.V;
  const int G = a.gamma;
  const float it = a.inv_temp;
  int k = 0;
  int next = 0;
  for (; k < G; ++k) {
    const int x = a.draft_tokens[(int64_t)k * a.batch + b];
    const float* trow = a.target_logits + (b * (G + 1) + k) * a.V;
    if (a.greedy) {
      const int best = row_argmax<EPT>(trow, V, sh);
      if (best != x) {
        next = best;
        break;
      }
      continue;
    }
    const float* drow = a.draft_logits + ((int64_t)k * a.batch + b) * a.V;
    const RowDist dq = a.params[(int64_t)k * a.batch + b];
    const RowDist dp = a.params[a.batch * G + b * (G + 1) + k];
    const bool in = x >= 0 && x < V;
    const float qx = in ? prob_at(drow, x, it, dq) : 0.f;
    const float px = in ? prob_at(trow, x, it, dp) : 0.f;
    if (a.u_accept[(int64_t)k * a.batch + b] * qx < px) continue;
    // rejected: draw from max(0, p - q)
    auto res = [&](int i) {
      const int v = threadIdx.x + kRowThreads * i;
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
          if (res(i) > 0.f) last = threadIdx.x + kRowThreads * i;
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
    if (a.greedy) {
      next = row_argmax<EPT>(trow, V, sh);
    } else {
      const RowDist dp = a.params[a.batch * G + b * (G + 1) + G];
      next = draw_kept<EPT>(trow, V, it, dp, a.u_sample[b], sh);
    }
  }
  if (threadIdx.x == 0) {
    a.n_accepted[b] = k;
    a.next_token[b] = next;
  }
}

using HeadWide = WideMma<128, 128, 2, 2, 2>;
using HeadGenBf16 = TileMma<Bf16, 128, 128, 2, 2>;
using HeadGenF32 = TileMma<F32, 128, 128, 2, 2>;

}  // namespace

int head_tile() { return 128; }
int row_elems_per_thread(int64_t V) {
  for (int e : {16, 32, 48, 64})
    if (V <= (int64_t)e * kRowThreads) return e;
  return 0;
}

hipError_t launch_head_logits(const HeadArgs& a, bool f32, bool wide, hipStream_t stream) {
  const dim3 grid((unsigned)a.n_tt * (unsigned)a.n_vt);
  if (f32)
    hipLaunchKernelGGL((head_logits_kernel<HeadGenF32, F32>), grid, dim3(HeadGenF32::NT), 0, stream,
                       a);
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

hipError_t launch_verify(const VerifyArgs& a, int ept, hipStream_t stream) {
  const dim3 grid((unsigned)a.batch);
  switch (ept) {
    case 16: hipLaunchKernelGGL(verify_kernel<16>, grid, dim3(kRowThreads), 0, stream, a); break;
    case 32: hipLaunchKernelGGL(verify_kernel<32>, grid, dim3(kRowThreads), 0, stream, a); break;
    case 48: hipLaunchKernelGGL(verify_kernel<48>, grid, dim3(kRowThreads), 0, stream, a); break;
    case 64: hipLaunchKernelGGL(verify_kernel<64>, grid, dim3(kRowThreads), 0, stream, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace mls
