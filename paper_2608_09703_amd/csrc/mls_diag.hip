// Cross-model diagnostics (paper section 3, "Training Dynamics and Model
// Agreement"): for every ordered pair of sub-models (i, j), the mean over valid
// tokens of KL(p_i || p_j) at temperature 1 and the rate at which their top-1
// next-token predictions agree (argmax ties go to the lowest vocabulary index).
//
// One pass, normalising itself. One block owns one (vocabulary tile, token
// tile) pair, as the fused forward does, and computes the logits tile of every
// sub-model (all M accumulator sets stay in registers, M <= 4; larger suites
// run one such pass per subset of four sub-models, the subsets covering every
// pair). Per token and
// sub-model i, relative to the largest logit m_i seen so far:
//   Z_i  = sum_v exp(l_i - m_i)
//   S_ij = sum_v exp(l_i - m_i) (l_i - l_j)      for every ordered pair i != j
// and the argmax of l_i (its value is m_i). Two partial results (m, Z, S) and
// (m', Z', S') merge as m'' = max(m, m'), Z'' = Z e^{m - m''} + Z' e^{m' - m''},
// S'' likewise with the scale of model i. Across lanes, waves, vocabulary tiles
// and slices the same merge applies; at the end, with lse_i = m_i + log Z_i,
//   KL(p_i || p_j) = sum_v p_i (l_i - l_j) - lse_i + lse_j = S_ij / Z_i - lse_i + lse_j.
// No [T, V] tensor is formed and no forward statistics are needed.
#include <math.h>

#include "mls_core.h"
#include "mls_device.h"
#include "mls_launch.h"

namespace mls {

namespace {

template <int MM>
struct DiagRec {
  // per (vocabulary tile, token): S[MM][MM], Z[MM], best (= m)[MM], index[MM]
  static constexpr int kS = 0;
  static constexpr int kZ = MM * MM;
  static constexpr int kBest = MM * MM + MM;
  static constexpr int kIdx = MM * MM + 2 * MM;
  static constexpr int kFloats = MM * MM + 3 * MM;
};

// e^{x - m} for x <= m, where x = -inf marks an empty partial (its sums are 0)
__device__ __forceinline__ float rescale(float x, float m) {
  return x == -INFINITY ? 0.f : fast_exp2((x - m) * kLog2e);
}

// Merges partial (ob, oi, oz, os) into (b, bi, z, s) for one sub-model i; os/s
// are its MM pair sums S_i*.
template <int MM>
__device__ __forceinline__ void merge_part(float& b, int& bi, float& z, float* s, float ob, int oi,
                                           float oz, const float* os) {
  const float m = fmaxf(b, ob);
  const float sa = rescale(b, m);
  const float sb = rescale(ob, m);
  z = z * sa + oz * sb;
#pragma unroll
  for (int j = 0; j < MM; ++j) s[j] = s[j] * sa + os[j] * sb;
  if (ob > b || (ob == b && oi < bi)) {
    b = ob;
    bi = oi;
  }
}

template <class Mma, typename E, int MM, int MINB>
__global__ __launch_bounds__(Mma::NT, MINB) void diag_tile_kernel(DiagArgs a) {
  constexpr int BM = Mma::kBM;
  constexpr int BN = Mma::kBN;
  constexpr int WGM = Mma::kWGM;
  constexpr int FM = Mma::FM;
  constexpr int FN = Mma::FN;
  using R = DiagRec<MM>;
  constexpr int REC = R::kFloats;
  static_assert(WGM == kDiagParts, "one record per wave row");
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

  Mma mma[MM];
#pragma unroll
  for (int j = 0; j < MM; ++j) {
    const int64_t kb = a.d[j] * E::kBytes;
    mma[j].run(static_cast<const char*>(a.W[j]), kb, vbase, a.V, static_cast<const char*>(a.h[j]),
               kb, tbase, a.T, kb, smem, tid);
  }
  // record of this wave row: [vocabulary tile * WGM + wm][field][token]
  float* const out0 = a.partials + ((int64_t)vt * WGM + wm) * REC * a.T;

#pragma unroll
  for (int fn = 0; fn < FN; ++fn) {
    // first sweep over the lane's rows: argmax, whose value is the lane's maximum
    float best[MM];
    int bidx[MM];
#pragma unroll
    for (int i = 0; i < MM; ++i) {
      best[i] = -INFINITY;
      bidx[i] = 0x7fffffff;
    }
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int v = (int)vbase + Mma::row_of(wm, fm, r, lane);
        const bool ok = full || v < a.V;
#pragma unroll
        for (int i = 0; i < MM; ++i) {
          const float l = mma[i].acc[fm][fn][r];
          // rows are visited in increasing order within a lane: strict > keeps the lowest
          if (ok && l > best[i]) {
            best[i] = l;
            bidx[i] = v;
          }
        }
      }
    // second sweep: sums relative to that maximum (a lane with no row keeps 0)
    float mb[MM], Z[MM], S[MM][MM];
#pragma unroll
    for (int i = 0; i < MM; ++i) {
      mb[i] = best[i] == -INFINITY ? 0.f : best[i] * kLog2e;
      Z[i] = 0.f;
#pragma unroll
      for (int j = 0; j < MM; ++j) S[i][j] = 0.f;
    }
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int v = (int)vbase + Mma::row_of(wm, fm, r, lane);
        const bool ok = full || v < a.V;
        float l[MM], p[MM];
#pragma unroll
        for (int i = 0; i < MM; ++i) {
          l[i] = mma[i].acc[fm][fn][r];
          p[i] = ok ? fast_exp2(fmaf(l[i], kLog2e, -mb[i])) : 0.f;
          Z[i] += p[i];
        }
#pragma unroll
        for (int i = 0; i < MM; ++i)
#pragma unroll
          for (int j = 0; j < MM; ++j)
            if (j != i) S[i][j] = fmaf(p[i], l[i] - l[j], S[i][j]);
      }

    // lanes l and l ^ 32 hold the same token column: merge, and the lower
    // half writes the wave's record (consecutive lanes, consecutive tokens)
#pragma unroll
    for (int i = 0; i < MM; ++i) {
      float os[MM];
#pragma unroll
      for (int j = 0; j < MM; ++j) os[j] = __shfl_xor(S[i][j], 32, 64);
      const float oz = __shfl_xor(Z[i], 32, 64);
      const float ob = __shfl_xor(best[i], 32, 64);
      const int oi = __shfl_xor(bidx[i], 32, 64);
      merge_part<MM>(best[i], bidx[i], Z[i], S[i], ob, oi, oz, os);
    }
    const int64_t t = tbase + Mma::col_of(wn, fn, lane);
    if (hi == 0 && t < a.T) {
      float* out = out0 + t;
#pragma unroll
      for (int i = 0; i < MM; ++i) {
#pragma unroll
        for (int j = 0; j < MM; ++j) out[(int64_t)(R::kS + i * MM + j) * a.T] = S[i][j];
        out[(int64_t)(R::kZ + i) * a.T] = Z[i];
        out[(int64_t)(R::kBest + i) * a.T] = best[i];
        out[(int64_t)(R::kIdx + i) * a.T] = __int_as_float(bidx[i]);
      }
    }
  }
}

// Per token: merge the records of all vocabulary tiles (kDiagParts per tile),
// finish KL(p_i || p_j) and the argmax, and write the per-token values the
// mean reduction reads. A block takes kRowTok tokens; its kRowSlices thread
// rows each merge every kRowSlices-th record, and the slices are merged in a
// fixed order.
constexpr int kRowTok = 32;
constexpr int kRowSlices = 16;

template <int MM>
__global__ __launch_bounds__(kRowTok * kRowSlices) void diag_rows_kernel(DiagArgs a) {
  using R = DiagRec<MM>;
  constexpr int REC = R::kFloats;
  __shared__ float sh[kRowSlices][REC][kRowTok];
  const int c = threadIdx.x % kRowTok;
  const int g = threadIdx.x / kRowTok;
  const int64_t t = (int64_t)blockIdx.x * kRowTok + c;
  float S[MM][MM], Z[MM], best[MM];
  int bidx[MM];
#pragma unroll
  for (int i = 0; i < MM; ++i) {
    best[i] = -INFINITY;
    bidx[i] = 0x7fffffff;
    Z[i] = 0.f;
#pragma unroll
    for (int j = 0; j < MM; ++j) S[i][j] = 0.f;
  }
  if (t < a.T) {
    for (int q = g; q < a.n_vt * kDiagParts; q += kRowSlices) {
      const float* in = a.partials + (int64_t)q * REC * a.T + t;
#pragma unroll
      for (int i = 0; i < MM; ++i) {
        float os[MM];
#pragma unroll
        for (int j = 0; j < MM; ++j) os[j] = in[(int64_t)(R::kS + i * MM + j) * a.T];
        merge_part<MM>(best[i], bidx[i], Z[i], S[i], in[(int64_t)(R::kBest + i) * a.T],
                       __float_as_int(in[(int64_t)(R::kIdx + i) * a.T]),
                       in[(int64_t)(R::kZ + i) * a.T], os);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < MM; ++i) {
#pragma unroll
    for (int j = 0; j < MM; ++j) sh[g][R::kS + i * MM + j][c] = S[i][j];
    sh[g][R::kZ + i][c] = Z[i];
    sh[g][R::kBest + i][c] = best[i];
    sh[g][R::kIdx + i][c] = __int_as_float(bidx[i]);
  }
  __syncthreads();
  if (g != 0 || t >= a.T) return;
  for (int w = 1; w < kRowSlices; ++w) {
#pragma unroll
    for (int i = 0; i < MM; ++i) {
      float os[MM];
#pragma unroll
      for (int j = 0; j < MM; ++j) os[j] = sh[w][R::kS + i * MM + j][c];
      merge_part<MM>(best[i], bidx[i], Z[i], S[i], sh[w][R::kBest + i][c],
                     __float_as_int(sh[w][R::kIdx + i][c]), sh[w][R::kZ + i][c], os);
    }
  }
  const int64_t y = a.labels[t];
  const bool valid = y != a.ignore_index && y >= 0 && y < a.V;
  float lse[MM];
#pragma unroll
  for (int i = 0; i < MM; ++i) lse[i] = best[i] + logf(Z[i]);
  float* row = a.rowvals + t * (2 * MM * MM);
#pragma unroll
  for (int i = 0; i < MM; ++i) {
    const float invz = 1.f / Z[i];
#pragma unroll
    for (int j = 0; j < MM; ++j) {
      row[i * MM + j] = (valid && i != j) ? S[i][j] * invz - lse[i] + lse[j] : 0.f;
      row[MM * MM + i * MM + j] = (valid && bidx[i] == bidx[j]) ? 1.f : 0.f;
    }
    if (a.argmax) a.argmax[(int64_t)i * a.T + t] = bidx[i];
  }
}

constexpr int kRedThreads = 1024;

template <int MM>
__global__ __launch_bounds__(kRedThreads) void diag_mean_kernel(DiagArgs a) {
  constexpr int Q = 2 * MM * MM + 1;  // kl[MM][MM], agree[MM][MM], count
  __shared__ double part[kRedThreads / 64][Q];
  double acc[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) acc[q] = 0.0;
  for (int64_t t = threadIdx.x; t < a.T; t += kRedThreads) {
    const int64_t y = a.labels[t];
    if (y != a.ignore_index && y >= 0 && y < a.V) acc[Q - 1] += 1.0;
    const float* row = a.rowvals + t * (2 * MM * MM);
#pragma unroll
    for (int q = 0; q < 2 * MM * MM; ++q) acc[q] += row[q];
  }
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    double v = acc[q];
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    if (lane == 0) part[wave][q] = v;
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
  double tot[Q];
  for (int q = 0; q < Q; ++q) {
    tot[q] = 0.0;
    for (int w = 0; w < kRedThreads / 64; ++w) tot[q] += part[w][q];
  }
  const double n = tot[Q - 1];
  const double inv = n > 0 ? 1.0 / n : 0.0;
  for (int q = 0; q < MM * MM; ++q) {
    a.kl_pair[q] = (float)(tot[q] * inv);
    a.agree[q] = (float)(tot[MM * MM + q] * inv);
  }
}

// All M accumulator sets of a tile stay live. Up to M = 3 the wide bf16 path
// runs four waves of 64x64 (64 accumulators per lane per model) at two blocks
// per CU; for M = 4 that no longer fits, and four waves of 64x32 (32 per
// model) take a 128x64 tile, still two blocks per CU (two independent blocks
// hide each other's barriers better than one eight-wave block on 128x128).
// The general path uses the four-wave register-staged core on 128x64.
using DiagWide = WideMma<kFusedWideBM, kDiagBN, 2, 2, 2>;
using DiagWide4 = WideMma<kFusedWideBM, kDiagBN / 2, 2, 2, 2>;
template <typename E>
using DiagGen = TileMma<E, kFusedBM, kDiagGenBN, 2, 2>;

template <int MM>
hipError_t launch_tiles_m(const DiagArgs& a, bool f32, bool wide, hipStream_t stream) {
  const dim3 grid((unsigned)a.n_tt * (unsigned)a.n_vt);
  if (f32)
    hipLaunchKernelGGL((diag_tile_kernel<DiagGen<F32>, F32, MM, 2>), grid, dim3(kThreads), 0,
                       stream, a);
  else if (wide) {
    if constexpr (MM <= 3)
      hipLaunchKernelGGL((diag_tile_kernel<DiagWide, Bf16, MM, 2>), grid, dim3(DiagWide::NT), 0,
                         stream, a);
    else
      hipLaunchKernelGGL((diag_tile_kernel<DiagWide4, Bf16, MM, 2>), grid, dim3(DiagWide4::NT), 0,
                         stream, a);
  }
  else
    hipLaunchKernelGGL((diag_tile_kernel<DiagGen<Bf16>, Bf16, MM, 2>), grid, dim3(kThreads), 0,
                       stream, a);
  return hipGetLastError();
}

template <int MM>
hipError_t launch_reduce_m(const DiagArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(diag_rows_kernel<MM>, dim3((unsigned)((a.T + kRowTok - 1) / kRowTok)),
                     dim3(kRowTok * kRowSlices), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(diag_mean_kernel<MM>, dim3(1), dim3(kRedThreads), 0, stream, a);
  return hipGetLastError();
}

__global__ __launch_bounds__(kThreads) void diag_scatter_kernel(DiagScatterArgs a) {
  const int64_t t = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (t < (int64_t)a.n * a.n) {
    const int r = (int)t / a.n;
    const int c = (int)t % a.n;
    a.kl_pair[a.sub[r] * a.M + a.sub[c]] = a.kl_sub[t];
    a.agree[a.sub[r] * a.M + a.sub[c]] = a.agree_sub[t];
  }
  if (a.argmax && t < a.T) {
    for (int k = 0; k < a.n; ++k) a.argmax[(int64_t)a.sub[k] * a.T + t] = a.am_sub[(int64_t)k * a.T + t];
  }
}

}  // namespace

hipError_t launch_diag_scatter(const DiagScatterArgs& a, hipStream_t stream) {
  const int64_t n = a.T > 64 ? a.T : 64;
  hipLaunchKernelGGL(diag_scatter_kernel, dim3((unsigned)((n + kThreads - 1) / kThreads)), dim3(kThreads),
                     0, stream, a);
  return hipGetLastError();
}

int diag_tile_rows(bool wide) { return wide ? kFusedWideBM : kFusedBM; }
int diag_tile_cols(bool wide, int M) { return wide ? (M == 4 ? kDiagBN / 2 : kDiagBN) : kDiagGenBN; }
int diag_record_floats(int M) { return M * M + 3 * M; }

hipError_t launch_diag_tiles(const DiagArgs& a, bool f32, bool wide, hipStream_t stream) {
  switch (a.M) {
    case 1: return launch_tiles_m<1>(a, f32, wide, stream);
    case 2: return launch_tiles_m<2>(a, f32, wide, stream);
    case 3: return launch_tiles_m<3>(a, f32, wide, stream);
    case 4: return launch_tiles_m<4>(a, f32, wide, stream);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_diag_reduce(const DiagArgs& a, hipStream_t stream) {
  switch (a.M) {
    case 1: return launch_reduce_m<1>(a, stream);
    case 2: return launch_reduce_m<2>(a, stream);
    case 3: return launch_reduce_m<3>(a, stream);
    case 4: return launch_reduce_m<4>(a, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace mls
