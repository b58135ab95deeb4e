// Per-row kernels of the forward pass:
//  - label logits l_i[t, y_t] = <h_i[t], W_i[y_t]> (next-token cross-entropy,
//    paper section 2, "Inter-model Junction", last paragraph);
//  - merge of the per-tile partial statistics into per-row log-sum-exp values,
//    cross-entropy, KL(q || p_i^tau) and the teacher entropy (eq. (2) is
//    KL + entropy);
//  - the deterministic mean over valid tokens.
#include <math.h>

#include "mls_device.h"
#include "mls_launch.h"

namespace mls {

namespace {

template <typename E>
__global__ __launch_bounds__(kThreads) void label_logits_kernel(RowArgs a) {
  using S = typename E::storage;
  const int lane = threadIdx.x & 63;
  const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (w >= (int64_t)a.M * a.T) return;
  const int i = (int)(w / a.T);
  const int64_t t = w % a.T;
  const int64_t y = a.labels[t];
  const bool valid = y != a.ignore_index && y >= 0 && y < a.V;
  float s = 0.f;
  if (valid) {
    constexpr int kPer = 16 / E::kBytes;  // elements per 16-byte load
    const S* hp = static_cast<const S*>(a.h[i]) + t * a.d[i];
    const S* wp = static_cast<const S*>(a.W[i]) + y * a.d[i];
    for (int64_t k = (int64_t)lane * kPer; k < a.d[i]; k += 64 * kPer) {
      const uint4 hv = *reinterpret_cast<const uint4*>(hp + k);
      const uint4 wv = *reinterpret_cast<const uint4*>(wp + k);
      const uint32_t hu[4] = {hv.x, hv.y, hv.z, hv.w};
      const uint32_t wu[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (E::kBytes == 2) {
          s = fmaf(__uint_as_float(hu[q] << 16), __uint_as_float(wu[q] << 16), s);
          s = fmaf(__uint_as_float(hu[q] & 0xffff0000u), __uint_as_float(wu[q] & 0xffff0000u), s);
        } else {
          s = fmaf(__uint_as_float(hu[q]), __uint_as_float(wu[q]), s);
        }
      }
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
  if (lane == 0) a.lab[(int64_t)i * a.T + t] = s;
}

// Running merge of partial rows. Every sub-model keeps its own max m,
// sum exp(l - m) (s1) and sum exp((l - m) / tau) (st); the cross terms xr of
// every sub-model are weighted by the teacher's exponentials, so they are
// rescaled with the teacher's max. Slots follow the processing order, slot 0
// being the teacher; MM (the number of sub-models) is a compile-time constant,
// so every array is indexed with constants and stays in registers.
template <int MM>
struct RowState {
  float m[MM];
  float s1[MM];
  float st[MM];
  float xr[MM];
};

// rec[k] = partial of slot k over one vocabulary range (the same for all k)
template <int MM>
__device__ __forceinline__ void absorb(RowState<MM>& st, float ct, const float4* rec) {
  const float ms_new = fmaxf(st.m[0], rec[0].x);
  const float wa = fast_exp2((st.m[0] - ms_new) * ct);
  const float wb = fast_exp2((rec[0].x - ms_new) * ct);
#pragma unroll
  for (int k = 0; k < MM; ++k) {
    const float mo = st.m[k];
    const float mn = fmaxf(mo, rec[k].x);
    st.s1[k] = st.s1[k] * fast_exp2((mo - mn) * kLog2e) + rec[k].y * fast_exp2((rec[k].x - mn) * kLog2e);
    st.st[k] = st.st[k] * fast_exp2((mo - mn) * ct) + rec[k].z * fast_exp2((rec[k].x - mn) * ct);
    st.xr[k] = st.xr[k] * wa + rec[k].w * wb;
    st.m[k] = mn;
  }
}

// 4 tokens x 64 groups: 25 records per thread at the headline shape rather than
// 49 with 8 x 32 (row merge 39 -> 34 us per launch)
constexpr int kRowTok = 4;    // tokens per block
constexpr int kRowGrp = 64;   // partial groups per token, merged pairwise in a fixed tree
static_assert(kRowTok * kRowGrp == kThreads && (kRowGrp & (kRowGrp - 1)) == 0, "row merge shape");
static_assert(kFusedBN % kRowTok == 0, "a block's tokens lie in one token tile");

// Tokens [t0, t0 + Tc) of one forward chunk: its partial records are indexed
// by the token inside the chunk, the statistics by the token itself.
template <int MM>
__global__ __launch_bounds__(kThreads) void finalize_rows_kernel(RowArgs a) {
  __shared__ float4 sh[kRowGrp][kRowTok][MM];
  const int tl = threadIdx.x % kRowTok;
  const int grp = threadIdx.x / kRowTok;
  const int64_t tc = (int64_t)blockIdx.x * kRowTok + tl;  // token inside the chunk
  const float inv_tau = 1.0f / a.tau;
  const float ct = kLog2e * inv_tau;

  RowState<MM> st;
#pragma unroll
  for (int i = 0; i < MM; ++i) {
    st.m[i] = -INFINITY;
    st.s1[i] = 0.f;
    st.st[i] = 0.f;
    st.xr[i] = 0.f;
  }
  if (tc < a.Tc) {
    const int64_t n_tt = (a.Tc + kFusedBN - 1) / kFusedBN;
    const float4* part = a.partials + (tc / kFusedBN) * a.n_rec * kFusedBN + tc % kFusedBN;
#pragma unroll 4
    for (int j = grp; j < a.n_rec; j += kRowGrp) {
      float4 rec[MM];
#pragma unroll
      for (int k = 0; k < MM; ++k) rec[k] = part[((int64_t)k * n_tt * a.n_rec + j) * kFusedBN];
      if (rec[0].x != -INFINITY) absorb<MM>(st, ct, rec);  // else rows all beyond V
    }
  }
  // group g absorbs group g + w for w = kRowGrp / 2, ..., 1 (every thread
  // takes part in the barriers; columns past T only merge among themselves)
#pragma unroll
  for (int i = 0; i < MM; ++i) sh[grp][tl][i] = make_float4(st.m[i], st.s1[i], st.st[i], st.xr[i]);
#pragma unroll
  for (int w = kRowGrp / 2; w >= 1; w >>= 1) {
    __syncthreads();
    if (grp < w) {
      float4 rec[MM];
#pragma unroll
      for (int i = 0; i < MM; ++i) rec[i] = sh[grp + w][tl][i];
      if (rec[0].x != -INFINITY) {  // else that group saw no record
        absorb<MM>(st, ct, rec);
        if (w > 1) {
#pragma unroll
          for (int i = 0; i < MM; ++i)
            sh[grp][tl][i] = make_float4(st.m[i], st.s1[i], st.st[i], st.xr[i]);
        }
      }
    }
  }
  if (grp != 0 || tc >= a.Tc) return;

  const int64_t t = a.t0 + tc;
  const int64_t y = a.labels[t];
  const bool valid = y != a.ignore_index && y >= 0 && y < a.V;
  const int64_t T = a.T;
  float* lse1 = a.stats;
  float* lset = a.stats + (int64_t)MM * T;
  float* ce_row = a.stats + 2 * (int64_t)MM * T;
  float* kl_row = a.stats + 3 * (int64_t)MM * T;
  float* h_row = a.stats + 4 * (int64_t)MM * T;
  const float lset_s = st.m[0] * inv_tau + logf(st.st[0]);
  const float den = a.tau * st.st[0];
  const float xr_s = st.xr[0];
#pragma unroll
  for (int k = 0; k < MM; ++k) {
    const int64_t i = a.order[k];
    const float l1 = st.m[k] + logf(st.s1[k]);
    const float lt = st.m[k] * inv_tau + logf(st.st[k]);
    lse1[i * T + t] = l1;
    lset[i * T + t] = lt;
    ce_row[i * T + t] = valid ? l1 - a.lab[i * T + t] : 0.f;
    kl_row[i * T + t] = (valid && k != 0) ? (xr_s - st.xr[k]) / den - lset_s + lt : 0.f;
  }
  h_row[t] = valid ? lset_s - xr_s / den : 0.f;
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

constexpr int kRedThreads = 1024;

// MM = the number of sub-models, so that every load of a token is issued
// before the first sum needs one (one memory round trip per token rather than
// one per sub-model); the sums run in the same order for every MM.
template <int MM>
__global__ __launch_bounds__(kRedThreads) void reduce_losses_kernel(RowArgs a) {
  constexpr int kQ = 2 * kMaxModels + 4;  // ce[8], kl[8], h, count, flag, sum of every lse
  __shared__ double part[kRedThreads / 64][kQ];
  constexpr int M = MM;
  const int64_t T = a.T;
  double acc[kQ];
#pragma unroll
  for (int q = 0; q < kQ; ++q) acc[q] = 0.0;
  const float* ce_row = a.stats + 2 * (int64_t)M * T;
  const float* kl_row = a.stats + 3 * (int64_t)M * T;
  const float* h_row = a.stats + 4 * (int64_t)M * T;
  const float* lse = a.stats;  // lse1[M][T] then lset[M][T]
  for (int64_t t = threadIdx.x; t < T; t += kRedThreads) {
    const int64_t y = a.labels[t];
    float ce[MM], kl[MM], l1[MM], lt[MM];
#pragma unroll
    for (int i = 0; i < MM; ++i) {
      ce[i] = ce_row[i * T + t];
      kl[i] = kl_row[i * T + t];
      l1[i] = lse[i * T + t];
      lt[i] = lse[(M + i) * T + t];
    }
    const float hv = h_row[t];
    if (y != a.ignore_index) {
      if (y >= 0 && y < a.V) acc[2 * kMaxModels + 1] += 1.0;
      else acc[2 * kMaxModels + 2] = 1.0;
    }
#pragma unroll
    for (int i = 0; i < MM; ++i) {
      acc[i] += ce[i];
      acc[kMaxModels + i] += kl[i];
      acc[2 * kMaxModels + 3] += (double)l1[i] + (double)lt[i];
    }
    acc[2 * kMaxModels] += hv;
  }
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
#pragma unroll
  for (int q = 0; q < kQ; ++q) {
    const double v = wave_sum(acc[q]);
    if (lane == 0) part[wave][q] = v;
  }
  __syncthreads();
  // one thread per quantity sums the waves' parts in wave order
  __shared__ double tot_sh[kQ];
  if (threadIdx.x < kQ) {
    double v = 0.0;
    for (int w = 0; w < kRedThreads / 64; ++w) v += part[w][threadIdx.x];
    tot_sh[threadIdx.x] = v;
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
  double tot[kQ];
#pragma unroll
  for (int q = 0; q < kQ; ++q) tot[q] = tot_sh[q];
  const double n = tot[2 * kMaxModels + 1];
  const double inv = n > 0 ? 1.0 / n : 0.0;
  for (int i = 0; i < M; ++i) {
    a.ce[i] = (float)(tot[i] * inv);
    a.kl[i] = i == a.teacher ? 0.f : (float)(tot[kMaxModels + i] * inv);
  }
  if (a.entropy) *a.entropy = (float)(tot[2 * kMaxModels] * inv);
  // losses of ignored tokens are exact zeros; the log-sum-exp rows of every
  // token (ignored ones too) are summed as well
  bool finite = isfinite(tot[2 * kMaxModels]) && isfinite(tot[2 * kMaxModels + 3]);
  for (int i = 0; i < M; ++i) finite = finite && isfinite(tot[i]) && isfinite(tot[kMaxModels + i]);
  a.header[0] = (int32_t)n;
  a.header[1] = (tot[2 * kMaxModels + 2] > 0 ? MLS_DEVFLAG_LABEL_RANGE : 0) |
                (finite ? 0 : MLS_DEVFLAG_NONFINITE);
}

// Number of valid tokens into the statistics header (the fused forward +
// backward needs it before the loss mean is taken).
__global__ __launch_bounds__(kRedThreads) void count_valid_kernel(RowArgs a) {
  __shared__ int part[kRedThreads / 64];
  int n = 0;
  for (int64_t t = threadIdx.x; t < a.T; t += kRedThreads) {
    const int64_t y = a.labels[t];
    n += (y != a.ignore_index && y >= 0 && y < a.V) ? 1 : 0;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) n += __shfl_xor(n, o, 64);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = n;
  __syncthreads();
  if (threadIdx.x != 0) return;
  int tot = 0;
  for (int w = 0; w < kRedThreads / 64; ++w) tot += part[w];
  a.header[0] = tot;
}

// Logit gradient of one token chunk from its stored logits, in place:
//   G_i = ( g_ce,i (softmax(l_i) - onehot(y)) + g_kl,i / tau (softmax(l_i / tau) - q) ) / N
// (eq. (2) with stop_grad on q = softmax(l_s / tau), eq. (3) through the
// coefficients), with l = m + d rebuilt from the stored fp16 distance d to the
// partial record's maximum m. One wave per token row, 8 vocabulary entries per
// lane (16-byte loads and stores), the teacher first so that its q stays in
// registers for the students. Ignored tokens, padding rows and entries past V
// get exact zeros. The slab is streamed once through, with non-temporal loads
// and stores (0.419 -> 0.403 ms per step at the headline shape).
constexpr int kGradTok = 4;    // token rows per block, one per wave
constexpr int kGradSpan = 512; // vocabulary entries per wave

__device__ __forceinline__ void unpack_f16x8(uint4 v, float* d) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    d[2 * k] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w[k] & 0xffffu));
    d[2 * k + 1] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w[k] >> 16));
  }
}

__device__ __forceinline__ uint4 pack_bf16x8(const float* g) {
  uint32_t w[4];
#pragma unroll
  for (int k = 0; k < 4; ++k)
    w[k] = (uint32_t)to_storage<Bf16>(g[2 * k]) | ((uint32_t)to_storage<Bf16>(g[2 * k + 1]) << 16);
  return make_uint4(w[0], w[1], w[2], w[3]);
}

template <bool TAU1>
__global__ __launch_bounds__(kThreads) void grad_logits_kernel(GradArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t tc = (int64_t)blockIdx.y * kGradTok + wave;
  const int64_t v0 = (int64_t)blockIdx.x * kGradSpan + (int64_t)lane * 8;
  if (tc >= a.Tc_pad || v0 >= a.ld) return;  // no barrier follows
  const int64_t stride = a.Tc_pad * a.ld;
  const int64_t t = a.t0 + tc;
  int64_t y = tc < a.Tc ? a.labels[t] : a.ignore_index;
  const bool valid = tc < a.Tc && y != a.ignore_index && y >= 0 && y < a.V;
  if (!valid) {
    for (int oi = 0; oi < a.M; ++oi)
      store16_nt(a.slab + a.order[oi] * stride + tc * a.ld + v0, make_uint4(0, 0, 0, 0));
    return;
  }
  const int nv = *a.n_valid;
  const float invN = nv > 0 ? 1.0f / (float)nv : 0.0f;
  const int yrel = (int)(y - v0);  // onehot position among this lane's 8 entries, if in [0, 8)
  const float ct = kLog2e * a.inv_tau;
  // partial record of this token and 64-entry group, for each slot
  const int64_t slot = (a.Tc_pad / kFusedBN) * a.n_rec * kFusedBN;
  const float4* rec = a.partials + ((tc / kFusedBN) * a.n_rec + v0 / 64) * kFusedBN + tc % kFusedBN;
  float q[8];
  for (int oi = 0; oi < a.M; ++oi) {
    const int i = a.order[oi];
    uint16_t* ptr = a.slab + i * stride + tc * a.ld + v0;
    float d[8];
    unpack_f16x8(load16_nt(ptr), d);
    const float m = rec[oi * slot].x;
    const float l1s = a.lse1[(int64_t)i * a.T + t] * kLog2e;
    const float lts = a.lset[(int64_t)i * a.T + t] * kLog2e;
    const float gce = a.g_ce ? a.g_ce[i] : a.host_gce[i];
    const float gkl = a.g_kl ? a.g_kl[i] : a.host_gkl[i];
    const float cg = gce * invN;
    const float ck = oi != 0 ? gkl * invN * a.inv_tau : 0.f;
    float g[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const bool ok = v0 + j < a.V;
      const float l = d[j] + m;
      const float oh = j == yrel ? 1.f : 0.f;
      if (oi == 0) {
        const float qj = ok ? fast_exp2(fmaf(l, ct, -lts)) : 0.f;
        q[j] = qj;
        const float p1 = TAU1 ? qj : (ok ? fast_exp2(fmaf(l, kLog2e, -l1s)) : 0.f);
        g[j] = cg * (p1 - oh);
      } else {
        const float p1 = ok ? fast_exp2(fmaf(l, kLog2e, -l1s)) : 0.f;
        const float pt = TAU1 ? p1 : (ok ? fast_exp2(fmaf(l, ct, -lts)) : 0.f);
        g[j] = fmaf(cg, p1 - oh, ck * (pt - q[j]));
      }
      g[j] = ok ? g[j] : 0.f;
    }
    store16_nt(ptr, pack_bf16x8(g));
  }
}

}  // namespace

hipError_t launch_count_valid(const RowArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(count_valid_kernel, dim3(1), dim3(kRedThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_grad_logits(const GradArgs& a, hipStream_t stream) {
  dim3 grid((unsigned)((a.ld + kGradSpan - 1) / kGradSpan), (unsigned)((a.Tc_pad + kGradTok - 1) / kGradTok));
  if (a.inv_tau == 1.0f)
    hipLaunchKernelGGL(grad_logits_kernel<true>, grid, dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(grad_logits_kernel<false>, grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_label_logits(const RowArgs& a, bool f32, hipStream_t stream) {
  const int64_t waves = (int64_t)a.M * a.T;
  dim3 grid((unsigned)((waves + 3) / 4));
  if (f32)
    hipLaunchKernelGGL(label_logits_kernel<F32>, grid, dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(label_logits_kernel<Bf16>, grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

template <int MM>
hipError_t launch_finalize_rows_m(const RowArgs& a, hipStream_t stream) {
  dim3 grid((unsigned)((a.Tc + kRowTok - 1) / kRowTok));
  hipLaunchKernelGGL(finalize_rows_kernel<MM>, grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_finalize_rows(const RowArgs& a, hipStream_t stream) {
  static_assert(kMaxModels == 8, "one instantiation per model count");
  switch (a.M) {
    case 1: return launch_finalize_rows_m<1>(a, stream);
    case 2: return launch_finalize_rows_m<2>(a, stream);
    case 3: return launch_finalize_rows_m<3>(a, stream);
    case 4: return launch_finalize_rows_m<4>(a, stream);
    case 5: return launch_finalize_rows_m<5>(a, stream);
    case 6: return launch_finalize_rows_m<6>(a, stream);
    case 7: return launch_finalize_rows_m<7>(a, stream);
    case 8: return launch_finalize_rows_m<8>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

template <int MM>
hipError_t launch_reduce_losses_m(const RowArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(reduce_losses_kernel<MM>, dim3(1), dim3(kRedThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_reduce_losses(const RowArgs& a, hipStream_t stream) {
  switch (a.M) {
    case 1: return launch_reduce_losses_m<1>(a, stream);
    case 2: return launch_reduce_losses_m<2>(a, stream);
    case 3: return launch_reduce_losses_m<3>(a, stream);
    case 4: return launch_reduce_losses_m<4>(a, stream);
    case 5: return launch_reduce_losses_m<5>(a, stream);
    case 6: return launch_reduce_losses_m<6>(a, stream);
    case 7: return launch_reduce_losses_m<7>(a, stream);
    case 8: return launch_reduce_losses_m<8>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace mls
