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
// rescaled with the teacher's max.
struct RowState {
  float m[kMaxModels];
  float s1[kMaxModels];
  float st[kMaxModels];
  float xr[kMaxModels];
};

// arr[s] for a runtime s, with compile-time indices (keeps arr in registers)
template <typename X>
__device__ __forceinline__ X pick(const X* arr, int s) {
  X r = arr[0];
#pragma unroll
  for (int i = 1; i < kMaxModels; ++i)
    if (i == s) r = arr[i];
  return r;
}

__device__ __forceinline__ void absorb(RowState& st, int M, int s, float ct, const float4* rec) {
  // rec[i] = partial of sub-model i (same vocabulary range for all i). The
  // teacher's entries are picked with compile-time indices so that rec and st
  // stay in registers.
  float ms_old = 0.f, rs_x = 0.f;
#pragma unroll
  for (int i = 0; i < kMaxModels; ++i)
    if (i == s) {
      ms_old = st.m[i];
      rs_x = rec[i].x;
    }
  const float ms_new = fmaxf(ms_old, rs_x);
  const float wa = fast_exp2((ms_old - ms_new) * ct);
  const float wb = fast_exp2((rs_x - ms_new) * ct);
#pragma unroll
  for (int i = 0; i < kMaxModels; ++i) {
    if (i >= M) continue;  // (not break: keeps the loop fully unrolled)
    const float mo = st.m[i];
    const float mn = fmaxf(mo, rec[i].x);
    st.s1[i] = st.s1[i] * fast_exp2((mo - mn) * kLog2e) + rec[i].y * fast_exp2((rec[i].x - mn) * kLog2e);
    st.st[i] = st.st[i] * fast_exp2((mo - mn) * ct) + rec[i].z * fast_exp2((rec[i].x - mn) * ct);
    st.xr[i] = st.xr[i] * wa + rec[i].w * wb;
    st.m[i] = mn;
  }
}

constexpr int kRowTok = 16;   // tokens per block
constexpr int kRowGrp = 16;   // partial groups per token (merged in a fixed order)

__global__ __launch_bounds__(kThreads) void finalize_rows_kernel(RowArgs a) {
  __shared__ float4 sh[kRowGrp - 1][kRowTok][kMaxModels];
  const int tl = threadIdx.x % kRowTok;
  const int grp = threadIdx.x / kRowTok;
  const int64_t t = (int64_t)blockIdx.x * kRowTok + tl;
  const int M = a.M;
  const int s = a.teacher;
  const float inv_tau = 1.0f / a.tau;
  const float ct = kLog2e * inv_tau;

  RowState st;
#pragma unroll
  for (int i = 0; i < kMaxModels; ++i) {
    st.m[i] = -INFINITY;
    st.s1[i] = 0.f;
    st.st[i] = 0.f;
    st.xr[i] = 0.f;
  }
  if (t < a.T) {
#pragma unroll 4
    for (int j = grp; j < a.n_vt; j += kRowGrp) {
      float4 rec[kMaxModels];
#pragma unroll
      for (int i = 0; i < kMaxModels; ++i)
        if (i < M) rec[i] = a.partials[((int64_t)i * a.n_vt + j) * a.T + t];
      absorb(st, M, s, ct, rec);
    }
  }
  if (grp > 0) {
#pragma unroll
    for (int i = 0; i < kMaxModels; ++i)
      if (i < M) sh[grp - 1][tl][i] = make_float4(st.m[i], st.s1[i], st.st[i], st.xr[i]);
  }
  __syncthreads();
  if (grp != 0 || t >= a.T) return;
  for (int g2 = 0; g2 < kRowGrp - 1; ++g2) {
    float4 rec[kMaxModels];
#pragma unroll
    for (int i = 0; i < kMaxModels; ++i)
      if (i < M) rec[i] = sh[g2][tl][i];
    if (pick(rec, s).x == -INFINITY) continue;  // group saw no tile
    absorb(st, M, s, ct, rec);
  }

  const int64_t y = a.labels[t];
  const bool valid = y != a.ignore_index && y >= 0 && y < a.V;
  const int64_t T = a.T;
  float* lse1 = a.stats;
  float* lset = a.stats + (int64_t)M * T;
  float* ce_row = a.stats + 2 * (int64_t)M * T;
  float* kl_row = a.stats + 3 * (int64_t)M * T;
  float* h_row = a.stats + 4 * (int64_t)M * T;
  const float m_s = pick(st.m, s), st_s = pick(st.st, s), xr_s = pick(st.xr, s);
  const float lset_s = m_s * inv_tau + logf(st_s);
  const float den = a.tau * st_s;
#pragma unroll
  for (int i = 0; i < kMaxModels; ++i) {
    if (i >= M) continue;
    const float l1 = st.m[i] + logf(st.s1[i]);
    const float lt = st.m[i] * inv_tau + logf(st.st[i]);
    lse1[i * T + t] = l1;
    lset[i * T + t] = lt;
    ce_row[i * T + t] = valid ? l1 - a.lab[i * T + t] : 0.f;
    kl_row[i * T + t] = (valid && i != s) ? (xr_s - st.xr[i]) / den - lset_s + lt : 0.f;
  }
  h_row[t] = valid ? lset_s - xr_s / den : 0.f;
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

constexpr int kRedThreads = 1024;

__global__ __launch_bounds__(kRedThreads) void reduce_losses_kernel(RowArgs a) {
  constexpr int kQ = 2 * kMaxModels + 3;  // ce[8], kl[8], h, count, flag
  __shared__ double part[kRedThreads / 64][kQ];
  const int M = a.M;
  const int64_t T = a.T;
  double acc[kQ];
#pragma unroll
  for (int q = 0; q < kQ; ++q) acc[q] = 0.0;
  const float* ce_row = a.stats + 2 * (int64_t)M * T;
  const float* kl_row = a.stats + 3 * (int64_t)M * T;
  const float* h_row = a.stats + 4 * (int64_t)M * T;
  for (int64_t t = threadIdx.x; t < T; t += kRedThreads) {
    const int64_t y = a.labels[t];
    if (y != a.ignore_index) {
      if (y >= 0 && y < a.V) acc[2 * kMaxModels + 1] += 1.0;
      else acc[2 * kMaxModels + 2] = 1.0;
    }
#pragma unroll
    for (int i = 0; i < kMaxModels; ++i) {
      if (i >= M) continue;
      acc[i] += ce_row[i * T + t];
      acc[kMaxModels + i] += kl_row[i * T + t];
    }
    acc[2 * kMaxModels] += h_row[t];
  }
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
#pragma unroll
  for (int q = 0; q < kQ; ++q) {
    const double v = wave_sum(acc[q]);
    if (lane == 0) part[wave][q] = v;
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
  double tot[kQ];
  for (int q = 0; q < kQ; ++q) {
    tot[q] = 0.0;
    for (int w = 0; w < kRedThreads / 64; ++w) tot[q] += part[w][q];
  }
  const double n = tot[2 * kMaxModels + 1];
  const double inv = n > 0 ? 1.0 / n : 0.0;
  for (int i = 0; i < M; ++i) {
    a.ce[i] = (float)(tot[i] * inv);
    a.kl[i] = i == a.teacher ? 0.f : (float)(tot[kMaxModels + i] * inv);
  }
  if (a.entropy) *a.entropy = (float)(tot[2 * kMaxModels] * inv);
  a.header[0] = (int32_t)n;
  a.header[1] = tot[2 * kMaxModels + 2] > 0 ? MLS_DEVFLAG_LABEL_RANGE : 0;
}

}  // namespace

hipError_t launch_label_logits(const RowArgs& a, bool f32, hipStream_t stream) {
  const int64_t waves = (int64_t)a.M * a.T;
  dim3 grid((unsigned)((waves + 3) / 4));
  if (f32)
    hipLaunchKernelGGL(label_logits_kernel<F32>, grid, dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(label_logits_kernel<Bf16>, grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_finalize_rows(const RowArgs& a, hipStream_t stream) {
  dim3 grid((unsigned)((a.T + kRowTok - 1) / kRowTok));
  hipLaunchKernelGGL(finalize_rows_kernel, grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_reduce_losses(const RowArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(reduce_losses_kernel, dim3(1), dim3(kRedThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace mls
