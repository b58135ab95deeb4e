// Inter-model junction (paper section 2, "Inter-model Junction", eq. (1)),
// forward and backward. Per token, the output o (width d_prev) of sub-model m
// is rescaled to the Euclidean norm of the fresh embedding e (width d_fresh)
// of sub-model m+1 and the two are concatenated:
//   s = ||e|| / ||o||,   x = [s*o | e]  (or [e | s*o])
// With g the upstream gradient on the s*o channels and g_e0 the one on the e
// channels:
//   dL/do = s * (g - (g.o) o / ||o||^2)
//   dL/de = g_e0 + (g.o) / ||o|| * e / ||e||
// A zero norm makes s and both ratio terms 0.
//
// Memory-bound: each operand is read once and each result written once.
// TPR threads own one token row (TPR/64 waves); every lane holds CPL chunks
// of 8 elements of each operand in registers: in the forward 8 consecutive
// elements (16-byte bf16 accesses), in the backward two groups of 4
// consecutive elements TPR groups apart, so that its fp32 accesses cover whole
// 1 KB runs per wave instruction. The row's dot products are reduced in fp32
// (wave shuffles, then LDS across the row's waves).
#include "mls_device.h"
#include "mls_launch.h"

namespace mls {

namespace {

constexpr int kJBlock = 256;

// Cache policy of each pass (both junctions of T = 32768 tokens at widths
// 1536 / 3072 / 4608, ms per step): non-temporal in the forward (0.179 ->
// 0.165) and in the backward with its lane mapping (0.448 -> 0.413; with the
// forward's mapping, 0.452 -> 0.462)
constexpr bool kFwdNT = true;
constexpr bool kBwdNT = true;

typedef unsigned int u32x2j __attribute__((ext_vector_type(2)));
template <bool NT>
__device__ __forceinline__ uint2 ld8(const void* p) {
  if (NT) {
    const u32x2j v = __builtin_nontemporal_load(static_cast<const u32x2j*>(p));
    return make_uint2(v.x, v.y);
  }
  return *reinterpret_cast<const uint2*>(p);
}
template <bool NT>
__device__ __forceinline__ void st8(void* p, uint2 v) {
  if (NT)
    __builtin_nontemporal_store(u32x2j{v.x, v.y}, static_cast<u32x2j*>(p));
  else
    *reinterpret_cast<uint2*>(p) = v;
}
template <bool NT>
__device__ __forceinline__ uint4 ld16(const void* p) {
  return NT ? load16_nt(p) : *reinterpret_cast<const uint4*>(p);
}
template <bool NT>
__device__ __forceinline__ void st16(void* p, uint4 v) {
  if (NT)
    store16_nt(p, v);
  else
    *reinterpret_cast<uint4*>(p) = v;
}

// 8 consecutive elements <-> 8 floats, 16-byte accesses (the forward's lane
// mapping)
template <bool NT>
__device__ __forceinline__ void load8(const uint16_t* p, float* v) {
  const uint4 r = ld16<NT>(p);
  const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(w[i] << 16);
    v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
template <bool NT>
__device__ __forceinline__ void load8(const float* p, float* v) {
  const uint4 a = ld16<NT>(p);
  const uint4 b = ld16<NT>(p + 4);
  v[0] = __uint_as_float(a.x); v[1] = __uint_as_float(a.y);
  v[2] = __uint_as_float(a.z); v[3] = __uint_as_float(a.w);
  v[4] = __uint_as_float(b.x); v[5] = __uint_as_float(b.y);
  v[6] = __uint_as_float(b.z); v[7] = __uint_as_float(b.w);
}
template <bool NT>
__device__ __forceinline__ void store8(uint16_t* p, const float* v) {
  uint4 r;
  r.x = (uint32_t)to_storage<Bf16>(v[0]) | ((uint32_t)to_storage<Bf16>(v[1]) << 16);
  r.y = (uint32_t)to_storage<Bf16>(v[2]) | ((uint32_t)to_storage<Bf16>(v[3]) << 16);
  r.z = (uint32_t)to_storage<Bf16>(v[4]) | ((uint32_t)to_storage<Bf16>(v[5]) << 16);
  r.w = (uint32_t)to_storage<Bf16>(v[6]) | ((uint32_t)to_storage<Bf16>(v[7]) << 16);
  st16<NT>(p, r);
}
template <bool NT>
__device__ __forceinline__ void store8(float* p, const float* v) {
  st16<NT>(p, make_uint4(__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]),
                         __float_as_uint(v[3])));
  st16<NT>(p + 4, make_uint4(__float_as_uint(v[4]), __float_as_uint(v[5]), __float_as_uint(v[6]),
                             __float_as_uint(v[7])));
}

// 4 consecutive elements <-> 4 floats, 8-byte (bf16) or 16-byte (fp32)
// accesses (the backward's lane mapping)
template <bool NT>
__device__ __forceinline__ void load4(const uint16_t* p, float* v) {
  const uint2 r = ld8<NT>(p);
  v[0] = __uint_as_float(r.x << 16);
  v[1] = __uint_as_float(r.x & 0xffff0000u);
  v[2] = __uint_as_float(r.y << 16);
  v[3] = __uint_as_float(r.y & 0xffff0000u);
}
template <bool NT>
__device__ __forceinline__ void load4(const float* p, float* v) {
  const uint4 r = ld16<NT>(p);
  v[0] = __uint_as_float(r.x);
  v[1] = __uint_as_float(r.y);
  v[2] = __uint_as_float(r.z);
  v[3] = __uint_as_float(r.w);
}
template <bool NT>
__device__ __forceinline__ void store4(uint16_t* p, const float* v) {
  st8<NT>(p, make_uint2((uint32_t)to_storage<Bf16>(v[0]) | ((uint32_t)to_storage<Bf16>(v[1]) << 16),
                        (uint32_t)to_storage<Bf16>(v[2]) | ((uint32_t)to_storage<Bf16>(v[3]) << 16)));
}
template <bool NT>
__device__ __forceinline__ void store4(float* p, const float* v) {
  st16<NT>(p, make_uint4(__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]),
                         __float_as_uint(v[3])));
}

template <typename T>
struct Elt;
template <>
struct Elt<Bf16> {
  typedef uint16_t type;
};
template <>
struct Elt<F32> {
  typedef float type;
};

// Sums NV values over the TPR threads of a row: wave shuffles, then the
// row's waves through LDS. Every thread of the block must call it.
template <int TPR, int NV>
__device__ __forceinline__ void row_sums(float* v, float (*red)[NV]) {
#pragma unroll
  for (int q = 0; q < NV; ++q)
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v[q] += __shfl_xor(v[q], o, 64);
  if (TPR == 64) return;
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0)
#pragma unroll
    for (int q = 0; q < NV; ++q) red[wave][q] = v[q];
  __syncthreads();
  const int first = wave / (TPR / 64) * (TPR / 64);
#pragma unroll
  for (int q = 0; q < NV; ++q) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < TPR / 64; ++w) s += red[first + w][q];
    v[q] = s;
  }
}

// Backward lane mapping: element offset of group g (0 or 1) of chunk c of
// lane j; groups of 4 elements, 2 * CPL of them per lane, TPR groups apart.
template <int TPR>
__device__ __forceinline__ int64_t group_at(int c, int g, int j) {
  return ((int64_t)(2 * c + g) * TPR + j) * 4;
}

template <typename A, int TPR, int CPL>
__global__ __launch_bounds__(kJBlock) void junction_fwd_kernel(JunctionArgs a) {
  typedef typename Elt<A>::type TA;
  __shared__ float red[kJBlock / 64][2];
  const int r = threadIdx.x / TPR;  // row within the block
  const int j = threadIdx.x % TPR;
  const int64_t t = (int64_t)blockIdx.x * (kJBlock / TPR) + r;
  const bool live = t < a.T;  // dead rows still join the block's barrier
  const int64_t dp = a.d_prev, df = a.d_fresh, w = dp + df;
  const TA* o = static_cast<const TA*>(a.o) + t * dp;
  const TA* e = static_cast<const TA*>(a.e) + t * df;
  float ov[CPL][8], ev[CPL][8];
  float s[2] = {0.f, 0.f};
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int64_t k = ((int64_t)c * TPR + j) * 8;
    if (live && k < dp) {
      load8<kFwdNT>(o + k, ov[c]);
#pragma unroll
      for (int i = 0; i < 8; ++i) s[0] = fmaf(ov[c][i], ov[c][i], s[0]);
    }
    if (live && k < df) {
      load8<kFwdNT>(e + k, ev[c]);
#pragma unroll
      for (int i = 0; i < 8; ++i) s[1] = fmaf(ev[c][i], ev[c][i], s[1]);
    }
  }
  row_sums<TPR, 2>(s, red);
  if (!live) return;
  const float scale = (s[0] > 0.f && s[1] > 0.f) ? sqrtf(s[1]) / sqrtf(s[0]) : 0.f;
  TA* x = static_cast<TA*>(a.x) + t * w;
  TA* xp = x + (a.prev_first ? 0 : df);
  TA* xf = x + (a.prev_first ? dp : 0);
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int64_t k = ((int64_t)c * TPR + j) * 8;
    if (k < dp) {
#pragma unroll
      for (int i = 0; i < 8; ++i) ov[c][i] *= scale;
      store8<kFwdNT>(xp + k, ov[c]);
    }
    if (k < df) store8<kFwdNT>(xf + k, ev[c]);
  }
}

template <typename A, typename G, int TPR, int CPL>
__global__ __launch_bounds__(kJBlock) void junction_bwd_kernel(JunctionArgs a) {
  typedef typename Elt<A>::type TA;
  typedef typename Elt<G>::type TG;
  __shared__ float red[kJBlock / 64][3];
  const int r = threadIdx.x / TPR;
  const int j = threadIdx.x % TPR;
  const int64_t t = (int64_t)blockIdx.x * (kJBlock / TPR) + r;
  const bool live = t < a.T;
  const int64_t dp = a.d_prev, df = a.d_fresh, w = dp + df;
  const TA* o = static_cast<const TA*>(a.o) + t * dp;
  const TA* e = static_cast<const TA*>(a.e) + t * df;
  const TG* gx = static_cast<const TG*>(a.g_x) + t * w;
  const TG* gp = gx + (a.prev_first ? 0 : df);
  const TG* gf = gx + (a.prev_first ? dp : 0);
  float ov[CPL][8], gv[CPL][8];
  float s[3] = {0.f, 0.f, 0.f};  // ||o||^2, ||e||^2, g.o
#pragma unroll
  for (int c = 0; c < CPL; ++c)
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      const int64_t k = group_at<TPR>(c, g, j);
      if (live && k < dp) {
        load4<kBwdNT>(o + k, &ov[c][4 * g]);
        load4<kBwdNT>(gp + k, &gv[c][4 * g]);
#pragma unroll
        for (int i = 4 * g; i < 4 * g + 4; ++i) {
          s[0] = fmaf(ov[c][i], ov[c][i], s[0]);
          s[2] = fmaf(gv[c][i], ov[c][i], s[2]);
        }
      }
    }
  // the fresh block's gradient is loaded here too, so that it is in flight
  // while the row reduction runs
  float ev[CPL][8], gdv[CPL][8];
#pragma unroll
  for (int c = 0; c < CPL; ++c)
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      const int64_t k = group_at<TPR>(c, g, j);
      if (live && k < df) {
        load4<kBwdNT>(e + k, &ev[c][4 * g]);
        load4<kBwdNT>(gf + k, &gdv[c][4 * g]);
#pragma unroll
        for (int i = 4 * g; i < 4 * g + 4; ++i) s[1] = fmaf(ev[c][i], ev[c][i], s[1]);
      }
    }
  row_sums<TPR, 3>(s, red);
  if (!live) return;
  const bool ok = s[0] > 0.f && s[1] > 0.f;
  const float no = sqrtf(s[0]), ne = sqrtf(s[1]);
  const float sc = ok ? ne / no : 0.f;              // s
  const float proj = ok ? s[2] / s[0] : 0.f;        // (g.o) / ||o||^2
  const float fe = ok ? (s[2] / no) / ne : 0.f;     // (g.o) / (||o|| ||e||)
  TG* go = static_cast<TG*>(a.g_o) + t * dp;
  TG* ge = static_cast<TG*>(a.g_e) + t * df;
#pragma unroll
  for (int c = 0; c < CPL; ++c)
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      const int64_t k = group_at<TPR>(c, g, j);
      if (k < dp) {
        float out[4];
        if (a.accumulate) load4<kBwdNT>(go + k, out);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float v = sc * fmaf(-proj, ov[c][4 * g + i], gv[c][4 * g + i]);
          out[i] = a.accumulate ? out[i] + v : v;
        }
        store4<kBwdNT>(go + k, out);
      }
      if (k < df) {
        float out[4];
        if (a.accumulate) load4<kBwdNT>(ge + k, out);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float v = fmaf(fe, ev[c][4 * g + i], gdv[c][4 * g + i]);
          out[i] = a.accumulate ? out[i] + v : v;
        }
        store4<kBwdNT>(ge + k, out);
      }
    }
}

template <typename A, int TPR>
hipError_t fwd_cpl(const JunctionArgs& a, int cpl, dim3 grid, hipStream_t s) {
  switch (cpl) {
    case 1: hipLaunchKernelGGL((junction_fwd_kernel<A, TPR, 1>), grid, dim3(kJBlock), 0, s, a); break;
    case 2: hipLaunchKernelGGL((junction_fwd_kernel<A, TPR, 2>), grid, dim3(kJBlock), 0, s, a); break;
    case 4: hipLaunchKernelGGL((junction_fwd_kernel<A, TPR, 4>), grid, dim3(kJBlock), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename A, typename G, int TPR>
hipError_t bwd_cpl(const JunctionArgs& a, int cpl, dim3 grid, hipStream_t s) {
  switch (cpl) {
    case 1: hipLaunchKernelGGL((junction_bwd_kernel<A, G, TPR, 1>), grid, dim3(kJBlock), 0, s, a); break;
    case 2: hipLaunchKernelGGL((junction_bwd_kernel<A, G, TPR, 2>), grid, dim3(kJBlock), 0, s, a); break;
    case 4: hipLaunchKernelGGL((junction_bwd_kernel<A, G, TPR, 4>), grid, dim3(kJBlock), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename A>
hipError_t fwd_tpr(const JunctionArgs& a, int tpr, int cpl, dim3 grid, hipStream_t s) {
  switch (tpr) {
    case 64: return fwd_cpl<A, 64>(a, cpl, grid, s);
    case 128: return fwd_cpl<A, 128>(a, cpl, grid, s);
    case 256: return fwd_cpl<A, 256>(a, cpl, grid, s);
  }
  return hipErrorInvalidValue;
}

template <typename A, typename G>
hipError_t bwd_tpr(const JunctionArgs& a, int tpr, int cpl, dim3 grid, hipStream_t s) {
  switch (tpr) {
    case 64: return bwd_cpl<A, G, 64>(a, cpl, grid, s);
    case 128: return bwd_cpl<A, G, 128>(a, cpl, grid, s);
    case 256: return bwd_cpl<A, G, 256>(a, cpl, grid, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

// Threads per row and 8-element chunks per lane for rows of up to `width`
// elements per operand: the fewest threads with at most 2 chunks each (more
// memory-level parallelism per byte of registers), else 256 threads with 4.
bool junction_shape(int64_t width, int* tpr, int* cpl) {
  const int64_t chunks = (width + 7) / 8;
  for (int t : {64, 128, 256})
    for (int c : {1, 2})
      if ((int64_t)t * c >= chunks) {
        *tpr = t;
        *cpl = c;
        return true;
      }
  if (chunks <= (int64_t)kJBlock * 4) {
    *tpr = kJBlock;
    *cpl = 4;
    return true;
  }
  return false;
}

int64_t junction_max_width() { return (int64_t)kJBlock * 4 * 8; }

hipError_t launch_junction_fwd(const JunctionArgs& a, bool act_f32, hipStream_t stream) {
  int tpr, cpl;
  if (!junction_shape(a.d_prev > a.d_fresh ? a.d_prev : a.d_fresh, &tpr, &cpl))
    return hipErrorInvalidValue;
  const dim3 grid((unsigned)((a.T + kJBlock / tpr - 1) / (kJBlock / tpr)));
  return act_f32 ? fwd_tpr<F32>(a, tpr, cpl, grid, stream) : fwd_tpr<Bf16>(a, tpr, cpl, grid, stream);
}

hipError_t launch_junction_bwd(const JunctionArgs& a, bool act_f32, bool grad_f32,
                               hipStream_t stream) {
  int tpr, cpl;
  if (!junction_shape(a.d_prev > a.d_fresh ? a.d_prev : a.d_fresh, &tpr, &cpl))
    return hipErrorInvalidValue;
  const dim3 grid((unsigned)((a.T + kJBlock / tpr - 1) / (kJBlock / tpr)));
  if (act_f32)
    return grad_f32 ? bwd_tpr<F32, F32>(a, tpr, cpl, grid, stream)
                    : bwd_tpr<F32, Bf16>(a, tpr, cpl, grid, stream);
  return grad_f32 ? bwd_tpr<Bf16, F32>(a, tpr, cpl, grid, stream)
                  : bwd_tpr<Bf16, Bf16>(a, tpr, cpl, grid, stream);
}

}  // namespace mls
