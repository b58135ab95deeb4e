// Wave-wide reductions and scans over the 64 lanes of a wave.
//
// Lane values move through the DPP datapath: quad permutes and row mirrors
// or right shifts inside each 16-lane row, then lane reads (v_readlane) of the
// four row results. A cross-lane permute through the LDS crossbar costs a full
// LDS round trip per step; these cost a few VALU cycles each, which matters for
// the many short, serially dependent reductions of per-row sampling.
//
// Requirements and guarantees:
// * all 64 lanes of the wave are active (call from wave-uniform control flow);
// * every lane receives the same reduction result, and the combination order
//   is fixed, so floating-point results are bitwise reproducible. Each pair
//   step adds a value to its partner's and the partner adds them the other
//   way round; IEEE addition is commutative, so both lanes agree bitwise.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>

namespace mls {

namespace dppc {
constexpr int kXor1 = 0xB1;        // quad_perm [1,0,3,2]: lane i <- i ^ 1
constexpr int kXor2 = 0x4E;        // quad_perm [2,3,0,1]: lane i <- i ^ 2
constexpr int kHalfMirror = 0x141; // lane i <- 7 - i within each 8-lane half row
constexpr int kMirror = 0x140;     // lane i <- 15 - i within each 16-lane row
constexpr int kShr = 0x110;        // kShr + n: lane i <- lane i - n of the same row
}  // namespace dppc

// Value of the DPP source lane; lanes whose source lies outside their row
// (row shifts) receive `fill`.
template <int Ctrl>
__device__ __forceinline__ float dpp_move(float v, float fill) {
  return __int_as_float(
      __builtin_amdgcn_update_dpp(__float_as_int(fill), __float_as_int(v), Ctrl, 0xf, 0xf, false));
}
template <int Ctrl>
__device__ __forceinline__ int dpp_move(int v, int fill) {
  return __builtin_amdgcn_update_dpp(fill, v, Ctrl, 0xf, 0xf, false);
}

__device__ __forceinline__ float lane_read(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}
__device__ __forceinline__ int lane_read(int v, int lane) {
  return __builtin_amdgcn_readlane(v, lane);
}

__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_move<dppc::kXor1>(v, 0.f);
  v += dpp_move<dppc::kXor2>(v, 0.f);
  v += dpp_move<dppc::kHalfMirror>(v, 0.f);
  v += dpp_move<dppc::kMirror>(v, 0.f);
  return (lane_read(v, 0) + lane_read(v, 16)) + (lane_read(v, 32) + lane_read(v, 48));
}

__device__ __forceinline__ int wave_sum(int v) {
  v += dpp_move<dppc::kXor1>(v, 0);
  v += dpp_move<dppc::kXor2>(v, 0);
  v += dpp_move<dppc::kHalfMirror>(v, 0);
  v += dpp_move<dppc::kMirror>(v, 0);
  return (lane_read(v, 0) + lane_read(v, 16)) + (lane_read(v, 32) + lane_read(v, 48));
}

__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_move<dppc::kXor1>(v, -INFINITY));
  v = fmaxf(v, dpp_move<dppc::kXor2>(v, -INFINITY));
  v = fmaxf(v, dpp_move<dppc::kHalfMirror>(v, -INFINITY));
  v = fmaxf(v, dpp_move<dppc::kMirror>(v, -INFINITY));
  return fmaxf(fmaxf(lane_read(v, 0), lane_read(v, 16)), fmaxf(lane_read(v, 32), lane_read(v, 48)));
}

// (val, idx) with the largest val, the lowest idx among equal values.
__device__ __forceinline__ bool argmax_better(float ov, int oi, float v, int i) {
  return ov > v || (ov == v && oi < i);
}
template <int Ctrl>
__device__ __forceinline__ void argmax_step(float& v, int& i) {
  const float ov = dpp_move<Ctrl>(v, v);
  const int oi = dpp_move<Ctrl>(i, i);
  if (argmax_better(ov, oi, v, i)) {
    v = ov;
    i = oi;
  }
}
__device__ __forceinline__ void wave_argmax(float& v, int& i) {
  argmax_step<dppc::kXor1>(v, i);
  argmax_step<dppc::kXor2>(v, i);
  argmax_step<dppc::kHalfMirror>(v, i);
  argmax_step<dppc::kMirror>(v, i);
  float bv = lane_read(v, 0);
  int bi = lane_read(i, 0);
#pragma unroll
  for (int r = 16; r < 64; r += 16) {
    const float ov = lane_read(v, r);
    const int oi = lane_read(i, r);
    if (argmax_better(ov, oi, bv, bi)) {
      bv = ov;
      bi = oi;
    }
  }
  v = bv;
  i = bi;
}

// Inclusive prefix sum over the lanes in lane order.
__device__ __forceinline__ float wave_incl_scan(float v) {
  v += dpp_move<dppc::kShr + 1>(v, 0.f);
  v += dpp_move<dppc::kShr + 2>(v, 0.f);
  v += dpp_move<dppc::kShr + 4>(v, 0.f);
  v += dpp_move<dppc::kShr + 8>(v, 0.f);
  const int row = (threadIdx.x & 63) >> 4;
  const float t0 = lane_read(v, 15);
  const float t1 = lane_read(v, 31);
  const float t2 = lane_read(v, 47);
  const float t01 = t0 + t1;
  const float off = row == 0 ? 0.f : row == 1 ? t0 : row == 2 ? t01 : t01 + t2;
  return row == 0 ? v : v + off;
}

__device__ __forceinline__ int wave_incl_scan(int v) {
  v += dpp_move<dppc::kShr + 1>(v, 0);
  v += dpp_move<dppc::kShr + 2>(v, 0);
  v += dpp_move<dppc::kShr + 4>(v, 0);
  v += dpp_move<dppc::kShr + 8>(v, 0);
  const int row = (threadIdx.x & 63) >> 4;
  const int t0 = lane_read(v, 15);
  const int t1 = lane_read(v, 31);
  const int t2 = lane_read(v, 47);
  return v + (row == 0 ? 0 : row == 1 ? t0 : row == 2 ? t0 + t1 : t0 + t1 + t2);
}

}  // namespace mls
