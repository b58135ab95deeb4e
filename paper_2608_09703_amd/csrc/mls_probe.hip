// Measurement aid: the MFMA ceiling of the part. Every wave issues long runs
// of independent v_mfma_f32_32x32x16_bf16 on operands held in registers (no
// memory traffic, no LDS), either all-zero or random bf16 values: the rate it
// reaches bounds what any kernel built on this instruction can do, and the
// difference between the two operand kinds shows the clock's response to the
// data's switching activity.
#include <hip/hip_runtime.h>

#include "mls.h"
#include "mls_device.h"
#include "mls_launch.h"

namespace mls {

namespace {

constexpr int kProbeBlocks = 2048;
constexpr int kProbeThreads = 256;
constexpr int kProbeChains = 8;  // independent accumulators per wave

__device__ __forceinline__ uint32_t hash32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

__global__ __launch_bounds__(kProbeThreads) void mfma_probe_kernel(int random, int iters, float* sink) {
  const uint32_t id = blockIdx.x * kProbeThreads + threadIdx.x;
  uint4 a[2], b[2];
  for (int k = 0; k < 2; ++k) {
    uint32_t w[8];
    for (int j = 0; j < 8; ++j) {
      // random bf16 pairs in [-2, 2) (exponent field kept in range), or zeros
      const uint32_t r = hash32(id * 16u + k * 8u + j);
      w[j] = random ? (r & 0x807f807fu) | 0x3f803f80u : 0u;
    }
    a[k] = make_uint4(w[0], w[1], w[2], w[3]);
    b[k] = make_uint4(w[4], w[5], w[6], w[7]);
  }
  f32x16_t acc[kProbeChains];
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[c][r] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kProbeChains; ++c) mma_step<Bf16>(acc[c], a[c & 1], b[(c >> 1) & 1]);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  sink[id] = s;
}

}  // namespace

hipError_t launch_mfma_probe(int random, int iters, float* sink, hipStream_t stream) {
  hipLaunchKernelGGL(mfma_probe_kernel, dim3(kProbeBlocks), dim3(kProbeThreads), 0, stream, random,
                     iters, sink);
  return hipGetLastError();
}

double mfma_probe_flops(int iters) {
  // 32 x 32 x 16 multiply-adds per instruction, per wave
  return 2.0 * 32 * 32 * 16 * (double)kProbeChains * iters * (kProbeBlocks * kProbeThreads / 64);
}

int64_t mfma_probe_sink_floats() { return (int64_t)kProbeBlocks * kProbeThreads; }

}  // namespace mls
