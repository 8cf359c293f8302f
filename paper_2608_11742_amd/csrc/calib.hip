// Register-only MFMA throughput of the device, for the benchmark's roofline:
// v_mfma_f32_16x16x32_bf16 back to back on operands held in registers, no
// memory traffic.  With constant operands the MFMA datapath toggles little;
// with operands that change at every instruction (random bf16 values, as a
// GEMM on real data feeds it) it draws more power and the sustained clock,
// and with it the attainable rate, drops below the published peak.
#include "kernels.h"
#include "common.h"

namespace dllm {

// written only if a result takes an impossible value; external linkage, so
// that the store, and with it the MFMA chain, stays observable
__device__ float mfma_calib_sink;

namespace {

constexpr int kCalThreads = 512;   // 8 waves, two per SIMD
constexpr int kCalAcc = 16;        // independent accumulators per lane

__device__ __forceinline__ float cal_rand(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352dU;
  x ^= x >> 15;
  x *= 0x846ca68bU;
  x ^= x >> 16;
  return (float(x & 0xFFFFFF) / 16777216.0f - 0.5f) * 4.0f;
}

template <bool RAND>
__global__ __launch_bounds__(kCalThreads, 2) void mfma_calib_kernel(int iters, uint32_t seed) {
  u32x4 a[8], b[8];
  const uint32_t t = blockIdx.x * kCalThreads + threadIdx.x;
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t e = uint32_t(j * 4 + w);
      a[j][w] = RAND ? pack_bf16x2(cal_rand(seed + t * 131u + 2 * e), cal_rand(seed + t * 131u + 2 * e + 1))
                     : pack_bf16x2(0.25f, 0.25f);
      b[j][w] = RAND ? pack_bf16x2(cal_rand(seed * 7u + t * 71u + 2 * e + 1000u),
                                   cal_rand(seed * 7u + t * 71u + 2 * e + 1001u))
                     : pack_bf16x2(0.5f, 0.5f);
    }
  f32x4 acc[kCalAcc];
#pragma unroll
  for (int j = 0; j < kCalAcc; ++j) acc[j] = f32x4{cal_rand(t + j), cal_rand(t + j + 5), cal_rand(t + j + 9), 0.f};
  for (int it = 0; it < iters; ++it) {
    // every instruction takes a different (a, b) pair than the one before
#pragma unroll
    for (int j = 0; j < kCalAcc; ++j) Mfma<bf16_t>::run(acc[j], a[j & 7], b[(j * 3 + 1) & 7]);
#pragma unroll
    for (int j = 0; j < kCalAcc; ++j) Mfma<bf16_t>::run(acc[j], a[(j * 5 + 2) & 7], b[j & 7]);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < kCalAcc; ++j) s += acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
  if (s == 1.2345e-30f) mfma_calib_sink = s;
}

}  // namespace

hipError_t mfma_calibration(bool random_operands, int iters, int workgroups, double* flop, hipStream_t s) {
  if (iters < 1 || workgroups < 1) return hipErrorInvalidValue;
  *flop = double(workgroups) * (kCalThreads / kWave) * double(iters) * 2 * kCalAcc * (2.0 * 16 * 16 * 32);
  if (random_operands)
    hipLaunchKernelGGL(mfma_calib_kernel<true>, dim3(workgroups), dim3(kCalThreads), 0, s, iters, 12345u);
  else
    hipLaunchKernelGGL(mfma_calib_kernel<false>, dim3(workgroups), dim3(kCalThreads), 0, s, iters, 12345u);
  return hipGetLastError();
}

}  // namespace dllm
