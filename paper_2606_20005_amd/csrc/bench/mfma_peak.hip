// Measured bf16 MFMA throughput of the chip, for the benchmark's "% of
// measured peak" figure (libstreamkl_bench.so; not part of the attention-KL
// library). Every wave loads eight A and eight B operands of
// v_mfma_f32_32x32x16_bf16 once from memory and then issues `iters` rounds of
// 16 MFMAs over four independent accumulators, each MFMA on a different
// operand pair, so the multipliers see the data's own switching activity
// (random operands draw more power than constant ones and lower the clock
// the chip sustains). Nothing else runs in the loop. Measured on MI355X,
// one such wave per SIMD sustains the most (about 1780 TFLOP/s on N(0,1)
// operands, 2450 on constant ones); two to eight waves per SIMD that each
// keep only two to four accumulators in flight sustain 25-30% less, unless
// each keeps eight.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWavesPerBlock = 4;
constexpr int kOperands = 16;   // 8 A + 8 B per wave, 64 lanes x 16 bytes each

__global__ void __launch_bounds__(64 * kWavesPerBlock)
mfma_peak_kernel(const u32x4* __restrict__ src, int iters, float* __restrict__ sink) {
  const int lane = threadIdx.x & 63;
  const size_t wave = (size_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
  const u32x4* p = src + wave * kOperands * 64 + lane;
  bf16x8 a[8], b[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = __builtin_bit_cast(bf16x8, p[64 * i]);
    b[i] = __builtin_bit_cast(bf16x8, p[64 * (8 + i)]);
  }
  f32x16 acc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[c][e] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 16; ++i)
      acc[i & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i & 7], b[(3 * i) & 7], acc[i & 3], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[c][e];
  sink[wave * 64 + lane] = s;
}

}  // namespace

// Launches `waves` waves (a multiple of 4) of the MFMA loop on `stream`.
// src: device memory of waves * 16 * 64 * 16 bytes of bf16 operands; sink:
// waves * 64 floats. Returns 0, or 1 for bad arguments, 3 if the launch
// failed. Flops per call: waves * iters * 16 * 32768.
extern "C" int streamkl_bench_mfma_peak(const void* src, int waves, int iters, float* sink, hipStream_t stream) {
  if (!src || !sink || waves <= 0 || waves % kWavesPerBlock != 0 || iters <= 0) return 1;
  if ((reinterpret_cast<uintptr_t>(src) & 15) != 0) return 1;
  hipLaunchKernelGGL(mfma_peak_kernel, dim3(waves / kWavesPerBlock), dim3(64 * kWavesPerBlock), 0, stream,
                     static_cast<const u32x4*>(src), iters, sink);
  return hipGetLastError() == hipSuccess ? 0 : 3;
}
