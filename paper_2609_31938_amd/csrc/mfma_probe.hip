// Measurement support: the rate the bf16 matrix cores sustain on this device
// with nothing else to do.  Each wave issues v_mfma_f32_16x16x32_bf16 back to
// back on 8 independent accumulators (enough to cover the instruction's
// latency), reads no memory in the loop, and writes one reduction per lane
// at the end so the work is kept.  The rate is the published peak scaled by
// the clock the device holds under matrix-core load.
#include "c3c_internal.h"

namespace c3c {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));

constexpr int CHAINS = 8;

__global__ __launch_bounds__(256, 1) void mfma_probe(float* out, int iters) {
  const int tid = threadIdx.x;
  // operands from the lane index (not constants the compiler could fold):
  // small values so that the sums stay finite
  const short v = static_cast<short>(0x3c00 + (tid & 7));  // bf16 in [2^-7, 2^-6)
  const i16x8 ai = {v, v, v, v, v, v, v, v};
  const bf16x8 a = __builtin_bit_cast(bf16x8, ai), b = a;
  f32x4 acc[CHAINS];
#pragma unroll
  for (int q = 0; q < CHAINS; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};
  // four iterations per loop trip (iters is rounded up to a multiple of 4 by
  // the host)
  // Each product is written with its accumulator as both source and
  // destination (a tied "+a" operand), so every accumulator stays in the same
  // registers for the whole loop: with the compiler's builtin, the register
  // allocator rotated the accumulators through other registers at every loop
  // trip, and those moves, not the matrix cores, set the one-wave rate.
  for (int i = 0; i < iters; i += 4) {
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int q = 0; q < CHAINS; ++q)
        asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc[q]) : "v"(a), "v"(b));
  }
  float s = 0.f;
#pragma unroll
  for (int q = 0; q < CHAINS; ++q) s += acc[q][0] + acc[q][1] + acc[q][2] + acc[q][3];
  out[static_cast<int64_t>(blockIdx.x) * 256 + tid] = s;
}

}  // namespace

hipError_t launch_mfma_probe(int64_t blocks, int64_t iters, float* out, hipStream_t s) {
  if (blocks <= 0 || blocks > 0x7fffffff || iters <= 0 || iters > 0x7ffffff0 || out == nullptr)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(mfma_probe, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, out,
                     static_cast<int>((iters + 3) / 4 * 4));
  return hipGetLastError();
}

double mfma_probe_flops(int64_t blocks, int64_t iters) {
  // 4 waves per workgroup, CHAINS products of 16 x 16 x 32 per iteration,
  // iterations rounded up to a multiple of 4 as launched
  return 2.0 * 16 * 16 * 32 * CHAINS * 4.0 * static_cast<double>(blocks) *
         static_cast<double>((iters + 3) / 4 * 4);
}

}  // namespace c3c
