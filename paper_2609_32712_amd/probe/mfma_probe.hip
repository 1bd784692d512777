// Measurement probe for the benchmark: the rate at which one MI355X runs
// v_mfma_f32_32x32x16_bf16 when nothing else limits it (operands in registers, four
// independent accumulator chains per wavefront, three wavefronts per SIMD, no memory
// traffic in the loop).  It states the practical MFMA ceiling and clock of the
// machine a benchmark ran on, beside the rated 2.5 PFLOP/s that the roofline
// fraction uses.
// Not part of libmala.so.
#include <hip/hip_runtime.h>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kChains = 4;

__global__ __launch_bounds__(256) void mfma_probe_kernel(float* out, int iters) {
  // operands that depend on the thread, so that nothing folds
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(1e-3f * (float)((threadIdx.x + i) & 7));
    b[i] = (__bf16)(1e-3f * (float)((threadIdx.x * 3 + i) & 7));
  }
  f32x16 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[c][r] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kChains; ++c)
      acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

}  // namespace

extern "C" {

// Enqueues the probe on `stream` (a hipStream_t): `blocks` workgroups of 256 threads,
// each wavefront running iters x 4 MFMAs of 32 x 32 x 16 (32768 flops each); `out`
// is a device buffer of blocks x 256 floats.  Returns 0, or -4 if the launch failed.
int mala_probe_mfma(float* out, int blocks, int iters, void* stream) {
  if (!out || blocks <= 0 || iters <= 0) return -1;
  hipLaunchKernelGGL(mfma_probe_kernel, dim3((unsigned)blocks), dim3(256), 0,
                     (hipStream_t)stream, out, iters);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // extern "C"
