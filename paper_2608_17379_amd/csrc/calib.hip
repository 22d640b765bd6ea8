// Measurement support (not part of the attention path): the sustained bf16
// MFMA rate of the chip under full load, against which the kernels' fraction
// of peak is read.  The quoted dense peak, 2516.6 TFLOP/s, is 256 CUs x
// 2.4 GHz x 4096 flop per clock per CU, i.e. one v_mfma_f32_32x32x16_bf16
// (32768 flop) per 32 clocks on each of a CU's four SIMDs.  The kernel runs
// that instruction in independent chains on register operands, with no
// memory traffic in the loop, so its rate divided by the CU count and the
// measured graphics clock gives the flop per clock per CU that the chip
// actually sustains.
//
// Built into libcalib.so, which only the benchmark's calibration mode loads.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;

constexpr int kChains = 8;   // independent accumulators per wavefront
constexpr int kThreads = 256;

// Each wavefront: iters x kChains MFMAs.  The operands depend on the lane so
// that nothing folds; every lane writes one sum of its accumulators, which
// keeps the work live.
__global__ __launch_bounds__(kThreads, 2) void mfma_rate_kernel(int iters, float* out) {
  const int t = (int)threadIdx.x;
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(0.001f * (float)((t + e) & 7));
    b[e] = (__bf16)(0.002f * (float)((t * 3 + e) & 7));
  }
  f32x16 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[c][r] = 0.f;
  for (int i = 0; i < iters; ++i)
#pragma unroll
    for (int c = 0; c < kChains; ++c)
      acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  out[(int64_t)blockIdx.x * kThreads + t] = s;
}

}  // namespace

// Enqueue `blocks` workgroups of 4 wavefronts, each wavefront issuing
// iters * 8 v_mfma_f32_32x32x16_bf16 (32768 flop each); `out` is a device
// buffer of blocks * 256 floats.  Returns 0, or -1 on bad arguments, or the
// hipError_t of the launch.
extern "C" int calib_mfma_rate(int blocks, int iters, float* out, hipStream_t stream) {
  if (blocks <= 0 || iters <= 0 || !out) return -1;
  hipLaunchKernelGGL(mfma_rate_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, stream, iters,
                     out);
  return (int)hipGetLastError();
}

extern "C" int calib_mfma_chains(void) { return kChains; }
