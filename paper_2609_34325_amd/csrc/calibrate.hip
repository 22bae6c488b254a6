// Measurement helper for the benchmark (not part of the DORA boundary): a
// kernel that keeps the bf16 matrix units busy, so the benchmark can report
// attention throughput against the MFMA rate this device actually sustains
// next to the data-sheet peak.
//
// Every wave runs `iters` rounds of 8 independent v_mfma_f32_16x16x32_bf16
// chains on register operands (16 x 16 x 32 x 2 = 16384 flops each) and
// writes one float per lane so nothing is optimised away.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kChains = 8;

__global__ __launch_bounds__(256) void mfma_bf16_loop(int iters, float seed, float* out) {
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = static_cast<__bf16>(seed * (threadIdx.x + e));
    b[e] = static_cast<__bf16>(seed * (blockIdx.x - e));
  }
  floatx4 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) acc[c] = floatx4{0.f, 0.f, 0.f, static_cast<float>(c)};
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c) s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
  out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

}  // namespace

// Launches `blocks` workgroups of 256 threads (4 waves), each wave issuing
// iters * 8 MFMAs; returns 0 or the HIP error code.  `out` holds blocks * 256
// floats.
extern "C" int dora_calibrate_mfma_bf16(int blocks, int iters, float* out, void* stream) {
  hipLaunchKernelGGL(mfma_bf16_loop, dim3(blocks), dim3(256), 0, static_cast<hipStream_t>(stream), iters, 1e-3f,
                     out);
  return static_cast<int>(hipGetLastError());
}

// Flops one launch performs.
extern "C" double dora_calibrate_mfma_bf16_flops(int blocks, int iters) {
  return static_cast<double>(blocks) * 4 * iters * kChains * 16384.0;
}
