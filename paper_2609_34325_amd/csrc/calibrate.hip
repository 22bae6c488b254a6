// Measurement helpers for the benchmark (not part of the DORA boundary): a
// kernel that keeps the bf16 matrix units busy, and a streaming copy, so the
// benchmark can report attention and the HBM-bound kernels against what this
// device actually sustains next to the data-sheet peaks.
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

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Grid-stride copy of n16 16-byte vectors: one non-temporal load and one
// store per lane per step.  THROUGH stores with the write-through,
// non-temporal cache policy the library's output stores use (sc1 | nt);
// otherwise plain stores (lines left dirty in the L2, written back later).
template <bool THROUGH>
__global__ __launch_bounds__(256) void copy_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst, size_t n16) {
  const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
  for (size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n16; i += stride) {
    const u32x4 v = __builtin_nontemporal_load(src + i);
    if constexpr (THROUGH) {
      // The byte offset stays below 2^31: the host accepts at most 1 GiB.
      __builtin_amdgcn_raw_buffer_store_b128(v, __builtin_amdgcn_make_buffer_rsrc(dst, 0, 0x7FFFFFFF, 0x00020000),
                                             static_cast<uint32_t>(i * 16), 0, 16 | 2);
    } else {
      dst[i] = v;
    }
  }
}

}  // namespace

// Copies `bytes` (a multiple of 16, at most 1 GiB) from src to dst with
// `blocks` workgroups of 256 threads; through != 0 selects the write-through
// stores.  Returns 0, or the HIP error code, or -1 for a size out of range.
extern "C" int dora_calibrate_copy(const void* src, void* dst, size_t bytes, int blocks, int through, void* stream) {
  if (bytes == 0 || bytes % 16 != 0 || bytes > (size_t(1) << 30) || blocks < 1) return -1;
  const auto* s = static_cast<const u32x4*>(src);
  auto* d = static_cast<u32x4*>(dst);
  if (through)
    hipLaunchKernelGGL(copy_kernel<true>, dim3(blocks), dim3(256), 0, static_cast<hipStream_t>(stream), s, d, bytes / 16);
  else
    hipLaunchKernelGGL(copy_kernel<false>, dim3(blocks), dim3(256), 0, static_cast<hipStream_t>(stream), s, d, bytes / 16);
  return static_cast<int>(hipGetLastError());
}

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
