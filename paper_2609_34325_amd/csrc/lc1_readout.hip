// Readout input of a DINOv2 linear classifier on the packed, pruned tokens.
// DORA (arXiv 2609.34325), App. E.3 "Baseline implementations": the LC1
// readout joins the normalised CLS token with the mean of the normalised
// surviving visual tokens.  A segmented reduction over the packed buffer
// (Sec. 3.5 "Inference": one sequence per image between cu_seqlens entries),
// fused with the backbone's final LayerNorm, so each packed row is read once
// and only B x 2C values are written.
//
// One workgroup per image (16 waves; 8 for the widest rows).  Wave w takes
// rows r0 + w, r0 + w + 16, ..., two per step (one for wide rows), with the
// next step's rows in flight while it reduces the current ones.  Loads are
// unconditional from clamped, in-bounds addresses and the loop body is one
// basic block, so the compiler counts the loads in order instead of waiting
// for all of them; values past the sequence or the row are masked where they
// are used.  A lane holds up to VPL 16-byte pieces of a row; the row's mean
// and biased variance come from two wave reductions (DPP butterflies and row
// swaps; the variance from centred values).  CLS leaves the loop normalised,
// (x - mean) / sqrt(var + eps), into LDS; for the other rows each lane
// accumulates the same quantity.  The waves' sums meet in LDS in two rounds
// and are added in wave order (the result does not depend on timing); then
// gamma * sum / (n - 1) + beta is the mean of the normalised rows and
// gamma * cls + beta the normalised CLS.
//
// Small batches (a caller workspace given): the rows of an image are split
// into up to 8 contiguous parts, one workgroup each, so that about 256
// workgroups run; each writes its sum of normalised rows to the workspace and
// lc1_combine_kernel, launched next, adds the parts in order.  The launch
// boundary makes the sums visible: a last-workgroup-combines protocol needs
// an agent-scope release per workgroup, which writes back the die's whole L2
// and serialised the workgroups (55 ns each).
#include <algorithm>

#include "dora_internal.h"

namespace dora {
namespace {

constexpr int kLCCombine = 8;  // waves whose partial sums meet in LDS (LDS holds kLCCombine x C floats)
constexpr int kLCMaxRowBytes = 4096;  // 64 lanes x 4 pieces of 16 bytes
constexpr int kLCMaxSplit = 8;        // workgroups per image with a workspace
constexpr int32_t kLCMaxB = 1 << 24;  // images per call (B x kLCMaxSplit workgroups fit a grid)

struct LCParams {
  const uint4* x;      // packed rows
  const int32_t* cu;   // [B+1]
  const float* gamma;  // [C]
  const float* beta;   // [C]
  float eps;
  int32_t B, C, vpr;   // vpr: 16-byte pieces per row
  int64_t total;
  float* out;          // [B, 2C]
  int32_t* status;
  int32_t split;       // workgroups per image
  float* part;         // split > 1: [B, split, C] sums of the workgroups
};

template <bool BF16>
struct Piece;
template <>
struct Piece<true> {
  static constexpr int kElems = 8;
  __device__ static void unpack(uint4 v, float* f) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
};
template <>
struct Piece<false> {
  static constexpr int kElems = 4;
  __device__ static void unpack(uint4 v, float* f) {
    f[0] = __uint_as_float(v.x);
    f[1] = __uint_as_float(v.y);
    f[2] = __uint_as_float(v.z);
    f[3] = __uint_as_float(v.w);
  }
};

// Sum over the wave, every lane receiving the same value: butterflies inside
// each 16-lane row by DPP (quad permutes, half-row and row mirrors), then the
// row swaps v_permlane16_swap and v_permlane32_swap.  Each step adds two
// values that every lane of the pair sees in the same two operands, so all
// lanes agree bit for bit.
__device__ __forceinline__ float wave_total(float v) {
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x141, 0xF, 0xF, false));  // row_half_mirror
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x140, 0xF, 0xF, false));  // row_mirror
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto c = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(c[0]) + __uint_as_float(c[1]);
}

// Shape of the work of one workgroup for rows of VPL pieces of E values per
// lane: two rows per step on 16 waves, or one on 8 waves for the widest rows
// (within the register budget of the occupancy).
template <int VPL, int E>
struct Flight {
  static constexpr int kRows = VPL * E > 16 || VPL >= 4 ? 1 : 2;
  static constexpr int kWaves = VPL * E > 16 || VPL >= 4 ? 8 : 16;
};

template <int VPL, bool BF16>
__global__ __launch_bounds__((Flight<VPL, Piece<BF16>::kElems>::kWaves * 64)) void lc1_readout_kernel(LCParams p) {
  constexpr int E = Piece<BF16>::kElems;
  constexpr int R = Flight<VPL, E>::kRows;
  constexpr int kLCWaves = Flight<VPL, E>::kWaves;
  constexpr int kLCThreads = kLCWaves * 64;
  static_assert(kLCWaves == kLCCombine || kLCWaves == 2 * kLCCombine, "two combine rounds at most");
  extern __shared__ float s_acc[];  // [kLCCombine][C], then the normalised CLS row [C]
  float* s_cls = s_acc + kLCCombine * p.C;
  const int b = blockIdx.x / p.split, part_id = blockIdx.x - b * p.split;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lo = p.cu[b], hi = p.cu[b + 1];
  if (!(lo >= 0 && hi > lo && hi <= p.total && (b > 0 || lo == 0))) {
    if (threadIdx.x == 0 && part_id == 0) {
      atomicOr(p.status, DORA_DEV_CU_SEQLENS);
      for (int c = 0; c < 2 * p.C; ++c) p.out[static_cast<int64_t>(b) * 2 * p.C + c] = __builtin_nanf("");
    }
    return;
  }
  // This workgroup's rows [rlo, rhi) of the image; CLS (row lo) falls in part 0.
  const int per_part = (hi - lo + p.split - 1) / p.split;
  const int rlo = min(hi, lo + part_id * per_part), rhi = min(hi, rlo + per_part);
  // Per lane: the sum over this wave's visual rows of (x - mean) * rstd for
  // its channels; gamma and beta are applied once at the end (the affine map
  // commutes with the mean).
  float acc[VPL][E];
#pragma unroll
  for (int i = 0; i < VPL; ++i)
#pragma unroll
    for (int e = 0; e < E; ++e) acc[i][e] = 0.0f;
  const float inv_c = 1.0f / static_cast<float>(p.C);
  // Wave w takes rows lo + w + j * kLCWaves, R of them per step, with two
  // buffers: the next step's rows are in flight while the current ones are
  // reduced.  Loads are unconditional from clamped (in-bounds) addresses, so
  // the compiler can count them in order instead of waiting for all of them;
  // values past the sequence or the row are masked to zero where they are used.
  constexpr int kStep = R * kLCWaves;
  // An empty range (rlo == rhi == hi) reads the image's last row, masked.
  const int last_row = min(max(rhi, rlo + 1), hi) - 1, last_vec = p.vpr - 1;
  auto load = [&](int r0, uint4 (&dst)[R][VPL]) {
#pragma unroll
    for (int q = 0; q < R; ++q)
#pragma unroll
      for (int i = 0; i < VPL; ++i) {
        const int r = min(r0 + q * kLCWaves, last_row), v = min(lane + 64 * i, last_vec);
        dst[q][i] = p.x[static_cast<int64_t>(r) * p.vpr + v];
      }
  };
  auto process = [&](int r0, const uint4 (&src)[R][VPL]) {
    float x[R][VPL][E], s[R], ss[R];
#pragma unroll
    for (int q = 0; q < R; ++q) {
      s[q] = 0.0f;
      const bool row_in = r0 + q * kLCWaves < rhi;
#pragma unroll
      for (int i = 0; i < VPL; ++i) {
        const uint32_t mk = (row_in && lane + 64 * i < p.vpr) ? ~0u : 0u;
        const uint4 t = src[q][i];
        Piece<BF16>::unpack(make_uint4(t.x & mk, t.y & mk, t.z & mk, t.w & mk), x[q][i]);
#pragma unroll
        for (int e = 0; e < E; ++e) s[q] += x[q][i][e];
      }
    }
#pragma unroll
    for (int q = 0; q < R; ++q) s[q] = wave_total(s[q]);
#pragma unroll
    for (int q = 0; q < R; ++q) {
      const float mu = s[q] * inv_c;
      ss[q] = 0.0f;
#pragma unroll
      for (int i = 0; i < VPL; ++i) {
        const float keep = lane + 64 * i < p.vpr ? 1.0f : 0.0f;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const float d = (x[q][i][e] - mu) * keep;
          x[q][i][e] = d;
          ss[q] += d * d;
        }
      }
    }
#pragma unroll
    for (int q = 0; q < R; ++q) ss[q] = wave_total(ss[q]);
#pragma unroll
    for (int q = 0; q < R; ++q) {
      // a row past the sequence has d = 0; its scale is kept finite (1) so it
      // adds exactly nothing, without a branch
      const int r = r0 + q * kLCWaves;
      const float pad = r < rhi ? 0.0f : 1.0f;
      const float rstd = 1.0f / sqrtf(ss[q] * inv_c + p.eps + pad);
      if (r == lo) {  // CLS: kept in LDS, gamma and beta applied at the end
#pragma unroll
        for (int i = 0; i < VPL; ++i) {
          const int v = lane + 64 * i;
          if (v < p.vpr)
#pragma unroll
            for (int e = 0; e < E; ++e) s_cls[v * E + e] = x[q][i][e] * rstd;
        }
      } else {
#pragma unroll
        for (int i = 0; i < VPL; ++i)
#pragma unroll
          for (int e = 0; e < E; ++e) acc[i][e] += x[q][i][e] * rstd;
      }
    }
  };
  uint4 buf_a[R][VPL], buf_b[R][VPL];
  int r0 = rlo + wave;
  load(r0, buf_a);
  // Whole rounds of two steps, one basic block (so no load is moved next to
  // its use); a step past the sequence sees masked rows and adds nothing.
  for (; r0 < rhi; r0 += 2 * kStep) {
    load(r0 + kStep, buf_b);
    process(r0, buf_a);
    load(r0 + 2 * kStep, buf_a);
    process(r0 + kStep, buf_b);
  }
  // Waves kLCCombine.. hand their sums to waves 0.., which add them to their
  // own; the kLCCombine sums are then added in wave order.
  float* mine = s_acc + (wave % kLCCombine) * p.C;
  if (wave >= kLCCombine) {
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
      const int v = lane + 64 * i;
      if (v < p.vpr)
#pragma unroll
        for (int e = 0; e < E; ++e) mine[v * E + e] = acc[i][e];
    }
  }
  __syncthreads();
  if (wave < kLCCombine) {
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
      const int v = lane + 64 * i;
      if (v < p.vpr)
#pragma unroll
        for (int e = 0; e < E; ++e) mine[v * E + e] = (kLCWaves > kLCCombine ? mine[v * E + e] : 0.0f) + acc[i][e];
    }
  }
  __syncthreads();
  const float inv_n = 1.0f / static_cast<float>(hi - lo - 1);
  float* o = p.out + static_cast<int64_t>(b) * 2 * p.C + p.C;
  if (p.split == 1) {
    for (int c = threadIdx.x; c < p.C; c += kLCThreads) {
      float t = 0.0f;
#pragma unroll
      for (int w = 0; w < kLCCombine; ++w) t += s_acc[w * p.C + c];
      const float gc = p.gamma[c], bc = p.beta[c];
      o[c] = hi - lo > 1 ? t * inv_n * gc + bc : __builtin_nanf("");
      o[c - p.C] = s_cls[c] * gc + bc;
    }
    return;
  }
  // Several workgroups per image: each writes its sum, part 0 the CLS half;
  // lc1_combine_kernel, the next launch, adds the sums.
  float* mine_part = p.part + (static_cast<int64_t>(b) * p.split + part_id) * p.C;
  for (int c = threadIdx.x; c < p.C; c += kLCThreads) {
    float t = 0.0f;
#pragma unroll
    for (int w = 0; w < kLCCombine; ++w) t += s_acc[w * p.C + c];
    mine_part[c] = t;
    if (part_id == 0) o[c - p.C] = s_cls[c] * p.gamma[c] + p.beta[c];
  }
}

// Mean half of the split readout: the parts' sums of image b added in part
// order (the result does not depend on timing), scaled, gamma and beta.  An
// invalid sequence keeps the NaN row the first launch wrote.
__global__ __launch_bounds__(256) void lc1_combine_kernel(LCParams p) {
  const int b = blockIdx.x, c = blockIdx.y * 256 + threadIdx.x;
  const int lo = p.cu[b], hi = p.cu[b + 1];
  if (c >= p.C || !(lo >= 0 && hi > lo && hi <= p.total && (b > 0 || lo == 0))) return;
  // One channel per thread; the loads of all parts are issued together
  // (parts past split re-read the last one and add zero), and the empty asm
  // keeps the compiler from moving each load into a branch of its own.
  const float* parts = p.part + static_cast<int64_t>(b) * p.split * p.C + c;
  float v[kLCMaxSplit];
#pragma unroll
  for (int q = 0; q < kLCMaxSplit; ++q) v[q] = parts[static_cast<int64_t>(min(q, p.split - 1)) * p.C];
#pragma unroll
  for (int q = 0; q < kLCMaxSplit; ++q) asm volatile("" : "+v"(v[q]));
  float t = 0.0f;
#pragma unroll
  for (int q = 0; q < kLCMaxSplit; ++q) t += q < p.split ? v[q] : 0.0f;
  const float inv_n = 1.0f / static_cast<float>(hi - lo - 1);
  p.out[static_cast<int64_t>(b) * 2 * p.C + p.C + c] = hi - lo > 1 ? t * inv_n * p.gamma[c] + p.beta[c]
                                                                  : __builtin_nanf("");
}

template <int VPL, bool BF16>
hipError_t launch_lc1(const LCParams& p, hipStream_t stream) {
  const size_t lds = static_cast<size_t>(kLCCombine + 1) * p.C * sizeof(float);
  constexpr int threads = Flight<VPL, Piece<BF16>::kElems>::kWaves * 64;
  hipLaunchKernelGGL((lc1_readout_kernel<VPL, BF16>), dim3(p.B * p.split), dim3(threads), lds, stream, p);
  if (p.split > 1) hipLaunchKernelGGL(lc1_combine_kernel, dim3(p.B, (p.C + 255) / 256), dim3(256), 0, stream, p);
  return hipGetLastError();
}


}  // namespace
}  // namespace dora

extern "C" size_t dora_lc1_readout_workspace_size(int32_t B, int32_t C) {
  using namespace dora;
  if (B < 1 || C < 1 || B > kLCMaxB || C > kLCMaxRowBytes / 2) return 0;
  return static_cast<size_t>(B) * kLCMaxSplit * C * sizeof(float);  // [B, kLCMaxSplit, C] partial sums
}

extern "C" int dora_lc1_readout(const void* x, const int32_t* cu_seqlens, int64_t total, int32_t B, int32_t C,
                                dora_dtype dtype, const float* gamma, const float* beta, float eps, float* out,
                                void* workspace, size_t workspace_bytes, int32_t* dev_status, void* stream) {
  using namespace dora;
  if (!x || !cu_seqlens || !gamma || !beta || !out || !dev_status) return DORA_ERR_NULL;
  if (dtype != DORA_BF16 && dtype != DORA_F32) return DORA_ERR_DTYPE;
  const int elt = dtype == DORA_BF16 ? 2 : 4;
  if (B < 1 || B > kLCMaxB || C < 1 || total < 1 || total > 0x7FFFFFFF || !(eps >= 0.0f))
    return DORA_ERR_SHAPE;
  if ((static_cast<int64_t>(C) * elt) % 16 != 0 || reinterpret_cast<uintptr_t>(x) & 15u) return DORA_ERR_ALIGN;
  if (static_cast<int64_t>(C) * elt > kLCMaxRowBytes) return DORA_ERR_UNSUPPORTED;
  LCParams p{static_cast<const uint4*>(x), cu_seqlens, gamma, beta, eps, B, C, C * elt / 16, total, out,
             dev_status, 1, nullptr};
  if (workspace) {
    if (reinterpret_cast<uintptr_t>(workspace) & 255u) return DORA_ERR_ALIGN;
    if (workspace_bytes < dora_lc1_readout_workspace_size(B, C)) return DORA_ERR_WORKSPACE;
    // About 256 workgroups in all, each with at least ~64 rows on average.
    const int64_t by_grid = (256 + B - 1) / B, by_rows = total / (64 * static_cast<int64_t>(B));
    p.split = static_cast<int32_t>(std::max<int64_t>(1, std::min<int64_t>({by_grid, by_rows, kLCMaxSplit})));
    p.part = static_cast<float*>(workspace);
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int vpl = (p.vpr + 63) / 64;
  hipError_t err;
  if (dtype == DORA_BF16) {
    err = vpl <= 1 ? launch_lc1<1, true>(p, st) : vpl <= 2 ? launch_lc1<2, true>(p, st) : launch_lc1<4, true>(p, st);
  } else {
    err = vpl <= 1 ? launch_lc1<1, false>(p, st) : vpl <= 2 ? launch_lc1<2, false>(p, st)
                                                          : launch_lc1<4, false>(p, st);
  }
  return err == hipSuccess ? DORA_OK : DORA_ERR_HIP;
}
