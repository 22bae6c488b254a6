// Readout input of a DINOv2 linear classifier on the packed, pruned tokens.
// DORA (arXiv 2609.34325), App. E.3 "Baseline implementations": the LC1
// readout joins the normalised CLS token with the mean of the normalised
// surviving visual tokens.  A segmented reduction over the packed buffer
// (Sec. 3.5 "Inference": one sequence per image between cu_seqlens entries),
// fused with the backbone's final LayerNorm, so each packed row is read once
// and only B x 2C values are written.
//
// One workgroup of 8 waves per image.  A row of P 16-byte pieces is held by
// a group of L = 16, 32 or 64 lanes, up to 4 pieces a lane, the shape that
// leaves the fewest lanes idle (768 bf16 channels: 32 lanes of 3 pieces, two
// rows per wave).  The groups are row slots taking every (slots)-th row, with
// the next row in flight while they reduce the current one.  Loads are
// unconditional from clamped, in-bounds addresses; a row past the end gets
// weight 0.  A row's sum comes from bf16 dot products with (1, 1) on the
// packed values, its mean and biased variance (from centred values) from
// group reductions (DPP butterflies and row swaps), and 1 / sqrt(var + eps)
// from the hardware reciprocal square root.  CLS is normalised apart, into
// LDS; for the other rows each lane accumulates (x - mean) / sqrt(var + eps).
// The groups' sums are merged by row swaps and the waves' sums meet in LDS
// in two rounds, added in wave order (the result does not depend on timing);
// then gamma * sum / (n - 1) + beta is the mean of the normalised rows and
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

constexpr int kLCCombine = 4;  // waves whose partial sums meet in LDS (LDS holds kLCCombine x C floats)
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

// Sum over a group of L lanes (16, 32 or 64), every lane of the group
// receiving the same value: butterflies inside each 16-lane row by DPP
// (quad permutes, half-row and row mirrors), then for wider groups the row
// swaps v_permlane16_swap and v_permlane32_swap.  Each step adds two values
// that every lane of the pair sees in the same two operands, so all lanes of
// a group agree bit for bit.
template <int L>
__device__ __forceinline__ float group_total(float v) {
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x141, 0xF, 0xF, false));  // row_half_mirror
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x140, 0xF, 0xF, false));  // row_mirror
  if constexpr (L >= 32) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  }
  if constexpr (L >= 64) {
    const auto c = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(c[0]) + __uint_as_float(c[1]);
  }
  return v;
}

// Sum of the value a lane holds and the values the lanes at the same place
// in the wave's other L-lane groups hold (the same channels of other rows).
template <int L>
__device__ __forceinline__ float merge_groups(float v) {
  if constexpr (L <= 16) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  }
  if constexpr (L <= 32) {
    const auto c = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(c[0]) + __uint_as_float(c[1]);
  }
  return v;
}

constexpr int kLCWaves = 8;
constexpr int kLCThreads = kLCWaves * 64;
static_assert(kLCWaves == 2 * kLCCombine, "two combine rounds");
static_assert(kLCMaxRowBytes / 2 <= 4 * kLCThreads, "every quad of output channels has a thread");

// Partial-sum buffers of C = P * E floats in LDS hold 16-byte quads: quad h
// (elements 4h .. 4h + 3) of piece v at quad index h * P + v.  The lanes of a
// group, which hold consecutive pieces, store and load consecutive quads
// (16-byte accesses without bank conflicts).
__device__ __forceinline__ float4* lds_quad(float* base, int P, int v, int h) {
  return reinterpret_cast<float4*>(base) + (h * P + v);
}

// Sum of the 2 E bf16 or E fp32 values of a piece, before unpacking: one
// dot product with (1, 1) per pair of bf16 values.
template <bool BF16>
__device__ __forceinline__ float piece_sum(uint4 v, float s) {
  if constexpr (BF16) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 one = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, v.x), one, s, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, v.y), one, s, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, v.z), one, s, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, v.w), one, s, false);
    return s;
  } else {
    return s + __uint_as_float(v.x) + __uint_as_float(v.y) + __uint_as_float(v.z) + __uint_as_float(v.w);
  }
}

// One workgroup per image part (8 waves).  A row of P 16-byte pieces is held
// by a group of L lanes, VPL pieces a lane (L * VPL >= P, chosen by the host
// to leave few lanes idle: 96-piece rows, DeiT-B and DINOv2-B in bf16, are two
// rows per wave on 32-lane groups with three pieces a lane); PAD says that
// some lanes' last piece lies past the row's end.  The 64 / L groups of the
// 8 waves are the row slots: slot g takes rows r0 + g, r0 + g + slots, ...,
// with its next row in flight while it reduces the current one.
template <int L, int VPL, bool PAD, bool BF16>
__global__ __launch_bounds__(kLCThreads) void lc1_readout_kernel(LCParams p) {
  constexpr int E = Piece<BF16>::kElems;
  constexpr int kGroups = 64 / L;
  constexpr int kSlots = kLCWaves * kGroups;  // rows per step
  extern __shared__ float s_acc[];  // [kLCCombine][C], then the normalised CLS row [C]
  float* s_cls = s_acc + kLCCombine * p.C;
  const int b = blockIdx.x / p.split, part_id = blockIdx.x - b * p.split;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = lane / L, t = lane % L;
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
  const float inv_c = 1.0f / static_cast<float>(p.C);
  // Only a lane's last piece can lie past the row's end (L * (VPL - 1) < P):
  // it reads the row's last piece and is masked to zero (PAD only).
  const bool last_ok = !PAD || t + L * (VPL - 1) < p.vpr;
  const uint32_t last_mask = last_ok ? ~0u : 0u;
  const int last_piece = PAD ? min(t + L * (VPL - 1), p.vpr - 1) : t + L * (VPL - 1);
  // Loads are unconditional from clamped (in-bounds) addresses, so the
  // compiler counts them in order instead of waiting for all of them.  A row
  // past this part's end reads the part's last row and is given weight 0.  An
  // empty part (rlo == rhi == hi) reads the image's last row.
  const int last_row = min(max(rhi, rlo + 1), hi) - 1;
  auto load = [&](int r, uint4 (&dst)[VPL]) {
    const uint4* row = p.x + static_cast<int64_t>(min(r, last_row)) * p.vpr;
#pragma unroll
    for (int i = 0; i < VPL; ++i) dst[i] = row[i + 1 < VPL ? t + L * i : last_piece];
  };
  // (x - mean) of the row's values this lane holds, and the row's
  // 1 / sqrt(var + eps) (biased variance from the centred values).
  auto normalise = [&](uint4 (&src)[VPL], float (&d)[VPL][E]) {
    if constexpr (PAD) {
      uint4& w = src[VPL - 1];
      w = make_uint4(w.x & last_mask, w.y & last_mask, w.z & last_mask, w.w & last_mask);
    }
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < VPL; ++i) s = piece_sum<BF16>(src[i], s);
    const float mu = group_total<L>(s) * inv_c;
    float ss = 0.0f;
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
      Piece<BF16>::unpack(src[i], d[i]);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        d[i][e] -= mu;
        if (!PAD || i + 1 < VPL) ss += d[i][e] * d[i][e];
      }
    }
    if constexpr (PAD) {
      float sl = 0.0f;
#pragma unroll
      for (int e = 0; e < E; ++e) sl += d[VPL - 1][e] * d[VPL - 1][e];
      ss += last_ok ? sl : 0.0f;
    }
    return __builtin_amdgcn_rsqf(group_total<L>(ss) * inv_c + p.eps);
  };
  // Per lane: the sum over this slot's visual rows of (x - mean) * rstd for
  // its channels; gamma and beta are applied once at the end (the affine map
  // commutes with the mean).
  float acc[VPL][E];
#pragma unroll
  for (int i = 0; i < VPL; ++i)
#pragma unroll
    for (int e = 0; e < E; ++e) acc[i][e] = 0.0f;
  auto process = [&](int r, uint4 (&src)[VPL]) {
    float d[VPL][E];
    const float rs = normalise(src, d);
    const float w = r < rhi ? rs : 0.0f;
#pragma unroll
    for (int i = 0; i < VPL; ++i)
#pragma unroll
      for (int e = 0; e < E; ++e) acc[i][e] += d[i][e] * w;
  };
  // The loop takes the visual rows, from lo + 1 in part 0.
  const int r0 = part_id == 0 ? lo + 1 : rlo;
  // Rounds of two steps; the loop runs on the wave's first row (uniform), and
  // the second step of a round is skipped when no row of the wave is left.
  // The empty asm statements, memory barriers to the compiler, keep loads
  // where they are written instead of next to their use.
  uint4 buf_a[VPL], buf_b[VPL];
  int rw = r0 + wave * kGroups;
  load(rw + grp, buf_a);
  // gamma and beta of this thread's four output channels 4u .. 4u + 3
  // (u = thread index; C is a multiple of 4), loaded now so that their
  // latency overlaps the rows' loads.
  const int u = threadIdx.x, cq = min(4 * u, p.C - 4);
  float gam[4], bet[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    gam[k] = p.gamma[cq + k];
    bet[k] = p.beta[cq + k];
  }
  asm volatile("" ::: "memory");
  // CLS (part 0): normalised by wave 0 into LDS, its loads issued after the
  // loop's first ones.
  if (part_id == 0 && wave == 0) {
    uint4 c[VPL];
    load(lo, c);
    float d[VPL][E];
    const float rs = normalise(c, d);
    if (grp == 0) {
#pragma unroll
      for (int i = 0; i < VPL; ++i)
        if (i + 1 < VPL || last_ok)
#pragma unroll
          for (int h = 0; h < E / 4; ++h)
            *lds_quad(s_cls, p.vpr, t + L * i, h) =
                make_float4(d[i][4 * h] * rs, d[i][4 * h + 1] * rs, d[i][4 * h + 2] * rs, d[i][4 * h + 3] * rs);
    }
  }
  for (; rw < rhi; rw += 2 * kSlots) {
    load(rw + grp + kSlots, buf_b);
    asm volatile("" ::: "memory");
    process(rw + grp, buf_a);
    load(rw + grp + 2 * kSlots, buf_a);
    if (rw + kSlots < rhi) process(rw + grp + kSlots, buf_b);
  }
  // The wave's groups hold the same channels of different rows: merge them,
  // then the waves' sums meet in LDS in two rounds and are added in wave
  // order (the result does not depend on timing).
#pragma unroll
  for (int i = 0; i < VPL; ++i)
#pragma unroll
    for (int e = 0; e < E; ++e) acc[i][e] = merge_groups<L>(acc[i][e]);
  float* mine = s_acc + (wave % kLCCombine) * p.C;
  if (wave >= kLCCombine && grp == 0) {
#pragma unroll
    for (int i = 0; i < VPL; ++i)
      if (i + 1 < VPL || last_ok)
#pragma unroll
        for (int h = 0; h < E / 4; ++h)
          *lds_quad(mine, p.vpr, t + L * i, h) =
              make_float4(acc[i][4 * h], acc[i][4 * h + 1], acc[i][4 * h + 2], acc[i][4 * h + 3]);
  }
  __syncthreads();
  if (wave < kLCCombine && grp == 0) {
#pragma unroll
    for (int i = 0; i < VPL; ++i)
      if (i + 1 < VPL || last_ok)
#pragma unroll
        for (int h = 0; h < E / 4; ++h) {
          float4* q = lds_quad(mine, p.vpr, t + L * i, h);
          const float4 o = *q;
          *q = make_float4(o.x + acc[i][4 * h], o.y + acc[i][4 * h + 1], o.z + acc[i][4 * h + 2],
                           o.w + acc[i][4 * h + 3]);
        }
  }
  __syncthreads();
  if (4 * u >= p.C) return;
  // Quad u holds channels 4u .. 4u + 3: quad h of piece v.
  const int v = 4 * u / E, h = (4 * u - v * E) / 4;
  float4 tsum = *lds_quad(s_acc, p.vpr, v, h);
#pragma unroll
  for (int w = 1; w < kLCCombine; ++w) {
    const float4 a = *lds_quad(s_acc + w * p.C, p.vpr, v, h);
    tsum = make_float4(tsum.x + a.x, tsum.y + a.y, tsum.z + a.z, tsum.w + a.w);
  }
  const float ts[4] = {tsum.x, tsum.y, tsum.z, tsum.w};
  const float4 cl = *lds_quad(s_cls, p.vpr, v, h);
  const float cls[4] = {cl.x, cl.y, cl.z, cl.w};
  float* o = p.out + static_cast<int64_t>(b) * 2 * p.C + 4 * u;  // CLS half; the mean half at + C
  if (p.split == 1) {
    const float inv_n = 1.0f / static_cast<float>(hi - lo - 1);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      o[k] = cls[k] * gam[k] + bet[k];
      o[p.C + k] = hi - lo > 1 ? ts[k] * inv_n * gam[k] + bet[k] : __builtin_nanf("");
    }
    return;
  }
  // Several workgroups per image: each writes its sum, part 0 the CLS half;
  // lc1_combine_kernel, the next launch, adds the sums.
  float* mine_part = p.part + (static_cast<int64_t>(b) * p.split + part_id) * p.C + 4 * u;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    mine_part[k] = ts[k];
    if (part_id == 0) o[k] = cls[k] * gam[k] + bet[k];
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

template <int L, int VPL, bool BF16>
hipError_t launch_lc1(const LCParams& p, hipStream_t stream) {
  const size_t lds = static_cast<size_t>(kLCCombine + 1) * p.C * sizeof(float);
  auto kernel = L * VPL == p.vpr ? lc1_readout_kernel<L, VPL, false, BF16> : lc1_readout_kernel<L, VPL, true, BF16>;
  hipLaunchKernelGGL(kernel, dim3(p.B * p.split), dim3(kLCThreads), lds, stream, p);
  if (p.split > 1) hipLaunchKernelGGL(lc1_combine_kernel, dim3(p.B, (p.C + 255) / 256), dim3(256), 0, stream, p);
  return hipGetLastError();
}

// Lanes per row group and pieces per lane for rows of P pieces: the fewest
// idle slots (L * VPL - P), then the widest group; at most 4 pieces a lane.
void lc1_shape(int P, int* L_out, int* vpl_out) {
  int best_l = 64, best_v = (P + 63) / 64, best_w = 1 << 30;
  for (int L : {64, 32, 16}) {
    const int v = (P + L - 1) / L;
    if (v > 4) continue;
    const int waste = L * v - P;
    if (waste < best_w) {
      best_w = waste;
      best_l = L;
      best_v = v;
    }
  }
  *L_out = best_l;
  *vpl_out = best_v;
}

template <bool BF16>
hipError_t launch_lc1_shape(const LCParams& p, hipStream_t st) {
  int L, v;
  lc1_shape(p.vpr, &L, &v);
#define DORA_LC1_CASE(LL, VV) \
  if (L == LL && v == VV) return launch_lc1<LL, VV, BF16>(p, st);
  DORA_LC1_CASE(64, 1) DORA_LC1_CASE(64, 2) DORA_LC1_CASE(64, 3) DORA_LC1_CASE(64, 4)
  DORA_LC1_CASE(32, 1) DORA_LC1_CASE(32, 2) DORA_LC1_CASE(32, 3) DORA_LC1_CASE(32, 4)
  DORA_LC1_CASE(16, 1) DORA_LC1_CASE(16, 2) DORA_LC1_CASE(16, 3) DORA_LC1_CASE(16, 4)
#undef DORA_LC1_CASE
  return hipErrorInvalidValue;
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
  const hipError_t err = dtype == DORA_BF16 ? launch_lc1_shape<true>(p, st) : launch_lc1_shape<false>(p, st);
  return err == hipSuccess ? DORA_OK : DORA_ERR_HIP;
}
