// Variable-length multi-head attention over the packed buffer.
// DORA (arXiv 2609.34325), Sec. 3.5 "Inference" and App. E.4: survivors of
// all images are packed with explicit sequence boundaries and processed by
// exact softmax attention that never crosses a boundary (no mask beyond the
// boundaries, no bias, no token-size term).
//
// Work decomposition (persistent, queue-driven):
//   plan     one workgroup builds the list of (sequence, head, 128-query tile)
//            items, sequences sorted by decreasing length (longest first), and
//            resets the queue counters.
//   execute  #CU x occupancy persistent workgroups; each takes item tickets
//            from an atomic counter until the list is drained; the last
//            workgroup to leave resets the counters so the plan can be
//            executed again (e.g. by the next layer).
//
// Per item, 4 waves x 32 queries.  K/V are streamed through LDS in blocks of
// 64 keys (K row-major, V transposed so both MFMA operands read contiguous
// runs).  S^T = K Q^T is computed with v_mfma_f32_16x16x32_bf16 so each lane
// owns one query column and the softmax reductions over keys stay mostly
// in-lane; the online softmax runs in fp32 with exp2 and a pre-folded
// scale*log2(e); P is rounded to bf16 and O^T += V^T P^T reuses the MFMA
// output registers of S^T directly as the B operand (the key order inside a
// 32-key step is permuted identically on both operands).
#include <limits.h>
#include <math.h>

#include "dora_internal.h"

namespace dora {
namespace {

constexpr int kD = 64;
constexpr int kBlockKeys = 64;
constexpr int kWaves = 4;
constexpr int kQPerWave = 32;
static_assert(kWaves * kQPerWave == kAttnQTile, "tile size");
constexpr int kThreads = kWaves * 64;
constexpr int kPlanThreads = 1024;
constexpr int kPlanBins = 1024;
constexpr float kLog2e = 1.4426950408889634f;

struct PlanParams {
  const int32_t* cu;
  int32_t B, H, max_seqlen;
  int64_t total;
  AttnPlanHeader* hdr;
  int32_t* order;
  int32_t* item_base;
  int2* items;
  int64_t max_items;
  int32_t* status;
};

struct AttnParams {
  const void* q;
  const void* k;
  const void* v;
  void* out;
  const int32_t* cu;
  int32_t B, H, max_seqlen;
  int64_t total;
  float scale_log2;  // softmax_scale * log2(e)
  AttnPlanHeader* hdr;
  const int2* items;
  int32_t max_items;  // capacity of items[] in this workspace
  int32_t* status;
};

__device__ __forceinline__ int block_exclusive_scan(int v, int* tmp, int* total_out) {
  // kPlanThreads-wide exclusive scan through LDS (Hillis-Steele).
  const int tid = threadIdx.x;
  tmp[tid] = v;
  __syncthreads();
  for (int off = 1; off < kPlanThreads; off <<= 1) {
    const int add = tid >= off ? tmp[tid - off] : 0;
    __syncthreads();
    tmp[tid] += add;
    __syncthreads();
  }
  const int incl = tmp[tid];
  *total_out = tmp[kPlanThreads - 1];
  __syncthreads();
  return incl - v;
}

__global__ __launch_bounds__(kPlanThreads) void attn_plan_kernel(PlanParams p) {
  __shared__ int hist[kPlanBins];
  __shared__ int scan_tmp[kPlanThreads];
  __shared__ int s_bad;
  const int tid = threadIdx.x;
  int shift = 0;
  while ((p.max_seqlen >> shift) >= kPlanBins) ++shift;

  for (int i = tid; i < kPlanBins; i += kPlanThreads) hist[i] = 0;
  if (tid == 0) s_bad = (p.cu[0] != 0);
  __syncthreads();

  // Validate the offsets and histogram the lengths.
  for (int b = tid; b < p.B; b += kPlanThreads) {
    const long long a = p.cu[b], e = p.cu[b + 1];
    const long long len = e - a;
    if (a < 0 || e > p.total || len < 0 || len > p.max_seqlen) {
      s_bad = 1;
    } else {
      atomicAdd(&hist[static_cast<int>(len) >> shift], 1);
    }
  }
  __syncthreads();
  if (s_bad) {
    if (tid == 0) {
      atomicOr(p.status, DORA_DEV_CU_SEQLENS);
      p.hdr->n_items = 0;
      p.hdr->counter = 0;
      p.hdr->exit_count = 0;
      p.hdr->B = p.B;
      p.hdr->H = p.H;
      p.hdr->max_seqlen = p.max_seqlen;
      p.hdr->q_tile = kAttnQTile;
      p.hdr->total = p.total;
      p.hdr->magic = kPlanMagic;
    }
    return;
  }

  // Start position of each length bin in decreasing-length order.
  {
    int sum_total;
    const int bin = kPlanBins - 1 - tid;  // thread t scans bin (top - t)
    const int cnt = hist[bin];
    __syncthreads();
    const int start = block_exclusive_scan(cnt, scan_tmp, &sum_total);
    hist[bin] = start;
    __syncthreads();
  }
  for (int b = tid; b < p.B; b += kPlanThreads) {
    const int len = p.cu[b + 1] - p.cu[b];
    const int pos = atomicAdd(&hist[len >> shift], 1);
    p.order[pos] = b;
  }
  __threadfence_block();
  __syncthreads();

  // Item offsets per sorted position, then the items themselves.
  int carry = 0;
  for (int base = 0; base < p.B; base += kPlanThreads) {
    const int pos = base + tid;
    int cnt = 0;
    if (pos < p.B) {
      const int b = p.order[pos];
      const int len = p.cu[b + 1] - p.cu[b];
      cnt = p.H * ((len + kAttnQTile - 1) / kAttnQTile);
    }
    int chunk_total;
    const int off = block_exclusive_scan(cnt, scan_tmp, &chunk_total);
    if (pos < p.B) {
      p.item_base[pos] = carry + off;
      const int b = p.order[pos];
      const int len = p.cu[b + 1] - p.cu[b];
      const int tiles = (len + kAttnQTile - 1) / kAttnQTile;
      int2* dst = p.items + carry + off;
      for (int h = 0; h < p.H; ++h)
        for (int t = 0; t < tiles; ++t) dst[h * tiles + t] = make_int2(b, (h << 16) | t);
    }
    carry += chunk_total;
  }
  if (tid == 0) {
    p.item_base[p.B] = carry;
    p.hdr->n_items = carry;
    p.hdr->counter = 0;
    p.hdr->exit_count = 0;
    p.hdr->B = p.B;
    p.hdr->H = p.H;
    p.hdr->max_seqlen = p.max_seqlen;
    p.hdr->q_tile = kAttnQTile;
    p.hdr->total = p.total;
    p.hdr->magic = kPlanMagic;
  }
}

__device__ __forceinline__ bool plan_matches(const AttnParams& p) {
  const AttnPlanHeader* h = p.hdr;
  return h->magic == kPlanMagic && h->B == p.B && h->H == p.H && h->max_seqlen == p.max_seqlen &&
         h->q_tile == kAttnQTile && h->total == p.total;
}

__device__ __forceinline__ void leave_queue(AttnPlanHeader* hdr) {
  // The last workgroup out resets the counters for the next execute.
  if (threadIdx.x == 0) {
    __threadfence();
    const int done = atomicAdd(&hdr->exit_count, 1);
    if (done == static_cast<int>(gridDim.x) - 1) {
      atomicExch(&hdr->counter, 0);
      atomicExch(&hdr->exit_count, 0);
    }
  }
}

__device__ __forceinline__ bool item_bounds(const AttnParams& p, int b, int h, int tile,
                                            long long* seq0, int* len) {
  if (b < 0 || b >= p.B || h < 0 || h >= p.H) return false;
  const long long a = p.cu[b], e = p.cu[b + 1];
  if (a < 0 || e > p.total || e - a < 0 || e - a > p.max_seqlen) return false;
  *seq0 = a;
  *len = static_cast<int>(e - a);
  return static_cast<long long>(tile) * kAttnQTile < e - a;
}

// ---------------------------------------------------------------------------
// bf16 inputs, v_mfma_f32_16x16x32_bf16.
//
// MFMA 16x16x32 operand layout (lane l, g = l / 16, c = l % 16):
//   A[16 x 32]: lane holds row c, k = 8g .. 8g+7
//   B[32 x 16]: lane holds column c, k = 8g .. 8g+7
//   D[16 x 16]: lane holds column c, rows 4g .. 4g+3
// ---------------------------------------------------------------------------
constexpr int kKStride = kD + 8;          // bf16 elements per K row in LDS
constexpr int kVStride = kBlockKeys + 8;  // bf16 elements per V^T row in LDS

__global__ __launch_bounds__(kThreads) void attn_fwd_bf16_kernel(AttnParams p) {
  __shared__ __attribute__((aligned(16))) uint16_t Ks[kBlockKeys * kKStride];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[kD * kVStride];
  __shared__ int s_ticket;

  if (!plan_matches(p)) {
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(p.status, DORA_DEV_PLAN);
    return;
  }
  const int n_items = min(p.hdr->n_items, p.max_items);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int c16 = lane & 15;
  const int g = lane >> 4;
  const uint16_t* Q = static_cast<const uint16_t*>(p.q);
  const uint16_t* K = static_cast<const uint16_t*>(p.k);
  const uint16_t* V = static_cast<const uint16_t*>(p.v);
  uint16_t* O = static_cast<uint16_t*>(p.out);
  const long long row_elems = static_cast<long long>(p.H) * kD;

  for (;;) {
    if (tid == 0) s_ticket = atomicAdd(&p.hdr->counter, 1);
    __syncthreads();
    const int ticket = s_ticket;
    if (ticket >= n_items) break;
    const int2 item = p.items[ticket];
    const int b = item.x, h = item.y >> 16, tile = item.y & 0xFFFF;
    long long seq0;
    int len;
    if (!item_bounds(p, b, h, tile, &seq0, &len)) {
      if (tid == 0) atomicOr(p.status, DORA_DEV_CU_SEQLENS);
      __syncthreads();
      continue;
    }
    const int q0 = tile * kAttnQTile + wave * kQPerWave;
    const bool active = q0 < len;

    // Q^T operands (B side of S^T = K Q^T): lane holds query c16, dims 8g..8g+7 (+32).
    bf16x8 qf[2][2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int qi = q0 + 16 * j + c16;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        if (qi < len) {
          qf[j][ks] = *reinterpret_cast<const bf16x8*>(Q + (seq0 + qi) * row_elems + h * kD + ks * 32 + g * 8);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) qf[j][ks][e] = static_cast<__bf16>(0.0f);
        }
      }
    }

    floatx4 o[2][4];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) o[j][dt] = floatx4{0.f, 0.f, 0.f, 0.f};
    float m_run[2] = {-INFINITY, -INFINITY};
    float l_run[2] = {0.f, 0.f};

    for (int kb0 = 0; kb0 < len; kb0 += kBlockKeys) {
      __syncthreads();
      // Stage K (row-major) and V (transposed) for keys kb0 .. kb0+63.
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int e = tid + u * kThreads;
        const int key = e >> 3, dv = e & 7;
        uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
        if (kb0 + key < len) {
          const long long off = (seq0 + kb0 + key) * row_elems + h * kD + dv * 8;
          kv = *reinterpret_cast<const uint4*>(K + off);
          vv = *reinterpret_cast<const uint4*>(V + off);
        }
        *reinterpret_cast<uint4*>(&Ks[key * kKStride + dv * 8]) = kv;
        const uint32_t w[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          Vt[(dv * 8 + 2 * i) * kVStride + key] = static_cast<uint16_t>(w[i] & 0xFFFFu);
          Vt[(dv * 8 + 2 * i + 1) * kVStride + key] = static_cast<uint16_t>(w[i] >> 16);
        }
      }
      __syncthreads();
      if (!active) continue;

      // S^T[key][query] for 4 key tiles of 16 and 2 query tiles of 16.
      floatx4 s[2][4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        const bf16x8 a0 = *reinterpret_cast<const bf16x8*>(&Ks[(kt * 16 + c16) * kKStride + g * 8]);
        const bf16x8 a1 = *reinterpret_cast<const bf16x8*>(&Ks[(kt * 16 + c16) * kKStride + 32 + g * 8]);
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          floatx4 acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, qf[j][0], floatx4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
          s[j][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, qf[j][1], acc, 0, 0, 0);
        }
      }

      // Online softmax (log2 domain).  Lane holds keys kt*16 + 4g + i of its query.
      const int kvalid = len - kb0;
      bf16x8 pb[2][2];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        float mx = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int key = kt * 16 + 4 * g + i;
            const float x = key < kvalid ? s[j][kt][i] * p.scale_log2 : -INFINITY;
            s[j][kt][i] = x;
            mx = fmaxf(mx, x);
          }
        mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        const float m_new = fmaxf(m_run[j], mx);
        const float alpha = __builtin_amdgcn_exp2f(m_run[j] - m_new);
        m_run[j] = m_new;
        float rs = 0.f;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float pv = __builtin_amdgcn_exp2f(s[j][kt][i] - m_new);
            s[j][kt][i] = pv;
            rs += pv;
          }
        l_run[j] = l_run[j] * alpha + rs;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) o[j][dt] *= alpha;
        // B operand of the PV step ks: k = 8g + e <-> key ks*32 + (e<4 ? 4g+e : 16+4g+e-4).
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            pb[j][ks][e] = static_cast<__bf16>(s[j][2 * ks][e]);
            pb[j][ks][4 + e] = static_cast<__bf16>(s[j][2 * ks + 1][e]);
          }
      }

      // O^T[dim][query] += V^T[dim][key] P^T[key][query].
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const uint16_t* vrow = &Vt[(dt * 16 + c16) * kVStride + ks * 32 + 4 * g];
          const bf16x4 lo = *reinterpret_cast<const bf16x4*>(vrow);
          const bf16x4 hi = *reinterpret_cast<const bf16x4*>(vrow + 16);
          const bf16x8 a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
          for (int j = 0; j < 2; ++j)
            o[j][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb[j][ks], o[j][dt], 0, 0, 0);
        }
      }
    }

    if (active) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        float l = l_run[j] + __shfl_xor(l_run[j], 16, 64);
        l += __shfl_xor(l, 32, 64);
        const float inv = 1.0f / l;
        const int qi = q0 + 16 * j + c16;
        if (qi < len) {
          uint16_t* dst = O + (seq0 + qi) * row_elems + h * kD + 4 * g;
#pragma unroll
          for (int dt = 0; dt < 4; ++dt) {
            bf16x4 r;
#pragma unroll
            for (int i = 0; i < 4; ++i) r[i] = static_cast<__bf16>(o[j][dt][i] * inv);
            *reinterpret_cast<bf16x4*>(dst + dt * 16) = r;
          }
        }
      }
    }
    __syncthreads();
  }
  leave_queue(p.hdr);
}

// ---------------------------------------------------------------------------
// fp32 inputs, v_mfma_f32_16x16x4_f32 (true fp32 products, fp32 accumulate).
//
// MFMA 16x16x4 f32 operand layout (lane l, g = l / 16, c = l % 16):
//   A[16 x 4]: lane holds row c, k = g;  B[4 x 16]: lane holds column c, k = g
//   D[16 x 16]: lane holds column c, rows 4g .. 4g+3
// ---------------------------------------------------------------------------
constexpr int kFStride = kD + 4;  // floats per K / V row in LDS

__global__ __launch_bounds__(kThreads) void attn_fwd_f32_kernel(AttnParams p) {
  __shared__ __attribute__((aligned(16))) float Ks[kBlockKeys * kFStride];
  __shared__ __attribute__((aligned(16))) float Vs[kBlockKeys * kFStride];
  __shared__ int s_ticket;

  if (!plan_matches(p)) {
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(p.status, DORA_DEV_PLAN);
    return;
  }
  const int n_items = min(p.hdr->n_items, p.max_items);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int c16 = lane & 15;
  const int g = lane >> 4;
  const float* Q = static_cast<const float*>(p.q);
  const float* K = static_cast<const float*>(p.k);
  const float* V = static_cast<const float*>(p.v);
  float* O = static_cast<float*>(p.out);
  const long long row_elems = static_cast<long long>(p.H) * kD;

  for (;;) {
    if (tid == 0) s_ticket = atomicAdd(&p.hdr->counter, 1);
    __syncthreads();
    const int ticket = s_ticket;
    if (ticket >= n_items) break;
    const int2 item = p.items[ticket];
    const int b = item.x, h = item.y >> 16, tile = item.y & 0xFFFF;
    long long seq0;
    int len;
    if (!item_bounds(p, b, h, tile, &seq0, &len)) {
      if (tid == 0) atomicOr(p.status, DORA_DEV_CU_SEQLENS);
      __syncthreads();
      continue;
    }
    const int q0 = tile * kAttnQTile + wave * kQPerWave;
    const bool active = q0 < len;

    float qf[2][16];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int qi = q0 + 16 * j + c16;
#pragma unroll
      for (int ks = 0; ks < 16; ++ks)
        qf[j][ks] = qi < len ? Q[(seq0 + qi) * row_elems + h * kD + 4 * ks + g] : 0.f;
    }
    floatx4 o[2][4];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) o[j][dt] = floatx4{0.f, 0.f, 0.f, 0.f};
    float m_run[2] = {-INFINITY, -INFINITY};
    float l_run[2] = {0.f, 0.f};

    for (int kb0 = 0; kb0 < len; kb0 += kBlockKeys) {
      __syncthreads();
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = tid + u * kThreads;  // 64 keys x 16 float4
        const int key = e >> 4, dv = e & 15;
        float4 kv = make_float4(0.f, 0.f, 0.f, 0.f), vv = kv;
        if (kb0 + key < len) {
          const long long off = (seq0 + kb0 + key) * row_elems + h * kD + dv * 4;
          kv = *reinterpret_cast<const float4*>(K + off);
          vv = *reinterpret_cast<const float4*>(V + off);
        }
        *reinterpret_cast<float4*>(&Ks[key * kFStride + dv * 4]) = kv;
        *reinterpret_cast<float4*>(&Vs[key * kFStride + dv * 4]) = vv;
      }
      __syncthreads();
      if (!active) continue;

      floatx4 s[2][4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
        for (int j = 0; j < 2; ++j) s[j][kt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < 16; ++ks) {
          const float a = Ks[(kt * 16 + c16) * kFStride + 4 * ks + g];
#pragma unroll
          for (int j = 0; j < 2; ++j)
            s[j][kt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, qf[j][ks], s[j][kt], 0, 0, 0);
        }
      }
      // The running max stays in raw score units and is subtracted before
      // scaling, so the terms near the max carry only a small rounding error.
      const int kvalid = len - kb0;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        float mx = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int key = kt * 16 + 4 * g + i;
            const float x = key < kvalid ? s[j][kt][i] : -INFINITY;
            s[j][kt][i] = x;
            mx = fmaxf(mx, x);
          }
        mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        const float m_new = fmaxf(m_run[j], mx);
        const float alpha = __builtin_amdgcn_exp2f((m_run[j] - m_new) * p.scale_log2);
        m_run[j] = m_new;
        float rs = 0.f;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float pv = __builtin_amdgcn_exp2f((s[j][kt][i] - m_new) * p.scale_log2);
            s[j][kt][i] = pv;
            rs += pv;
          }
        l_run[j] = l_run[j] * alpha + rs;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) o[j][dt] *= alpha;
      }
      // O^T += V^T P^T, one 4-key step per (kt, i): MFMA k = g <-> key kt*16 + 4g + i.
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int dt = 0; dt < 4; ++dt) {
            const float a = Vs[(kt * 16 + 4 * g + i) * kFStride + dt * 16 + c16];
#pragma unroll
            for (int j = 0; j < 2; ++j)
              o[j][dt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, s[j][kt][i], o[j][dt], 0, 0, 0);
          }
    }

    if (active) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        float l = l_run[j] + __shfl_xor(l_run[j], 16, 64);
        l += __shfl_xor(l, 32, 64);
        const float inv = 1.0f / l;
        const int qi = q0 + 16 * j + c16;
        if (qi < len) {
          float* dst = O + (seq0 + qi) * row_elems + h * kD + 4 * g;
#pragma unroll
          for (int dt = 0; dt < 4; ++dt)
            *reinterpret_cast<float4*>(dst + dt * 16) =
                make_float4(o[j][dt][0] * inv, o[j][dt][1] * inv, o[j][dt][2] * inv, o[j][dt][3] * inv);
        }
      }
    }
    __syncthreads();
  }
  leave_queue(p.hdr);
}

// Persistent grid: every compute unit filled to the kernel's occupancy.
template <typename KernelT>
int persistent_grid(KernelT kernel, int slot, int* grid) {
  static int per_cu_cache[64][2];
  int dev = 0;
  const int cus = device_cu_count(&dev);
  if (cus <= 0 || dev >= 64) return DORA_ERR_HIP;
  if (per_cu_cache[dev][slot] == 0) {
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kThreads, 0) != hipSuccess ||
        per_cu < 1)
      per_cu = 1;
    per_cu_cache[dev][slot] = per_cu;
  }
  *grid = cus * per_cu_cache[dev][slot];
  return DORA_OK;
}

int check_attn_sizes(int32_t B, int32_t H, int32_t max_seqlen, int64_t total) {
  if (B < 1 || H < 1 || H > 256 || max_seqlen < 1 || max_seqlen > DORA_MAX_SEQLEN || total < 0 ||
      total > INT_MAX)
    return DORA_ERR_SHAPE;
  const AttnWorkspaceLayout L = attn_workspace_layout(B, H, max_seqlen);
  if (L.max_items > INT_MAX) return DORA_ERR_UNSUPPORTED;
  return DORA_OK;
}

void fill_views(void* workspace, int32_t B, int32_t H, int32_t max_seqlen, AttnPlanHeader** hdr,
                int32_t** order, int32_t** base, int2** items, int64_t* max_items) {
  const AttnWorkspaceLayout L = attn_workspace_layout(B, H, max_seqlen);
  char* w = static_cast<char*>(workspace);
  *hdr = reinterpret_cast<AttnPlanHeader*>(w);
  *order = reinterpret_cast<int32_t*>(w + L.order_off);
  *base = reinterpret_cast<int32_t*>(w + L.base_off);
  *items = reinterpret_cast<int2*>(w + L.items_off);
  *max_items = L.max_items;
}

}  // namespace

int device_cu_count(int* device_out) {
  static int cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -1;
  if (device_out) *device_out = dev;
  if (dev < 0 || dev >= 64) return -1;
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -1;
    cache[dev] = n;
  }
  return cache[dev];
}

}  // namespace dora

extern "C" size_t dora_varlen_attn_workspace_size(int32_t B, int32_t H, int32_t max_seqlen) {
  if (dora::check_attn_sizes(B, H, max_seqlen, 0) != DORA_OK) return 0;
  return dora::attn_workspace_layout(B, H, max_seqlen).bytes;
}

extern "C" int dora_varlen_attn_plan(const int32_t* cu_seqlens, int32_t B, int32_t H,
                                     int32_t max_seqlen, int64_t total, void* workspace,
                                     size_t workspace_bytes, int32_t* dev_status, void* stream) {
  using namespace dora;
  if (!cu_seqlens || !dev_status) return DORA_ERR_NULL;
  const int sz = check_attn_sizes(B, H, max_seqlen, total);
  if (sz != DORA_OK) return sz;
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) ||
      workspace_bytes < attn_workspace_layout(B, H, max_seqlen).bytes)
    return DORA_ERR_WORKSPACE;
  PlanParams p;
  p.cu = cu_seqlens;
  p.B = B;
  p.H = H;
  p.max_seqlen = max_seqlen;
  p.total = total;
  p.status = dev_status;
  fill_views(workspace, B, H, max_seqlen, &p.hdr, &p.order, &p.item_base, &p.items, &p.max_items);
  hipLaunchKernelGGL(attn_plan_kernel, dim3(1), dim3(kPlanThreads), 0, static_cast<hipStream_t>(stream), p);
  return hipGetLastError() == hipSuccess ? DORA_OK : DORA_ERR_HIP;
}

extern "C" int dora_varlen_attn_execute(const void* q, const void* k, const void* v,
                                        const int32_t* cu_seqlens, int32_t B, int32_t H, int32_t D,
                                        int32_t max_seqlen, int64_t total, float softmax_scale,
                                        dora_dtype dtype, void* out, void* workspace,
                                        size_t workspace_bytes, int32_t* dev_status, void* stream) {
  using namespace dora;
  if (!q || !k || !v || !cu_seqlens || !out || !dev_status) return DORA_ERR_NULL;
  if (dtype != DORA_F32 && dtype != DORA_BF16) return DORA_ERR_DTYPE;
  if (D != DORA_HEAD_DIM) return DORA_ERR_SHAPE;
  const int sz = check_attn_sizes(B, H, max_seqlen, total);
  if (sz != DORA_OK) return sz;
  if ((reinterpret_cast<uintptr_t>(q) | reinterpret_cast<uintptr_t>(k) | reinterpret_cast<uintptr_t>(v) |
       reinterpret_cast<uintptr_t>(out)) & 15u)
    return DORA_ERR_ALIGN;
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) ||
      workspace_bytes < attn_workspace_layout(B, H, max_seqlen).bytes)
    return DORA_ERR_WORKSPACE;
  if (!(softmax_scale > 0.0f)) softmax_scale = 1.0f / sqrtf(static_cast<float>(D));

  AttnParams p;
  p.q = q;
  p.k = k;
  p.v = v;
  p.out = out;
  p.cu = cu_seqlens;
  p.B = B;
  p.H = H;
  p.max_seqlen = max_seqlen;
  p.total = total;
  p.scale_log2 = softmax_scale * kLog2e;
  p.status = dev_status;
  int32_t* order;
  int32_t* base;
  int2* items;
  int64_t max_items;
  fill_views(workspace, B, H, max_seqlen, &p.hdr, &order, &base, &items, &max_items);
  p.items = items;
  p.max_items = static_cast<int32_t>(max_items);

  int grid = 0;
  const int rc = dtype == DORA_BF16 ? persistent_grid(attn_fwd_bf16_kernel, 0, &grid)
                                    : persistent_grid(attn_fwd_f32_kernel, 1, &grid);
  if (rc != DORA_OK) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (dtype == DORA_BF16)
    hipLaunchKernelGGL(attn_fwd_bf16_kernel, dim3(grid), dim3(kThreads), 0, st, p);
  else
    hipLaunchKernelGGL(attn_fwd_f32_kernel, dim3(grid), dim3(kThreads), 0, st, p);
  return hipGetLastError() == hipSuccess ? DORA_OK : DORA_ERR_HIP;
}

extern "C" int dora_varlen_attn(const void* q, const void* k, const void* v,
                                const int32_t* cu_seqlens, int32_t B, int32_t H, int32_t D,
                                int32_t max_seqlen, int64_t total, float softmax_scale,
                                dora_dtype dtype, void* out, void* workspace, size_t workspace_bytes,
                                int32_t* dev_status, void* stream) {
  if (!q || !k || !v || !out) return DORA_ERR_NULL;
  if (dtype != DORA_F32 && dtype != DORA_BF16) return DORA_ERR_DTYPE;
  if (D != DORA_HEAD_DIM) return DORA_ERR_SHAPE;
  if ((reinterpret_cast<uintptr_t>(q) | reinterpret_cast<uintptr_t>(k) | reinterpret_cast<uintptr_t>(v) |
       reinterpret_cast<uintptr_t>(out)) & 15u)
    return DORA_ERR_ALIGN;
  int rc = dora_varlen_attn_plan(cu_seqlens, B, H, max_seqlen, total, workspace, workspace_bytes,
                                 dev_status, stream);
  if (rc != DORA_OK) return rc;
  return dora_varlen_attn_execute(q, k, v, cu_seqlens, B, H, D, max_seqlen, total, softmax_scale,
                                  dtype, out, workspace, workspace_bytes, dev_status, stream);
}

extern "C" const char* dora_status_string(int status) {
  switch (status) {
    case DORA_OK: return "DORA_OK";
    case DORA_ERR_NULL: return "DORA_ERR_NULL: a required pointer is NULL";
    case DORA_ERR_SHAPE: return "DORA_ERR_SHAPE: a size is out of range";
    case DORA_ERR_DTYPE: return "DORA_ERR_DTYPE: unknown dtype";
    case DORA_ERR_ALIGN: return "DORA_ERR_ALIGN: row data must be 16-byte aligned";
    case DORA_ERR_UNSUPPORTED: return "DORA_ERR_UNSUPPORTED: outside what this build implements";
    case DORA_ERR_CAPACITY: return "DORA_ERR_CAPACITY: output capacity out of range";
    case DORA_ERR_HIP: return "DORA_ERR_HIP: HIP runtime error at launch";
    case DORA_ERR_WORKSPACE: return "DORA_ERR_WORKSPACE: workspace missing, misaligned or too small";
    default: return "unknown dora status";
  }
}
