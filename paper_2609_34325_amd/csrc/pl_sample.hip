// Plackett-Luce deletion by Gumbel-top-k and its ordered log-probability.
// DORA (arXiv 2609.34325): Sec. 3.2 "Sampling and deployment" (training
// draws exactly k distinct tokens without replacement from a Plackett-Luce
// distribution over the selector's scores and keeps the drawing order);
// App. A.3, Eq. (app-actor-pl) (the ordered log-probability
// sum_t [ s_{i_t} - log sum_{j in R_t} exp(s_j) ], R_t the tokens not drawn
// before step t).
//
// One workgroup per image.  Sampling: the keys s_j + g_j (g Gumbel noise,
// passed in) of the visual tokens become 64-bit sort words (an
// order-preserving image of the FP32 key above the position), are sorted in
// LDS by a bitonic network, and the first k words give the draws in order.
// The same total order as select/pack on keep-scores -key (NaN drawn first,
// equal keys by higher position), so the drawn set is exactly what select /
// pack deletes with those keep-scores.  Log-probability: with m the largest
// visual score, e_u = exp(s_u - m) is laid out in drawing order (draws first,
// then the survivors), a reverse block scan gives every denominator
// sum_{v >= u} e_v at once, and the k terms are summed in a fixed order.
#include "dora_internal.h"

namespace dora {
namespace {

constexpr int kPLThreads = 256;
constexpr int kPLMaxSlots = DORA_MAX_ROW_TOKENS;  // sort / scan width (power of two >= visual tokens)
static_assert((kPLMaxSlots & (kPLMaxSlots - 1)) == 0, "bitonic width must be a power of two");

struct PLParams {
  const float* s;      // removal scores, select/pack layout
  const float* g;      // Gumbel noise, same layout (sampling only)
  const int32_t* k;    // draws per image (sampling only)
  const int32_t* order_in;     // given orders (evaluation only)
  const int32_t* cu_order_in;  // their offsets (evaluation only)
  const int32_t* cu_in;
  int64_t total_in;
  int32_t B, N;
  int32_t* order_out;
  int32_t* cu_order_out;
  float* logprob;
  int64_t cap;
  int32_t* status;
};

// Order-preserving image of an FP32 key as uint32 (-0 == +0; NaN above all).
__device__ __forceinline__ uint32_t key_bits(float x) {
  if (x != x) return 0xFFFFFFFFu;
  uint32_t u = __float_as_uint(x == 0.0f ? 0.0f : x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float block_sum(float v, float* s_red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  __syncthreads();
  if (lane == 0) s_red[wave] = v;
  __syncthreads();
  float t = 0.0f;
#pragma unroll
  for (int w = 0; w < kPLThreads / 64; ++w) t += s_red[w];
  return t;
}

__device__ __forceinline__ float block_max(float v, float* s_red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  __syncthreads();
  if (lane == 0) s_red[wave] = v;
  __syncthreads();
  float t = s_red[0];
#pragma unroll
  for (int w = 1; w < kPLThreads / 64; ++w) t = fmaxf(t, s_red[w]);
  return t;
}

__device__ __forceinline__ long long block_sum_ll(long long v, long long* s_red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  __syncthreads();
  if (lane == 0) s_red[wave] = v;
  __syncthreads();
  long long t = 0;
#pragma unroll
  for (int w = 0; w < kPLThreads / 64; ++w) t += s_red[w];
  return t;
}

// Larger and smaller of a lane's 64-bit word and the word of lane ^ STRIDE
// (STRIDE < 64, all lanes active), without a trip through the LDS crossbar
// where the hardware offers a register path: DPP quad permutations (1, 2),
// a DPP row rotation by 8 (XOR 8 within a row of 16 lanes), the swizzle's
// XOR mode (4), and the row swaps of v_permlane16/32_swap (16, 32), which
// hand each lane both words of its pair in some order -- all a min/max
// needs.
template <int STRIDE>
__device__ __forceinline__ void xor_minmax(unsigned long long x, unsigned long long& mx, unsigned long long& mn) {
  const uint32_t lo = static_cast<uint32_t>(x), hi = static_cast<uint32_t>(x >> 32);
  unsigned long long a = x, b;
  if constexpr (STRIDE == 16 || STRIDE == 32) {
    const auto l2 = STRIDE == 16 ? __builtin_amdgcn_permlane16_swap(lo, lo, false, false)
                                 : __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
    const auto h2 = STRIDE == 16 ? __builtin_amdgcn_permlane16_swap(hi, hi, false, false)
                                 : __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
    a = (static_cast<unsigned long long>(h2[0]) << 32) | l2[0];
    b = (static_cast<unsigned long long>(h2[1]) << 32) | l2[1];
  } else {
    uint32_t pl, ph;
    if constexpr (STRIDE == 1) {  // quad_perm [1, 0, 3, 2]
      pl = __builtin_amdgcn_update_dpp(0u, lo, 0xB1, 0xF, 0xF, false);
      ph = __builtin_amdgcn_update_dpp(0u, hi, 0xB1, 0xF, 0xF, false);
    } else if constexpr (STRIDE == 2) {  // quad_perm [2, 3, 0, 1]
      pl = __builtin_amdgcn_update_dpp(0u, lo, 0x4E, 0xF, 0xF, false);
      ph = __builtin_amdgcn_update_dpp(0u, hi, 0x4E, 0xF, 0xF, false);
    } else if constexpr (STRIDE == 8) {  // row_ror:8
      pl = __builtin_amdgcn_update_dpp(0u, lo, 0x128, 0xF, 0xF, false);
      ph = __builtin_amdgcn_update_dpp(0u, hi, 0x128, 0xF, 0xF, false);
    } else {  // STRIDE == 4: swizzle, bitmask mode, xor_mask 4, and_mask 0x1F
      static_assert(STRIDE == 4, "stride");
      pl = static_cast<uint32_t>(__builtin_amdgcn_ds_swizzle(static_cast<int>(lo), 0x101F));
      ph = static_cast<uint32_t>(__builtin_amdgcn_ds_swizzle(static_cast<int>(hi), 0x101F));
    }
    b = (static_cast<unsigned long long>(ph) << 32) | pl;
  }
  mx = a > b ? a : b;
  mn = a < b ? a : b;
}

// Descending bitonic sort of the P = E * kPLThreads sort words in LDS, E
// words per thread in registers (element e = i * kPLThreads + thread id in
// x[i]).  The same network as the LDS sort (pairs (lo, lo + stride),
// descending where lo & size == 0): a step with stride < 64 pairs lanes of
// one wave (xor_minmax, no barrier); stride 64 or 128 pairs waves through
// LDS between two barriers; stride >= kPLThreads pairs two registers of a
// thread.  Called by every thread of the workgroup (uniformly), after the
// words are in LDS and a barrier; the sorted words are back in LDS after a
// final barrier.
__device__ __forceinline__ void cross_lane(unsigned long long& x, int stride, bool take_max) {
  unsigned long long mx, mn;
  switch (stride) {
    case 1: xor_minmax<1>(x, mx, mn); break;
    case 2: xor_minmax<2>(x, mx, mn); break;
    case 4: xor_minmax<4>(x, mx, mn); break;
    case 8: xor_minmax<8>(x, mx, mn); break;
    case 16: xor_minmax<16>(x, mx, mn); break;
    default: xor_minmax<32>(x, mx, mn); break;
  }
  x = take_max ? mx : mn;
}

template <int E>
__device__ void block_sort(unsigned long long* words) {
  static_assert(kPLThreads == 256, "waves of 64 lanes, four per workgroup");
  const int t = threadIdx.x;
  unsigned long long x[E];
#pragma unroll
  for (int i = 0; i < E; ++i) x[i] = words[i * kPLThreads + t];
#pragma unroll
  for (int size = 2; size <= E * kPLThreads; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      if (stride >= kPLThreads) {
        const int rs = stride / kPLThreads;
#pragma unroll
        for (int i = 0; i < E; ++i) {
          if (i & rs) continue;
          const bool desc = ((i * kPLThreads + t) & size) == 0;
          const unsigned long long a = x[i], b = x[i | rs];
          const unsigned long long mx = a > b ? a : b, mn = a < b ? a : b;
          x[i] = desc ? mx : mn;
          x[i | rs] = desc ? mn : mx;
        }
      } else if (stride >= 64) {
        __syncthreads();  // every read of the previous exchange is done
#pragma unroll
        for (int i = 0; i < E; ++i) words[i * kPLThreads + t] = x[i];
        __syncthreads();
#pragma unroll
        for (int i = 0; i < E; ++i) {
          const int e = i * kPLThreads + t;
          const unsigned long long y = words[e ^ stride];
          const bool take_max = ((e & stride) == 0) == ((e & size) == 0);  // lo of a descending pair, or hi of an ascending one
          x[i] = take_max ? (x[i] > y ? x[i] : y) : (x[i] < y ? x[i] : y);
        }
      } else {
#pragma unroll
        for (int i = 0; i < E; ++i) {
          const int e = i * kPLThreads + t;
          cross_lane(x[i], stride, ((e & stride) == 0) == ((e & size) == 0));
        }
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < E; ++i) words[i * kPLThreads + t] = x[i];
  __syncthreads();
}

// In place: A[u] <- sum_{v >= u} A[v] over [0, P), P a multiple of kPLThreads.
// Thread t owns the consecutive slots [t c, (t + 1) c), c = P / kPLThreads.
__device__ void reverse_inclusive_scan(float* A, int P, float* s_red) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = P / kPLThreads, base = tid * c;
  float own = 0.0f;
  for (int i = c - 1; i >= 0; --i) own += A[base + i];
  // sum of the totals of the threads after this one
  float incl = own;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const float y = __shfl_down(incl, d);
    if (lane + d < 64) incl += y;
  }
  __syncthreads();
  if (lane == 0) s_red[wave] = incl;  // wave total
  __syncthreads();
  float after = incl - own;
#pragma unroll
  for (int w = 0; w < kPLThreads / 64; ++w) after += w > wave ? s_red[w] : 0.0f;
  float run = after;
  for (int i = c - 1; i >= 0; --i) {
    run += A[base + i];
    A[base + i] = run;
  }
  __syncthreads();
}

template <bool SAMPLE>
__global__ __launch_bounds__(kPLThreads) void pl_kernel(PLParams p) {
  __shared__ unsigned long long s_word[kPLMaxSlots];  // sort words (sampling)
  __shared__ float s_score[kPLMaxSlots];              // visual scores by position - 1
  __shared__ float s_e[kPLMaxSlots];                  // exp terms in drawing order, then suffix sums
  __shared__ int s_mark[kPLMaxSlots];                 // draws per position (evaluation)
  __shared__ float s_red[kPLThreads / 64];
  __shared__ long long s_red_ll[kPLThreads / 64];
  const int b = blockIdx.x, tid = threadIdx.x;

  // Segment of image b and its validity.
  int64_t off_in;
  int n;
  bool seg_ok = true;
  if (p.cu_in) {
    const int lo = p.cu_in[b], hi = p.cu_in[b + 1];
    off_in = lo;
    n = hi - lo;
    seg_ok = lo >= 0 && n >= 1 && n <= p.N && hi <= p.total_in && (b > 0 || lo == 0);
  } else {
    off_in = static_cast<int64_t>(b) * p.N;
    n = p.N;
  }
  const int nv = seg_ok ? n - 1 : 0;  // visual tokens

  // Draw count and output offset.
  int kb;
  int64_t out0 = 0;
  if constexpr (SAMPLE) {
    kb = p.k[b];
    long long part = 0;
    for (int j = tid; j < b; j += kPLThreads) part += min(max(p.k[j], 0), p.N);  // valid k never exceeds N - 1
    out0 = block_sum_ll(part, s_red_ll);
    if (tid == 0) {
      if (b == 0) p.cu_order_out[0] = 0;
      p.cu_order_out[b + 1] = static_cast<int32_t>(out0 + min(max(kb, 0), p.N));
    }
  } else {
    // The list of image b is [cu_order[b], cu_order[b+1]) inside the caller's
    // cu_order[B] entries; offsets outside that range are rejected before any
    // entry is read.
    const int o0 = p.cu_order_in[b], o1 = p.cu_order_in[b + 1], oend = p.cu_order_in[p.B];
    out0 = o0;
    kb = (o0 >= 0 && o1 >= o0 && o1 <= oend && p.cu_order_in[0] == 0) ? o1 - o0 : -1;
  }
  bool ok = seg_ok && kb >= 0 && kb <= nv;
  if (!seg_ok && tid == 0) atomicOr(p.status, DORA_DEV_CU_IN);

  const int P = max(kPLThreads, nv > 1 ? 1 << (32 - __clz(nv - 1)) : 1);  // power of two >= nv
  const float* sb = p.s + off_in;
  float mloc = -__builtin_inff();
  for (int j = tid; j < P; j += kPLThreads) {
    const float x = j < nv ? sb[j + 1] : 0.0f;
    s_score[j] = x;
    if (j < nv) mloc = fmaxf(mloc, x);
    if constexpr (SAMPLE) {
      s_word[j] = j < nv ? (static_cast<unsigned long long>(key_bits(x + p.g[off_in + j + 1])) << 32) |
                               static_cast<uint32_t>(j + 1)
                         : 0ull;  // padding sorts last
    } else {
      s_mark[j] = 0;
    }
  }
  const float m = block_max(mloc, s_red);  // includes a barrier after the LDS writes

  if constexpr (SAMPLE) {
    if (ok) {
      // Bitonic sort, descending (earliest draw first): in registers, P / 256
      // words per thread, up to 1024 words; wider rows in LDS, a barrier
      // per step.
      if (P == kPLThreads) {
        block_sort<1>(s_word);
      } else if (P == 2 * kPLThreads) {
        block_sort<2>(s_word);
      } else if (P == 4 * kPLThreads) {
        block_sort<4>(s_word);
      } else {
        for (int size = 2; size <= P; size <<= 1) {
          for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = tid; i < P / 2; i += kPLThreads) {
              const int lo = 2 * i - (i & (stride - 1)), hi = lo + stride;
              const bool desc = (lo & size) == 0;
              const unsigned long long x = s_word[lo], y = s_word[hi];
              if ((x < y) == desc) {
                s_word[lo] = y;
                s_word[hi] = x;
              }
            }
            __syncthreads();
          }
        }
      }
      for (int u = tid; u < P; u += kPLThreads) {
        const int pos = static_cast<int>(s_word[u] & 0xFFFFFFFFu);  // 0 for padding
        if (u < kb) {
          const int64_t dst = out0 + u;
          if (dst < p.cap) p.order_out[dst] = pos;
        }
        s_e[u] = u < nv ? expf(s_score[pos - 1] - m) : 0.0f;
      }
    }
  } else {
    // Given order: mark the draws, check them, and lay out their terms first.
    if (ok) {
      for (int t = tid; t < kb; t += kPLThreads) {
        const int pos = p.order_in[out0 + t];
        if (pos >= 1 && pos <= nv) atomicAdd(&s_mark[pos - 1], 1);
        else atomicAdd(&s_mark[0], 1 << 20);  // out of range: poisons the check below
      }
    }
    __syncthreads();
    int badloc = 0;
    float surv = 0.0f;
    for (int j = tid; j < P; j += kPLThreads) {
      badloc |= j < nv && s_mark[j] > 1;
      if (j < nv && s_mark[j] == 0) surv += expf(s_score[j] - m);
    }
    const float s_surv = block_sum(surv, s_red);
    const long long nbad = block_sum_ll(badloc, s_red_ll);
    ok = ok && nbad == 0;
    for (int u = tid; u < P; u += kPLThreads) {
      float e = 0.0f;
      if (ok && u < kb) e = expf(s_score[p.order_in[out0 + u] - 1] - m);
      else if (u == kb) e = s_surv;
      s_e[u] = e;
    }
  }
  if (!ok) {
    if (tid == 0) {
      p.logprob[b] = __builtin_nanf("");
      if (seg_ok) atomicOr(p.status, DORA_DEV_KEEP_RANGE);
    }
    return;
  }
  if constexpr (SAMPLE) {
    if (tid == 0 && out0 + kb > p.cap) atomicOr(p.status, DORA_DEV_CAPACITY);
  }
  __syncthreads();
  reverse_inclusive_scan(s_e, P, s_red);
  // Terms in drawing order; the score of draw u is read back by position.
  float part = 0.0f;
  for (int u = tid; u < kb; u += kPLThreads) {
    int pos;
    if constexpr (SAMPLE) pos = static_cast<int>(s_word[u] & 0xFFFFFFFFu);
    else pos = p.order_in[out0 + u];
    part += (s_score[pos - 1] - m) - logf(s_e[u]);
  }
  const float lp = block_sum(part, s_red);
  if (tid == 0) p.logprob[b] = lp;
}

int check_pl(const float* s, const int32_t* cu_in, int64_t total_in, int32_t B, int32_t N) {
  if (!s) return DORA_ERR_NULL;
  if (B < 1 || B > kPlanMaxB || N < 1 || N > DORA_MAX_ROW_TOKENS) return DORA_ERR_SHAPE;
  if (cu_in && (total_in < 0 || total_in > 0x7FFFFFFF)) return DORA_ERR_SHAPE;
  return DORA_OK;
}

}  // namespace
}  // namespace dora

extern "C" int dora_pl_sample(const float* scores, const float* gumbel, const int32_t* k, const int32_t* cu_in,
                              int64_t total_in, int32_t B, int32_t N, int32_t* order_out, int32_t* cu_order_out,
                              float* logprob_out, int64_t cap, int32_t* dev_status, void* stream) {
  using namespace dora;
  const int rc = check_pl(scores, cu_in, total_in, B, N);
  if (rc != DORA_OK) return rc;
  if (!gumbel || !k || !order_out || !cu_order_out || !logprob_out || !dev_status) return DORA_ERR_NULL;
  if (cap < 1 || cap > 0x7FFFFFFF) return DORA_ERR_CAPACITY;
  PLParams p{scores, gumbel, k, nullptr, nullptr, cu_in, total_in, B, N, order_out, cu_order_out,
             logprob_out, cap, dev_status};
  hipLaunchKernelGGL(pl_kernel<true>, dim3(B), dim3(kPLThreads), 0, static_cast<hipStream_t>(stream), p);
  return hipGetLastError() == hipSuccess ? DORA_OK : DORA_ERR_HIP;
}

extern "C" int dora_pl_logprob(const float* scores, const int32_t* order, const int32_t* cu_order,
                               const int32_t* cu_in, int64_t total_in, int32_t B, int32_t N, float* logprob_out,
                               int32_t* dev_status, void* stream) {
  using namespace dora;
  const int rc = check_pl(scores, cu_in, total_in, B, N);
  if (rc != DORA_OK) return rc;
  if (!order || !cu_order || !logprob_out || !dev_status) return DORA_ERR_NULL;
  PLParams p{scores, nullptr, nullptr, order, cu_order, cu_in, total_in, B, N, nullptr, nullptr,
             logprob_out, 0, dev_status};
  hipLaunchKernelGGL(pl_kernel<false>, dim3(B), dim3(kPLThreads), 0, static_cast<hipStream_t>(stream), p);
  return hipGetLastError() == hipSuccess ? DORA_OK : DORA_ERR_HIP;
}
