// Decode of the deterministic actor's outputs into the inputs of
// select/pack, on the device, with no host synchronisation.
// DORA (arXiv 2609.34325): Sec. 3.2 "Gate", "Budget head and selector" and
// "Sampling and deployment"; App. A.2 (budget grid {2, 4, ..., N0 - 4} with
// M = (N0 - 4) / 2 outputs; legal budgets leave at least four visual tokens);
// App. A.3 (deployment: gate at probability >= 0.5 when a budget is legal,
// the legal budget with the largest logit, the k highest removal scores go).
//
//   actor_gate_kernel    one workgroup: gate decision per image and the
//                        ordered compaction of the gate-on images (ballot +
//                        mbcnt within a wave, wave counts through LDS), so
//                        the controller can run on gate-on images only.
//   actor_decode_kernel  one wave per image: argmax over the legal budget
//                        logits (the first maximum; NaN above every number),
//                        keep = tokens - budget; all threads also negate the
//                        selector's removal scores into keep-scores.
#include "dora_internal.h"

namespace dora {
namespace {

constexpr int kGateThreads = 1024;
constexpr int kDecodeThreads = 256;
constexpr int kDecodeWaves = kDecodeThreads / 64;
constexpr int32_t kActorMaxB = 1 << 24;  // images per call (keeps every index in int32)

// Legal budgets 2(m+1), m < M, with 2(m+1) <= (n_tok - 1) - 4: their count.
__device__ __forceinline__ int legal_budgets(int n_tok, int M) {
  const int c = n_tok >= 5 ? (n_tok - 5) >> 1 : 0;
  return c < M ? c : M;
}

// Token count of image b (CLS included); 0 when its segment is invalid.
__device__ __forceinline__ int image_tokens(const int32_t* cu_in, int b, int N) {
  if (!cu_in) return N;
  const int lo = cu_in[b], hi = cu_in[b + 1];
  const int n = hi - lo;
  return (lo >= 0 && n >= 1 && n <= N) ? n : 0;
}

struct GateParams {
  const float* p_gate;
  const int32_t* cu_in;
  int32_t B, N, M;
  int32_t* on_rank;
  int32_t* on_list;
  int32_t* n_on;
  int32_t* status;
};

__global__ __launch_bounds__(kGateThreads) void actor_gate_kernel(GateParams p) {
  __shared__ int s_count[kGateThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int ranked = 0;  // gate-on images before the current chunk
  bool bad = false;
  for (int base = 0; base < p.B; base += kGateThreads) {
    const int b = base + tid;
    bool open = false;
    if (b < p.B) {
      const int n = image_tokens(p.cu_in, b, p.N);
      bad |= n == 0;
      open = n > 0 && p.p_gate[b] >= 0.5f && legal_budgets(n, p.M) > 0;
    }
    const uint64_t mask = __ballot(open);
    if (lane == 0) s_count[wave] = __popcll(mask);
    __syncthreads();
    int before = 0, chunk = 0;
#pragma unroll
    for (int w = 0; w < kGateThreads / 64; ++w) {
      const int c = s_count[w];
      before += w < wave ? c : 0;
      chunk += c;
    }
    if (b < p.B) {
      const int r = ranked + before + lanes_below(mask);
      p.on_rank[b] = open ? r : -1;
      if (open) p.on_list[r] = b;
    }
    ranked += chunk;
    __syncthreads();  // s_count is rewritten by the next chunk
  }
  for (int i = ranked + tid; i < p.B; i += kGateThreads) p.on_list[i] = -1;
  if (tid == 0) *p.n_on = ranked;
  if (bad) atomicOr(p.status, DORA_DEV_CU_IN);
}

struct DecodeParams {
  const float* logits;
  int64_t rows;
  int32_t M;
  const float* removal;
  float* keep_scores;
  int64_t n_scores;
  const int32_t* cu_in;
  int32_t B, N;
  const int32_t* on_rank;
  int32_t* keep;
  int32_t* status;
};

// a before b in the argmax order: NaN above every number, then larger values;
// equal values (or two NaNs) by the lower index.
__device__ __forceinline__ bool ranks_above(float a, int ia, float b, int ib) {
  const bool na = a != a, nb = b != b;
  if (na != nb) return na;
  if (!na && a != b) return a > b;
  return ia < ib;
}

__global__ __launch_bounds__(kDecodeThreads) void actor_decode_kernel(DecodeParams p) {
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * kDecodeWaves + (threadIdx.x >> 6);
  if (b < p.B) {
    const int n = image_tokens(p.cu_in, b, p.N);
    const int r = p.on_rank[b];
    int keep = n, flag = 0;
    if (n == 0) {
      flag = DORA_DEV_CU_IN;
    } else if (r >= 0) {
      const int legal = legal_budgets(n, p.M);
      if (legal == 0 || r >= p.rows) {
        flag = DORA_DEV_ACTOR;  // left unpruned
      } else {
        const float* row = p.logits + static_cast<int64_t>(r) * p.M;
        float best = -__builtin_inff();
        int ib = INT32_MAX;
        for (int m = lane; m < legal; m += 64) {
          const float x = row[m];
          if (ranks_above(x, m, best, ib)) best = x, ib = m;
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
          const float xo = __shfl_xor(best, off);
          const int io = __shfl_xor(ib, off);
          if (ranks_above(xo, io, best, ib)) best = xo, ib = io;
        }
        keep = n - 2 * (ib + 1);
      }
    }
    if (lane == 0) {
      p.keep[b] = keep;
      if (flag) atomicOr(p.status, flag);
    }
  }
  if (p.removal) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kDecodeThreads;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kDecodeThreads + threadIdx.x; i < p.n_scores; i += stride)
      p.keep_scores[i] = -p.removal[i];
  }
}

}  // namespace
}  // namespace dora

extern "C" int dora_actor_gate(const float* p_gate, const int32_t* cu_in, int32_t B, int32_t N, int32_t M,
                               int32_t* on_rank, int32_t* on_list, int32_t* n_on, int32_t* dev_status,
                               void* stream) {
  using namespace dora;
  if (!p_gate || !on_rank || !on_list || !n_on || !dev_status) return DORA_ERR_NULL;
  if (B < 1 || B > kActorMaxB || N < 1 || M < 1 || N > DORA_MAX_ROW_TOKENS) return DORA_ERR_SHAPE;
  GateParams p{p_gate, cu_in, B, N, M, on_rank, on_list, n_on, dev_status};
  hipLaunchKernelGGL(actor_gate_kernel, dim3(1), dim3(kGateThreads), 0, static_cast<hipStream_t>(stream), p);
  return hipGetLastError() == hipSuccess ? DORA_OK : DORA_ERR_HIP;
}

extern "C" int dora_actor_decode(const float* budget_logits, int64_t logit_rows, int32_t M,
                                 const float* removal_scores, const int32_t* cu_in, int64_t total_in, int32_t B,
                                 int32_t N, const int32_t* on_rank, int32_t* keep_out, float* scores_out,
                                 int32_t* dev_status, void* stream) {
  using namespace dora;
  if (!on_rank || !keep_out || !dev_status) return DORA_ERR_NULL;
  if ((removal_scores == nullptr) != (scores_out == nullptr)) return DORA_ERR_NULL;
  if (!budget_logits && logit_rows > 0) return DORA_ERR_NULL;
  if (B < 1 || B > kActorMaxB || N < 1 || M < 1 || N > DORA_MAX_ROW_TOKENS || logit_rows < 0 ||
      logit_rows > 0x7FFFFFFF)
    return DORA_ERR_SHAPE;
  const int64_t n_scores = cu_in ? total_in : static_cast<int64_t>(B) * N;
  if (n_scores < 0) return DORA_ERR_SHAPE;
  DecodeParams p{budget_logits, logit_rows, M, removal_scores, scores_out, n_scores, cu_in, B, N,
                 on_rank, keep_out, dev_status};
  // One wave per image; the score negation strides over whatever grid that
  // gives, widened to about four scores per thread (at most 2048 workgroups).
  const int64_t for_images = (static_cast<int64_t>(B) + kDecodeWaves - 1) / kDecodeWaves;
  int64_t for_scores = removal_scores ? (n_scores + kDecodeThreads * 4 - 1) / (kDecodeThreads * 4) : 0;
  if (for_scores > 2048) for_scores = 2048;
  const int64_t grid = for_images > for_scores ? for_images : for_scores;
  hipLaunchKernelGGL(actor_decode_kernel, dim3(static_cast<unsigned>(grid)), dim3(kDecodeThreads), 0,
                     static_cast<hipStream_t>(stream), p);
  return hipGetLastError() == hipSuccess ? DORA_OK : DORA_ERR_HIP;
}
