// FLOP accounting of realised token trajectories.
// DORA (arXiv 2609.34325), App. E.4: two FLOPs per multiply-accumulate over
// the complete forward (patch embedding, backbone, classifier and the actor),
// following each image's own token trajectory: at block l the attention runs
// over the N_l + 1 tokens that enter it and the MLP over the N_l - k_l + 1 it
// keeps.  Actor shapes from App. A.1: gate (d + 16 + 3) -> 64 -> 1 on the CLS
// key at every block with a legal budget; where tokens were removed the
// controller ran: input projection d -> 128 of every key and 3 -> 128 of the
// history, one width-128 Transformer block (4 heads, FFN 128 -> 256 -> 128),
// budget head 128 -> 128 -> M, the 1 -> 128 projection of k / N, selector
// 128 -> 64 -> 1 on the visual tokens.
//
// One workgroup; thread t takes images t, t + 1024, ...; each walks its L
// blocks in exact int64 arithmetic, and the per-image counts are summed in a
// fixed order into the total.
#include "dora_internal.h"

namespace dora {
namespace {

constexpr int kFlopThreads = 1024;
constexpr int64_t kActW = 128, kActFfn = 256, kGateHidden = 64, kGateEmbed = 16, kHist = 3, kSelHidden = 64;

__device__ __forceinline__ int64_t block_attn_macs(int64_t n, int64_t d) {
  return n * d * 3 * d + 2 * n * n * d + n * d * d;
}

struct FlopParams {
  const int32_t* tokens;  // [L+1][B]
  int32_t B;
  dora_flops_config c;
  int64_t* flops;
  int64_t* total;
  int32_t* status;
};

__global__ __launch_bounds__(kFlopThreads) void trajectory_flops_kernel(FlopParams p) {
  __shared__ long long s_red[kFlopThreads / 64];
  const int64_t d = p.c.d;
  const int64_t fixed = static_cast<int64_t>(p.c.N0) * p.c.in_chans * p.c.patch * p.c.patch * d +
                        static_cast<int64_t>(p.c.head_inputs) * d * p.c.classes;
  const int64_t mlp_tok = 2 * d * (static_cast<int64_t>(p.c.mlp_ratio) * d);
  const int64_t gate = (d + kGateEmbed + kHist) * kGateHidden + kGateHidden;
  long long sum = 0;
  bool bad = false;
  for (int b = threadIdx.x; b < p.B; b += kFlopThreads) {
    int64_t macs = fixed;
    int64_t n = p.tokens[b];
    bool ok = n == p.c.N0 + 1;
    for (int l = 0; l < p.c.L; ++l) {
      const int64_t m = p.tokens[static_cast<int64_t>(l + 1) * p.B + b];
      ok = ok && m >= 1 && m <= n;
      macs += block_attn_macs(n, d) + m * mlp_tok;
      if (p.c.actor) {
        if (n - 1 >= 6) macs += gate;
        if (m < n) {
          macs += n * d * kActW + kHist * kActW;                                    // input projections
          macs += block_attn_macs(n, kActW) + n * 2 * kActW * kActFfn;              // encoder block
          macs += kActW * kActW + kActW * static_cast<int64_t>(p.c.M);              // budget head
          macs += kActW + (n - 1) * (kActW * kSelHidden + kSelHidden);              // k / N projection, selector
        }
      }
      n = m;
    }
    p.flops[b] = ok ? 2 * macs : -1;
    if (ok) sum += 2 * macs;
    bad |= !ok;
  }
  // total in a fixed order: lanes, then waves
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off);
  if (lane == 0) s_red[wave] = sum;
  __syncthreads();
  if (threadIdx.x == 0) {
    long long t = 0;
    for (int w = 0; w < kFlopThreads / 64; ++w) t += s_red[w];
    *p.total = t;
  }
  if (bad) atomicOr(p.status, DORA_DEV_KEEP_RANGE);
}

}  // namespace
}  // namespace dora

extern "C" int dora_trajectory_flops(const int32_t* tokens, int32_t B, const dora_flops_config* config,
                                     int64_t* flops_out, int64_t* total_out, int32_t* dev_status, void* stream) {
  using namespace dora;
  if (!tokens || !config || !flops_out || !total_out || !dev_status) return DORA_ERR_NULL;
  const dora_flops_config& c = *config;
  if (B < 1 || B > (1 << 24) || c.d < 1 || c.d > 65536 || c.L < 1 || c.L > 1024 || c.N0 < 1 ||
      c.N0 > DORA_MAX_ROW_TOKENS || c.patch < 1 || c.patch > 64 || c.in_chans < 1 || c.in_chans > 16 ||
      c.classes < 1 || c.classes > (1 << 20) || c.head_inputs < 1 || c.head_inputs > 8 || c.mlp_ratio < 1 ||
      c.mlp_ratio > 16 || c.M < 1 || c.M > DORA_MAX_ROW_TOKENS || (c.actor != 0 && c.actor != 1))
    return DORA_ERR_SHAPE;
  FlopParams p{tokens, B, c, flops_out, total_out, dev_status};
  hipLaunchKernelGGL(trajectory_flops_kernel, dim3(1), dim3(kFlopThreads), 0, static_cast<hipStream_t>(stream), p);
  return hipGetLastError() == hipSuccess ? DORA_OK : DORA_ERR_HIP;
}
