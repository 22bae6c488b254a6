// Hard deletion + packing: per-image top-k with CLS pinned, running total of
// keep counts, and the gather of kept rows into one packed buffer.
// DORA (arXiv 2609.34325): Sec. 3.1 Eq. (1) (delete rows, keep CLS and the
// survivors' order), Sec. 3.2 "Sampling and deployment" and App. A.3 (remove
// the highest-scoring visual tokens), Sec. 3.5 "Inference" (packed buffer with
// explicit sequence boundaries), App. E.5 (FP32 score comparisons).
//
// dora_select_pack_residual packs the kept rows of h + a instead, the
// attention residual (Sec. 3.1, Eq. (1): rows are deleted after the residual
// add): the same kernel body reads the two rows, adds them in fp32 and rounds
// once to the storage type, so the full sum is never written.
//
// One launch.  Workgroup (b, s) handles image b; the `split` workgroups of an
// image each repeat the (cheap) selection and then copy a disjoint share of
// the kept rows, so the HBM-bound copy is spread over many workgroups.
//
//   wave 0        rows of at most 256 tokens: radix select on
//                 order-preserving uint32 keys, one bit per step, counting
//                 with wave ballots (keys live in VGPRs); ordered compaction
//                 of the keep flags with ballot + mbcnt.
//   waves 1..3    sum keep[0..b) -> this image's output offset (cu_out[b]).
//   all waves     longer rows: the four waves each hold a quarter of the
//                 positions and select by 8-bit digits together (LDS
//                 histograms, a barrier per digit), then compact in order.
//   all waves     16-byte row copies, 2 loads in flight per lane.
//
// dora_select_pack_plan also writes the attention work queue of the packed
// output (Sec. 3.5 "Inference": one sequence per image, keep[b] rows): it
// depends on the keep counts only, so workgroup (b, 0) places image b's
// items while it sums the keep counts for its output offset (queue order:
// longer sequences first, then lower image index), and workgroup (0, 0)
// writes the plan header.
#include <limits.h>
#include <stdlib.h>

#include "dora_internal.h"

namespace dora {
namespace {

constexpr int kThreads = 256;
constexpr int kDigitSelectSlots = 8;  // rows of more than 256 tokens select by 8-bit digits
constexpr int kCopyUnroll = 2;  // loads in flight per lane: few, so stores start early (measured best)
// Up to this many images each workgroup sums keep[0..b) itself (at most 8 KB
// of keep counts from the L2, cheaper than a second launch); above it one
// workgroup scans the keep counts into cu_out first.
constexpr int kFusedScanMaxB = 2048;
constexpr int kScanThreads = 1024;
constexpr int kScanPer = 8;  // keep counts per thread and tile

struct SelectPackParams {
  const float* scores;
  const int32_t* keep;
  const uint4* tokens;
  const uint4* addend;  // residual-add variant: rows added to the token rows (same layout), else null
  const int32_t* cu_in;
  int64_t total_in;
  int32_t B, N, row_vecs, split;
  int32_t* idx_out;
  int32_t* cu_out;
  uint4* packed;
  int64_t cap_rows;
  int32_t* status;
  // Attention plan of the packed output (plan_hdr == nullptr: none).
  AttnPlanHeader* plan_hdr;
  int2* plan_items;
  int32_t H, max_seqlen, max_items;
  int64_t plan_total;
  // cu_out was written by keep_scan_kernel before this launch (batches of
  // more than kFusedScanMaxB images): each workgroup reads its offset there.
  int32_t cu_ready;
};

// Order-preserving key: larger key = preferred for keeping.  -0 and +0 map
// to the same key; every NaN maps to 0, below -inf (0x007FFFFF).
__device__ __forceinline__ uint32_t keep_key(float x) {
  uint32_t u = __float_as_uint(x);
  if (x != x) return 0u;
  if (x == 0.0f) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ long long wave_sum(long long v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Inclusive running sum over the 64 lanes of a wave, in DPP steps: shifts by
// 1, 2, 4 and 8 within each row of 16 lanes (lanes shifted in from outside
// the row add 0), then lane 15 of each row is added to the next row and lane
// 31 to the upper half.
__device__ __forceinline__ uint32_t wave_inclusive_sum(uint32_t x) {
  x += __builtin_amdgcn_update_dpp(0u, x, 0x111, 0xF, 0xF, false);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0u, x, 0x112, 0xF, 0xF, false);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0u, x, 0x114, 0xF, 0xF, false);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0u, x, 0x118, 0xF, 0xF, false);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0u, x, 0x142, 0xA, 0xF, false);  // row_bcast:15 into rows 1 and 3
  x += __builtin_amdgcn_update_dpp(0u, x, 0x143, 0xC, 0xF, false);  // row_bcast:31 into rows 2 and 3
  return x;
}

// Threshold of the valid keys of a long row, the four waves of the
// workgroup each holding a quarter of them: T = the need-th largest valid key
// (counted with multiplicity) and q = how many keys equal to T are kept,
// found one 8-bit digit at a time from the most significant.  A pass builds
// the 256-bin histogram of the digit of every valid key that matches the
// digits fixed so far (each wave into its own copy in LDS, by LDS atomics),
// and, after a barrier, every wave adds the four copies and fixes the
// largest digit whose count of keys at or above it still reaches the number
// of keys left to take; the keys above that digit are all taken.  Four
// dependent passes instead of 32 one-bit steps; a quarter of the keys per
// wave, so the same-bin atomics of a pass serialise over a quarter as many
// lanes.  hist: 2 x 4 x 256 words (two buffers, a copy per wave): a buffer
// is cleared by its owner one pass after its last reads, behind a barrier.
template <int S>
__device__ __forceinline__ void block_digit_threshold(const uint32_t (&key)[S], const uint64_t (&valid)[S],
                                                      int need, uint32_t* hist, int lane, int wave,
                                                      uint32_t& T, int& q) {
  constexpr int kBuf = 4 * 256;
  reinterpret_cast<uint4*>(hist + wave * 256)[lane] = make_uint4(0u, 0u, 0u, 0u);
  reinterpret_cast<uint4*>(hist + kBuf + wave * 256)[lane] = make_uint4(0u, 0u, 0u, 0u);
  uint32_t prefix = 0u, fixed = 0u;
  uint32_t left = static_cast<uint32_t>(need);
#pragma unroll
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    uint32_t* buf = hist + (pass & 1) * kBuf;
#pragma unroll
    for (int r = 0; r < S; ++r)
      if (((valid[r] >> lane) & 1ull) && (key[r] & fixed) == prefix)
        atomicAdd(&buf[wave * 256 + ((key[r] >> shift) & 255u)], 1u);
    __syncthreads();
    // bins 4 lane .. 4 lane + 3, summed over the four copies
    uint4 h = reinterpret_cast<const uint4*>(buf)[lane];
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      const uint4 g = reinterpret_cast<const uint4*>(buf + w * 256)[lane];
      h = make_uint4(h.x + g.x, h.y + g.y, h.z + g.z, h.w + g.w);
    }
    // The other buffer was read by every wave before this pass's barrier:
    // clear this wave's copy of it for the pass after next.
    if (pass >= 1) reinterpret_cast<uint4*>(hist + ((pass & 1) ^ 1) * kBuf + wave * 256)[lane] = make_uint4(0u, 0u, 0u, 0u);
    const uint32_t s3 = h.w, s2 = h.z + s3, s1 = h.y + s2, s0 = h.x + s1;
    const uint32_t upto = wave_inclusive_sum(s0);
    const uint32_t above = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(upto), 63)) - upto;
    // at_or_above[i]: keys whose digit is >= 4 lane + i.
    const uint32_t c0 = above + s0, c1 = above + s1, c2 = above + s2, c3 = above + s3;
    const int d = __popcll(__ballot(c0 >= left)) + __popcll(__ballot(c1 >= left)) +
                  __popcll(__ballot(c2 >= left)) + __popcll(__ballot(c3 >= left)) - 1;
    uint32_t taken = 0u;  // keys whose digit is > d
    if (d < 255) {
      const int i = (d + 1) & 3;
      const uint32_t c = i == 0 ? c0 : i == 1 ? c1 : i == 2 ? c2 : c3;
      taken = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(c), (d + 1) >> 2));
    }
    left -= taken;
    prefix |= static_cast<uint32_t>(d) << shift;
    fixed |= 255u << shift;
  }
  T = prefix;
  q = static_cast<int>(left);
}

// Selection and ordered compaction of a long row by the four waves: wave w
// holds positions (w S + r) 64 + lane, r < S, so the waves' positions are
// in wave order.  After the threshold, each wave's counts of keys above it
// and equal to it meet in LDS; a wave's first kept index and first tie rank
// are the counts of the waves before it.  Every wave of the workgroup calls
// this (it holds barriers).
template <int S>
__device__ __forceinline__ void wide_select(const float (&x)[S], long long n, int kb, int lane, int wave,
                                            uint32_t* hist, int (*cnt)[4], int32_t* s_idx) {
  uint32_t key[S];
  uint64_t valid[S];
#pragma unroll
  for (int r = 0; r < S; ++r) {
    const int pos = (wave * S + r) * 64 + lane;
    const bool v = pos >= 1 && pos < n;
    key[r] = v ? keep_key(x[r]) : 0u;
    valid[r] = __ballot(v);
  }
  const int need = kb - 1;
  uint32_t T = 0xFFFFFFFFu;  // need == 0: nothing compares above or equal
  int q = 0;
  if (need > 0) block_digit_threshold<S>(key, valid, need, hist, lane, wave, T, q);
  int n_above = 0, n_tie = 0;
#pragma unroll
  for (int r = 0; r < S; ++r) {
    const bool is_valid = (valid[r] >> lane) & 1ull;
    n_above += __popcll(__ballot(is_valid && key[r] > T));
    n_tie += __popcll(__ballot(is_valid && key[r] == T));
  }
  if (lane == 0) {
    cnt[0][wave] = n_above;
    cnt[1][wave] = n_tie;
  }
  __syncthreads();
  int cum_eq = 0, cum_keep = wave > 0 ? 1 : 0;  // CLS (position 0) is wave 0's
  for (int w = 0; w < wave; ++w) {
    const int t = cnt[1][w];
    cum_keep += cnt[0][w] + min(max(q - cum_eq, 0), t);
    cum_eq += t;
  }
#pragma unroll
  for (int r = 0; r < S; ++r) {
    const int pos = (wave * S + r) * 64 + lane;
    const bool is_valid = (valid[r] >> lane) & 1ull;
    const bool above = is_valid && key[r] > T;
    const bool tie = is_valid && key[r] == T;
    const uint64_t tie_mask = __ballot(tie);
    const bool kept = pos == 0 || above || (tie && cum_eq + lanes_below(tie_mask) < q);
    const uint64_t kept_mask = __ballot(kept);
    if (kept) s_idx[cum_keep + lanes_below(kept_mask)] = pos;
    cum_eq += __popcll(tie_mask);
    cum_keep += __popcll(kept_mask);
  }
}

// What the copy writes for one 16-byte piece of a kept row.
enum PackMode { kCopy = 0, kAddBf16 = 1, kAddF32 = 2 };

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// tokens + addend for 8 bf16 or 4 fp32 values: the sum is formed in fp32 and
// rounded once to the token type (round to nearest even).
template <int MODE>
__device__ __forceinline__ u32x4 combine(uint4 x, uint4 y) {
  if constexpr (MODE == kCopy) {
    return u32x4{x.x, x.y, x.z, x.w};
  } else if constexpr (MODE == kAddF32) {
    return u32x4{__float_as_uint(__uint_as_float(x.x) + __uint_as_float(y.x)),
                 __float_as_uint(__uint_as_float(x.y) + __uint_as_float(y.y)),
                 __float_as_uint(__uint_as_float(x.z) + __uint_as_float(y.z)),
                 __float_as_uint(__uint_as_float(x.w) + __uint_as_float(y.w))};
  } else {
    const uint32_t a[4] = {x.x, x.y, x.z, x.w}, b[4] = {y.x, y.y, y.z, y.w};
    u32x4 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float lo = __uint_as_float(a[i] << 16) + __uint_as_float(b[i] << 16);
      const float hi = __uint_as_float(a[i] & 0xFFFF0000u) + __uint_as_float(b[i] & 0xFFFF0000u);
      const bf16x2 v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
      r[i] = __builtin_bit_cast(uint32_t, v);
    }
    return r;
  }
}

template <int SLOTS, int MODE>
__device__ __forceinline__ void select_pack_body(const SelectPackParams& p) {
  // Rows of more than 256 tokens are selected by all four waves, a quarter
  // of the positions each (kWide); shorter rows by wave 0 alone.
  constexpr bool kWide = SLOTS >= kDigitSelectSlots;
  constexpr int kSel = kWide ? SLOTS / 4 : SLOTS;  // score slots per lane of a selecting wave
  __shared__ int32_t s_idx[SLOTS * 64];
  __shared__ __align__(16) uint32_t s_hist[kWide ? 2 * 4 * 256 : 1];  // digit histograms of the long-row select
  __shared__ int s_cnt[2][4];                    // long rows: per wave, keys above and at the threshold
  __shared__ long long s_part[kThreads / 64];
  __shared__ long long s_before[kThreads / 64];  // plan items of the sequences with more chunks than b
  __shared__ int s_rank[kThreads / 64];          // sequences of b's chunk count ordered before b
  __shared__ int s_members[kThreads / 64];       // sequences of b's chunk count
  __shared__ long long s_items[kThreads / 64];   // plan items of all sequences
  __shared__ long long s_kept[kThreads / 64];    // sum of all keep counts
  __shared__ int s_bad[kThreads / 64];           // some keep count outside [1, max_seqlen]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int b = blockIdx.x / p.split;
  const int s = blockIdx.x - b * p.split;

  // Segment of image b in the input.
  long long off_in, n;
  bool seg_ok = true;
  if (p.cu_in != nullptr) {
    const long long a = p.cu_in[b], e = p.cu_in[b + 1];
    off_in = a;
    n = e - a;
    seg_ok = a >= 0 && e <= p.total_in && n >= 1 && n <= p.N && (b != 0 || a == 0);
  } else {
    off_in = static_cast<long long>(b) * p.N;
    n = p.N;
  }
  const int kb = p.keep[b];
  const long long cu_b = p.cu_ready ? static_cast<long long>(p.cu_out[b]) : 0;
  // Wave 0's score loads go out before the keep count is checked: they
  // depend on the segment only, so they overlap the keep count's load instead
  // of following it.  All SLOTS loads are issued before the first is used:
  // positions past the segment read its last score (they are not
  // candidates), and the empty asm consumes every loaded value, so the
  // compiler cannot sink a load into the branch of its only use, where each
  // would wait alone.
  float x[kSel];
  if ((kWide || wave == 0) && seg_ok) {
    const long long last = off_in + n - 1;
    const int g0 = kWide ? wave * kSel : 0;  // the wave's first slot
#pragma unroll
    for (int r = 0; r < kSel; ++r) x[r] = p.scores[min(off_in + (g0 + r) * 64 + lane, last)];
#pragma unroll
    for (int r = 0; r < kSel; ++r) asm volatile("" : "+v"(x[r]));
  }
  const bool img_ok = seg_ok && kb >= 1 && kb <= n;
  // With a plan, workgroup (b, 0) writes image b's attention items and
  // workgroup (0, 0) the plan header.
  const bool plan_img = p.plan_hdr != nullptr && s == 0;
  const bool plan_head = p.plan_hdr != nullptr && blockIdx.x == 0;

  // Waves 1-3: output offset of image b, keep[0] + ... + keep[b-1].  For the
  // plan (queue order: longer sequences first, then lower index), b's class
  // of sequences with its chunk count starts after the items of every
  // sequence with more chunks; inside the class b's rank is the number of
  // class members ordered before it.
  auto sum_keeps = [&]() {
    long long part = 0, before = 0, items = 0, kept = 0;
    int rank = 0, members = 0, bad = 0;
    const int chb = kb >= 1 && kb <= p.max_seqlen ? attn_chunks(kb) : 0;
    const int jend = plan_img ? p.B : b;
    for (int j = tid - 64; j < jend; j += kThreads - 64) {
      const int kj = p.keep[j];
      if (j < b) part += kj;
      if (plan_img) {
        const bool fits = kj >= 1 && kj <= p.max_seqlen;
        const int chj = fits ? attn_chunks(kj) : 0;
        if (chj > chb) before += p.H * chj;
        if (fits && chj == chb) {
          ++members;
          rank += kj > kb || (kj == kb && j < b);
        }
        if (plan_head) {
          items += p.H * chj;
          kept += kj;
          bad |= !fits;
        }
      }
    }
    part = wave_sum(part);
    if (lane == 0) s_part[wave] = part;
    if (plan_img) {
      before = wave_sum(before);
      const long long rk = wave_sum(static_cast<long long>(rank));
      const long long mb = wave_sum(static_cast<long long>(members));
      if (lane == 0) {
        s_before[wave] = before;
        s_rank[wave] = static_cast<int>(rk);
        s_members[wave] = static_cast<int>(mb);
      }
    }
    if (plan_head) {
      items = wave_sum(items);
      kept = wave_sum(kept);
      bad = __ballot(bad != 0) != 0ull;
      if (lane == 0) {
        s_items[wave] = items;
        s_kept[wave] = kept;
        s_bad[wave] = bad;
      }
    }
  };
  if constexpr (!kWide) {
    if (wave != 0) {
      if (!p.cu_ready) sum_keeps();
    } else if (img_ok) {
      // Candidates are positions 1..n-1 (CLS, position 0, is not a candidate).
      // Position pos = r*64 + lane lives in key[r] of that lane (score x[r],
      // loaded above).
      uint32_t key[SLOTS];
      uint64_t valid[SLOTS];
#pragma unroll
      for (int r = 0; r < SLOTS; ++r) {
        const int pos = r * 64 + lane;
        const bool v = pos >= 1 && pos < n;
        key[r] = v ? keep_key(x[r]) : 0u;
        valid[r] = __ballot(v);
      }
      // Threshold T = the need-th largest candidate key; q = how many of the
      // candidates equal to T are kept (the lowest positions among them).
      const int need = kb - 1;
      uint32_t T = 0xFFFFFFFFu;  // need == 0: nothing compares above or equal
      int q = 0;
      if (need > 0) {
        T = 0u;
        for (int bit = 31; bit >= 0; --bit) {
          const uint32_t t = T | (1u << bit);
          int cnt = 0;
#pragma unroll
          for (int r = 0; r < SLOTS; ++r) cnt += __popcll(__ballot(key[r] >= t));  // t >= 1: invalid keys (0) never count
          if (cnt >= need) T = t;
        }
        int gt = 0;
#pragma unroll
        for (int r = 0; r < SLOTS; ++r) gt += __popcll(__ballot(key[r] > T) & valid[r]);
        q = need - gt;
      }
      // Ordered compaction: kept positions in ascending order.
      int cum_eq = 0, cum_keep = 0;
#pragma unroll
      for (int r = 0; r < SLOTS; ++r) {
        const int pos = r * 64 + lane;
        const bool is_valid = (valid[r] >> lane) & 1ull;
        const bool above = is_valid && key[r] > T;
        const bool tie = is_valid && key[r] == T;
        const uint64_t tie_mask = __ballot(tie);
        const bool kept = pos == 0 || above || (tie && cum_eq + lanes_below(tie_mask) < q);
        const uint64_t kept_mask = __ballot(kept);
        if (kept) s_idx[cum_keep + lanes_below(kept_mask)] = pos;
        cum_eq += __popcll(tie_mask);
        cum_keep += __popcll(kept_mask);
      }
    }
  } else {
    if (wave != 0 && !p.cu_ready) sum_keeps();
    if (img_ok) wide_select<kSel>(x, n, kb, lane, wave, s_hist, s_cnt, s_idx);  // img_ok: uniform in the workgroup
  }
  __syncthreads();
  const long long off_out = p.cu_ready ? cu_b : s_part[1] + s_part[2] + s_part[3];

  if (plan_img && kb >= 1 && kb <= p.max_seqlen) {
    // Items (b, h, c) for head h and query chunk c, each in its slot of the
    // class (attn_item_slot).
    const long long cls_base = s_before[1] + s_before[2] + s_before[3];
    const int rank = s_rank[1] + s_rank[2] + s_rank[3];
    const int groups = (s_members[1] + s_members[2] + s_members[3]) * p.H;
    const int ch = attn_chunks(kb);
    for (int i = tid; i < p.H * ch; i += kThreads) {
      const int h = i / ch, c = i - h * ch;
      const long long slot = attn_item_slot(cls_base, groups, ch, rank * p.H + h, c);
      if (slot < p.max_items) p.plan_items[slot] = encode_item(static_cast<int>(off_out), kb, h, c);
    }
  }
  if (plan_head) {
    if (tid < 32) p.plan_hdr->zero_row[tid] = 0u;
    if (tid == 0) {
      const bool bad = s_bad[1] | s_bad[2] | s_bad[3] || s_kept[1] + s_kept[2] + s_kept[3] > p.plan_total;
      if (bad) atomicOr(p.status, DORA_DEV_CU_SEQLENS);
      write_plan_header(p.plan_hdr, bad ? 0 : static_cast<int>(s_items[1] + s_items[2] + s_items[3]), p.B, p.H,
                        p.max_seqlen, p.plan_total);
    }
  }
  if (!img_ok) {
    if (s == 0 && tid == 0) atomicOr(p.status, seg_ok ? DORA_DEV_KEEP_RANGE : DORA_DEV_CU_IN);
    return;
  }

  if (s == 0) {
    if (tid == 0) {
      if (off_out + kb > p.cap_rows) atomicOr(p.status, DORA_DEV_CAPACITY);
      if (!p.cu_ready) {
        p.cu_out[b + 1] = static_cast<int32_t>(off_out + kb);
        if (b == 0) p.cu_out[0] = 0;
      }
    }
    for (int i = tid; i < kb; i += kThreads) {
      const long long row = off_out + i;
      if (row >= 0 && row < p.cap_rows) p.idx_out[row] = s_idx[i];
    }
  }

  // This workgroup's share of the kept rows.
  const int rows_per = (kb + p.split - 1) / p.split;
  const int r0 = s * rows_per;
  const int r1 = min(kb, r0 + rows_per);
  if (r0 >= r1) return;
  const int vpr = p.row_vecs;
  const int nvec = (r1 - r0) * vpr;
  const int step_rows = kThreads / vpr;
  const int step_vecs = kThreads - step_rows * vpr;
  int row = tid / vpr;
  int vec = tid - row * vpr;
  // Stores go through a buffer resource based at this workgroup's first
  // output row (offsets below 2^31: at most N rows of at most 1 MB); a row at
  // or past cap_rows gets an offset past the resource and is dropped.
  const __amdgpu_buffer_rsrc_t out = raw_buffer(p.packed + (off_out + r0) * vpr);
  for (int base = tid; base < nvec; base += kThreads * kCopyUnroll) {
    uint4 buf[kCopyUnroll], add[kCopyUnroll];
    uint32_t dst[kCopyUnroll];
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) {
      const bool in_range = base + u * kThreads < nvec;
      const int pos = s_idx[in_range ? r0 + row : r0];
      const long long src_row = off_in + min(max(pos, 0), static_cast<int>(n) - 1);  // always inside the segment
      const long long out_row = off_out + r0 + row;
      buf[u] = in_range ? p.tokens[src_row * vpr + vec] : make_uint4(0u, 0u, 0u, 0u);
      if constexpr (MODE != kCopy) add[u] = in_range ? p.addend[src_row * vpr + vec] : make_uint4(0u, 0u, 0u, 0u);
      dst[u] = (in_range && out_row >= 0 && out_row < p.cap_rows) ? static_cast<uint32_t>(row * vpr + vec) * 16u
                                                                   : 0xFFFFFFF0u;
      row += step_rows;
      vec += step_vecs;
      if (vec >= vpr) {
        vec -= vpr;
        ++row;
      }
    }
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) store_through(out, dst[u], combine<MODE>(buf[u], add[u]));
  }
}

// One workgroup per (image, split) piece.  The plain variant copies rows; the
// residual variant writes h + a of each kept row.
template <int SLOTS>
__global__ __launch_bounds__(kThreads) void select_pack_kernel(SelectPackParams p) {
  select_pack_body<SLOTS, kCopy>(p);
}

template <int SLOTS, int MODE>
__global__ __launch_bounds__(kThreads) void select_pack_residual_kernel(SelectPackParams p) {
  select_pack_body<SLOTS, MODE>(p);
}

__device__ __forceinline__ long long wave_inclusive_scan64(long long v, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const long long t = __shfl_up(v, off, 64);
    if (lane >= off) v += t;
  }
  return v;
}

// Running total of the keep counts (Sec. 3.5 "Inference": the boundaries of
// the packed buffer): cu_out[0] = 0, cu_out[b+1] = keep[0] + ... + keep[b],
// held at the int32 range (a total past it is a capacity error either way).
// One workgroup walks the counts in tiles of kScanThreads * kScanPer: each
// thread sums its kScanPer counts, a block scan of those sums gives every
// thread's starting total, and a carry joins the tiles.
__global__ __launch_bounds__(kScanThreads) void keep_scan_kernel(const int32_t* keep, int32_t B, int32_t* cu_out) {
  __shared__ long long s_wave[kScanThreads / 64];
  __shared__ long long s_carry;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) {
    s_carry = 0;
    cu_out[0] = 0;
  }
  __syncthreads();
  for (long long base = 0; base < B; base += static_cast<long long>(kScanThreads) * kScanPer) {
    const long long first = base + static_cast<long long>(tid) * kScanPer;
    long long v[kScanPer];
    long long sum = 0;
#pragma unroll
    for (int i = 0; i < kScanPer; ++i) {
      v[i] = first + i < B ? keep[first + i] : 0;
      sum += v[i];
    }
    const long long incl = wave_inclusive_scan64(sum, lane);
    if (lane == 63) s_wave[wave] = incl;
    __syncthreads();
    if (wave == 0) {
      const long long x = lane < kScanThreads / 64 ? s_wave[lane] : 0;
      const long long xi = wave_inclusive_scan64(x, lane);
      if (lane < kScanThreads / 64) s_wave[lane] = xi - x;
    }
    __syncthreads();
    long long run = s_carry + s_wave[wave] + incl - sum;
#pragma unroll
    for (int i = 0; i < kScanPer; ++i) {
      run += v[i];
      if (first + i < B) cu_out[first + i + 1] = static_cast<int32_t>(max(min(run, static_cast<long long>(INT_MAX)),
                                                                             static_cast<long long>(INT_MIN)));
    }
    __syncthreads();
    if (tid == kScanThreads - 1) s_carry = run;
    __syncthreads();
  }
}

template <int SLOTS>
hipError_t launch(const SelectPackParams& p, int mode, hipStream_t stream) {
  const dim3 grid(p.B * p.split), block(kThreads);
  if (mode == kAddBf16)
    hipLaunchKernelGGL((select_pack_residual_kernel<SLOTS, kAddBf16>), grid, block, 0, stream, p);
  else if (mode == kAddF32)
    hipLaunchKernelGGL((select_pack_residual_kernel<SLOTS, kAddF32>), grid, block, 0, stream, p);
  else
    hipLaunchKernelGGL(select_pack_kernel<SLOTS>, grid, block, 0, stream, p);
  return hipGetLastError();
}

int pick_split(int B, int N) {
  int split = (1024 + B - 1) / B;  // ~4 workgroups per compute unit
  const int max_split = N / 16 > 1 ? N / 16 : 1;  // at least ~16 rows per workgroup
  if (split > max_split) split = max_split;
  if (split < 1) split = 1;
  while (static_cast<long long>(split) * B > INT_MAX) --split;
  return split;
}

// Checks the arguments of a select/pack call and fills `p` (no plan).
int prepare(const float* scores, const int32_t* keep, const void* tokens, const int32_t* cu_in, int64_t total_in,
            int32_t B, int32_t N, int32_t C, dora_dtype dtype, int32_t* idx_out, int32_t* cu_out, void* packed_out,
            int64_t cap_rows, int32_t* dev_status, SelectPackParams* p) {
  if (!scores || !keep || !tokens || !idx_out || !cu_out || !packed_out || !dev_status) return DORA_ERR_NULL;
  if (dtype != DORA_F32 && dtype != DORA_BF16) return DORA_ERR_DTYPE;
  if (B < 1 || N < 1 || N > DORA_MAX_ROW_TOKENS || C < 1) return DORA_ERR_SHAPE;
  if (cu_in != nullptr && total_in < 0) return DORA_ERR_SHAPE;
  const int64_t row_bytes = static_cast<int64_t>(C) * (dtype == DORA_F32 ? 4 : 2);
  if (row_bytes % 16 != 0) return DORA_ERR_ALIGN;
  if (row_bytes > (int64_t(1) << 20)) return DORA_ERR_UNSUPPORTED;
  if ((reinterpret_cast<uintptr_t>(tokens) | reinterpret_cast<uintptr_t>(packed_out)) & 15u) return DORA_ERR_ALIGN;
  if (cap_rows < 1 || cap_rows > INT_MAX) return DORA_ERR_CAPACITY;

  p->scores = scores;
  p->keep = keep;
  p->tokens = static_cast<const uint4*>(tokens);
  p->addend = nullptr;
  p->cu_in = cu_in;
  p->total_in = total_in;
  p->B = B;
  p->N = N;
  p->row_vecs = static_cast<int32_t>(row_bytes / 16);
  p->split = pick_split(B, N);
  p->idx_out = idx_out;
  p->cu_out = cu_out;
  p->packed = static_cast<uint4*>(packed_out);
  p->cap_rows = cap_rows;
  p->status = dev_status;
  p->plan_hdr = nullptr;
  p->plan_items = nullptr;
  p->H = p->max_seqlen = p->max_items = 0;
  p->plan_total = 0;
  p->cu_ready = 0;
  return DORA_OK;
}

int launch_select_pack(SelectPackParams p, void* stream, int mode = kCopy) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t err;
  if (p.B > kFusedScanMaxB) {
    // Large batch: the block scan writes cu_out first; a plan is then built
    // from cu_out by the attention plan kernel (sequences of at least one row).
    hipLaunchKernelGGL(keep_scan_kernel, dim3(1), dim3(kScanThreads), 0, st, p.keep, p.B, p.cu_out);
    if (hipGetLastError() != hipSuccess) return DORA_ERR_HIP;
    if (p.plan_hdr != nullptr) {
      const int rc = launch_attn_plan(p.cu_out, p.B, p.H, p.max_seqlen, p.plan_total, 1, p.plan_hdr, p.status, stream);
      if (rc != DORA_OK) return rc;
      p.plan_hdr = nullptr;
      p.plan_items = nullptr;
    }
    p.cu_ready = 1;
  }
  if (p.N <= 64) err = launch<1>(p, mode, st);
  else if (p.N <= 128) err = launch<2>(p, mode, st);
  else if (p.N <= 256) err = launch<4>(p, mode, st);
  else if (p.N <= 512) err = launch<8>(p, mode, st);
  else if (p.N <= 1024) err = launch<16>(p, mode, st);
  else err = launch<32>(p, mode, st);
  return err == hipSuccess ? DORA_OK : DORA_ERR_HIP;
}

}  // namespace
}  // namespace dora

extern "C" int dora_select_pack(const float* scores, const int32_t* keep, const void* tokens,
                                const int32_t* cu_in, int64_t total_in, int32_t B, int32_t N,
                                int32_t C, dora_dtype dtype, int32_t* idx_out, int32_t* cu_out,
                                void* packed_out, int64_t cap_rows, int32_t* dev_status,
                                void* stream) {
  using namespace dora;
  SelectPackParams p;
  const int rc = prepare(scores, keep, tokens, cu_in, total_in, B, N, C, dtype, idx_out, cu_out, packed_out,
                         cap_rows, dev_status, &p);
  if (rc != DORA_OK) return rc;
  return launch_select_pack(p, stream);
}

extern "C" int dora_select_pack_plan(const float* scores, const int32_t* keep, const void* tokens,
                                     const int32_t* cu_in, int64_t total_in, int32_t B, int32_t N,
                                     int32_t C, dora_dtype dtype, int32_t* idx_out, int32_t* cu_out,
                                     void* packed_out, int64_t cap_rows, int32_t H, int32_t max_seqlen,
                                     int64_t total, void* workspace, size_t workspace_bytes,
                                     int32_t* dev_status, void* stream) {
  using namespace dora;
  SelectPackParams p;
  int rc = prepare(scores, keep, tokens, cu_in, total_in, B, N, C, dtype, idx_out, cu_out, packed_out, cap_rows,
                   dev_status, &p);
  if (rc != DORA_OK) return rc;
  rc = check_attn_sizes(B, H, max_seqlen, total);
  if (rc != DORA_OK) return rc;
  const AttnWorkspaceLayout L = attn_workspace_layout(B, H, max_seqlen);
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) || workspace_bytes < L.bytes)
    return DORA_ERR_WORKSPACE;
  p.plan_hdr = static_cast<AttnPlanHeader*>(workspace);
  p.plan_items = reinterpret_cast<int2*>(static_cast<char*>(workspace) + L.items_off);
  p.H = H;
  p.max_seqlen = max_seqlen;
  p.max_items = static_cast<int32_t>(L.max_items);
  p.plan_total = total;
  return launch_select_pack(p, stream);
}

extern "C" int dora_select_pack_residual(const float* scores, const int32_t* keep, const void* h,
                                         const void* a, const int32_t* cu_in, int64_t total_in, int32_t B,
                                         int32_t N, int32_t C, dora_dtype dtype, int32_t* idx_out,
                                         int32_t* cu_out, void* packed_out, int64_t cap_rows,
                                         int32_t* dev_status, void* stream) {
  using namespace dora;
  SelectPackParams p;
  const int rc = prepare(scores, keep, h, cu_in, total_in, B, N, C, dtype, idx_out, cu_out, packed_out, cap_rows,
                         dev_status, &p);
  if (rc != DORA_OK) return rc;
  if (!a) return DORA_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(a) & 15u) return DORA_ERR_ALIGN;
  p.addend = static_cast<const uint4*>(a);
  return launch_select_pack(p, stream, dtype == DORA_BF16 ? kAddBf16 : kAddF32);
}
