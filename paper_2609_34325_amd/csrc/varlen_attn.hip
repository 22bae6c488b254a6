// Variable-length multi-head attention over the packed buffer.
// DORA (arXiv 2609.34325), Sec. 3.5 "Inference" and App. E.5: survivors of
// all images are packed with explicit sequence boundaries and processed by
// exact softmax attention that never crosses a boundary (no mask beyond the
// boundaries, no bias, no token-size term).
//
// Work decomposition (persistent, queue-driven):
//   plan     one workgroup validates cu_seqlens, orders the sequences by
//            decreasing length (counting sort) and writes the item list
//            (sequence, head, chunk of kAttnQTile queries), each item
//            carrying its first row and length so the executing kernel needs
//            no other lookup; it also resets the queue counters.
//   execute  persistent workgroups, as many as fit on the device, take item
//            tickets from an atomic counter until the list is drained; the
//            last workgroup to leave resets the counters so the plan can run
//            again (e.g. for every layer between two pruning steps).
//
// bf16 kernel, per work item: each of the 12 waves owns one 16-query tile of
// the chunk (three waves per SIMD: with one tile each a wave needs about 170
// registers, so three fit where two-tile waves fit only two, and the extra
// wave per SIMD overlaps more of the softmax with the matrix products).  K and V (row-major) stream through LDS in stages of kKRes keys by
// LDS DMA, double-buffered, so the transfer of the next stage (the rest of
// this item, or the next item) overlaps the MFMA work of the current one; the
// next item's queries also arrive in LDS by DMA, and the queue ticket and
// descriptor of the item after it are fetched one stage ahead.
//
// V^T operands come from the transposing LDS read (ds_read_b64_tr_b16), so V
// needs no transpose on its way into LDS.
// S^T = K Q^T is computed with v_mfma_f32_16x16x32_bf16 so each lane owns one
// query column and the softmax reductions over keys stay mostly in-lane; the
// online softmax runs in fp32 with exp2 of one FMA per score (scale*log2(e)
// folded in) and lazy rescaling; P is rounded to bf16 and O^T += V^T P^T takes
// the S^T output registers directly as its B operand (the key order inside a
// 32-key step is permuted the same way on both operands).  The softmax
// denominators come from the matrix unit as well: a block of ones times P^T.
#include <limits.h>
#include <math.h>

#include <atomic>

#include "dora_internal.h"

namespace dora {
namespace {

constexpr int kD = 64;
constexpr int kWaves = 12;
constexpr int kThreads = kWaves * 64;
constexpr int kTilesPerWave = 1;  // 16-query tiles per wave (1 or 2)
static_assert(kTilesPerWave == 1 || kTilesPerWave == 2, "tiles per wave");
static_assert(kWaves * kTilesPerWave * 16 >= kAttnQTile && kAttnQTile % 16 == 0, "tile size");
// fp32 kernel: a workgroup of 4 waves takes one part of 64 queries (a
// 16-query tile per wave) of an item; an item is kF32Parts tickets, so a
// short batch still spreads over many compute units.
constexpr int kF32Waves = 4;
constexpr int kF32Threads = kF32Waves * 64;
constexpr int kF32PartQ = kF32Waves * 16;
constexpr int kF32Parts = (kAttnQTile + kF32PartQ - 1) / kF32PartQ;
constexpr int kKRes = 256;             // keys resident in LDS per stage (bf16)
// Lane 0 of the last wave talks to the queue: the last wave holds the fewest
// query tiles of an item, so the queue's latency lands where there is slack.
constexpr int kQueueThread = kThreads - 64;
constexpr int kPlanThreads = 1024;
constexpr int kPlanMaxChunks = (DORA_MAX_SEQLEN + kAttnQTile - 1) / kAttnQTile;  // chunks of the longest sequence
constexpr int kPlanBins = 1024;
constexpr float kLog2e = 1.4426950408889634f;

struct PlanParams {
  const int32_t* cu;
  int32_t B, H, max_seqlen;
  int32_t min_len;  // shortest valid sequence (0; 1 for the plan of a select/pack output)
  int64_t total;
  AttnPlanHeader* hdr;
  int2* items;
  int32_t* status;
};

struct AttnParams {
  const void* q;
  const void* k;
  const void* v;
  void* out;
  int32_t B, H, max_seqlen;
  int64_t total;
  float scale_log2;  // softmax_scale * log2(e)
  AttnPlanHeader* hdr;
  const int2* items;
  int32_t max_items;  // capacity of items[] in this workspace
  int32_t* status;
};

// ------------------------------- plan -------------------------------------

__device__ __forceinline__ int wave_inclusive_scan(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int t = __shfl_up(v, off, 64);
    if (lane >= off) v += t;
  }
  return v;
}

// Exclusive scan of one value per thread across the 1024-thread block.
__device__ int block_exclusive_scan(int v, int* wave_sums, int* total) {
  constexpr int kW = kPlanThreads / 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int incl = wave_inclusive_scan(v);
  if (lane == 63) wave_sums[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    const int x = lane < kW ? wave_sums[lane] : 0;
    const int xi = wave_inclusive_scan(x);
    if (lane < kW) wave_sums[lane] = xi - x;
    if (lane == kW - 1) wave_sums[kW] = xi;
  }
  __syncthreads();
  const int r = incl - v + wave_sums[wave];
  *total = wave_sums[kW];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(kPlanThreads) void attn_plan_kernel(PlanParams p) {
  __shared__ int32_t s_cu[kPlanMaxB + 1];  // cu_seqlens, read from global memory once
  __shared__ int hist[kPlanBins];
  __shared__ uint32_t order[kPlanMaxB];  // sequence | len << 13, by decreasing length
  __shared__ int base[kPlanMaxB + 1];    // first item of each sorted position
  __shared__ int wave_sums[kPlanThreads / 64 + 1];
  __shared__ int cls_lo[kPlanMaxChunks + 1], cls_hi[kPlanMaxChunks + 1];  // class bounds by chunk count
  __shared__ int s_bad;
  const int tid = threadIdx.x;
  // Length bins: bin 0 for empty sequences, then (len - 1) >> shift + 1.
  // The smallest shift that fits is at most 5 (max_seqlen <= 16384), and
  // 2^shift divides kAttnQTile, so a bin never straddles a chunk boundary and
  // the sequences of equal chunk count stay contiguous in the sorted order.
  int shift = 0;
  while (((p.max_seqlen - 1) >> shift) + 1 >= kPlanBins) ++shift;
  auto bin_of = [shift](int len) { return len == 0 ? 0 : ((len - 1) >> shift) + 1; };

  for (int i = tid; i < kPlanBins; i += kPlanThreads) hist[i] = 0;
  for (int i = tid; i <= p.B; i += kPlanThreads) s_cu[i] = p.cu[i];
  if (tid == 0) s_bad = 0;
  __syncthreads();
  for (int b = tid; b < p.B; b += kPlanThreads) {
    const long long a = s_cu[b], e = s_cu[b + 1];
    const long long len = e - a;
    if (a < 0 || e > p.total || len < p.min_len || len > p.max_seqlen || (b == 0 && a != 0)) s_bad = 1;
    else atomicAdd(&hist[bin_of(static_cast<int>(len))], 1);
  }
  __syncthreads();
  if (s_bad) {
    if (tid == 0) {
      atomicOr(p.status, DORA_DEV_CU_SEQLENS);
      write_plan_header(p.hdr, 0, p.B, p.H, p.max_seqlen, p.total);
    }
    return;
  }

  // Counting sort by length, longest first.
  {
    const int bin = kPlanBins - 1 - tid;
    int unused;
    const int start = block_exclusive_scan(hist[bin], wave_sums, &unused);
    hist[bin] = start;
  }
  __syncthreads();
  for (int b = tid; b < p.B; b += kPlanThreads) {
    const int len = s_cu[b + 1] - s_cu[b];
    const int pos = atomicAdd(&hist[bin_of(len)], 1);
    order[pos] = static_cast<uint32_t>(b) | (static_cast<uint32_t>(len) << 13);
  }
  __syncthreads();

  // Items per sorted position, then their offsets.
  const int per = (p.B + kPlanThreads - 1) / kPlanThreads;
  int local = 0;
  for (int i = 0; i < per; ++i) {
    const int pos = tid * per + i;
    if (pos < p.B) local += p.H * attn_chunks(static_cast<int>(order[pos] >> 13));
  }
  int n_items;
  int run = block_exclusive_scan(local, wave_sums, &n_items);
  for (int i = 0; i < per; ++i) {
    const int pos = tid * per + i;
    if (pos < p.B) {
      base[pos] = run;
      run += p.H * attn_chunks(static_cast<int>(order[pos] >> 13));
    }
  }
  if (tid == 0) base[p.B] = n_items;
  __syncthreads();

  // Class bounds: sorted positions [cls_lo[ch], cls_hi[ch]) hold the
  // sequences of ch chunks (chunk counts fall with position).
  auto chunks_at = [&](int pos) { return attn_chunks(static_cast<int>(order[pos] >> 13)); };
  for (int pos = tid; pos < p.B; pos += kPlanThreads) {
    const int ch = chunks_at(pos);
    if (pos == 0 || chunks_at(pos - 1) != ch) cls_lo[ch] = pos;
    if (pos == p.B - 1 || chunks_at(pos + 1) != ch) cls_hi[ch] = pos + 1;
  }
  __syncthreads();
  // Emit, one sorted position per thread at a time: its H x chunks items go
  // to their slots in the class (attn_item_slot).
  for (int pos = tid; pos < p.B; pos += kPlanThreads) {
    const uint32_t o = order[pos];
    const int b = static_cast<int>(o & 0x1FFFu);
    const int len = static_cast<int>(o >> 13);
    const int ch = attn_chunks(len);
    if (ch == 0) continue;
    const int c0 = cls_lo[ch];
    const int groups = (cls_hi[ch] - c0) * p.H;
    const long long cbase = base[c0];
    for (int h = 0; h < p.H; ++h)
      for (int c = 0; c < ch; ++c)
        p.items[attn_item_slot(cbase, groups, ch, (pos - c0) * p.H + h, c)] = encode_item(s_cu[b], len, h, c);
  }
  if (tid < 32) p.hdr->zero_row[tid] = 0u;
  if (tid == 0) write_plan_header(p.hdr, n_items, p.B, p.H, p.max_seqlen, p.total);
}

// ------------------------------ execute -----------------------------------

struct Item {
  int seq0, len, h, chunk;
};

__device__ __forceinline__ bool plan_matches(const AttnParams& p) {
  const AttnPlanHeader* h = p.hdr;
  return h->magic == kPlanMagic && h->B == p.B && h->H == p.H && h->max_seqlen == p.max_seqlen &&
         h->q_tile == kAttnQTile && h->total == p.total;
}

// Decodes an item; an item that does not fit the sizes (a stale plan) is
// reported and replaced by an empty one so that nothing is read or written.
__device__ __forceinline__ Item decode_item(const AttnParams& p, int2 raw) {
  Item it;
  const uint32_t y = static_cast<uint32_t>(raw.y);
  it.seq0 = raw.x;
  it.len = static_cast<int>(y >> 17);
  it.h = static_cast<int>((y >> 9) & 0xFFu);
  it.chunk = static_cast<int>(y & 0x1FFu);
  const bool ok = raw.x >= 0 && it.len <= p.max_seqlen &&
                  static_cast<long long>(raw.x) + it.len <= p.total && it.h < p.H &&
                  it.chunk < attn_chunks(it.len);
  if (!ok) {
    if (threadIdx.x == 0) atomicOr(p.status, DORA_DEV_CU_SEQLENS);
    it.seq0 = 0;
    it.len = 0;
    it.h = 0;
    it.chunk = 0;
  }
  // Descriptors are the same in every lane; keep them in scalar registers.
  it.seq0 = __builtin_amdgcn_readfirstlane(it.seq0);
  it.len = __builtin_amdgcn_readfirstlane(it.len);
  it.h = __builtin_amdgcn_readfirstlane(it.h);
  it.chunk = __builtin_amdgcn_readfirstlane(it.chunk);
  return it;
}

// An item descriptor read from LDS is the same in every lane; say so, so the
// item's fields and the branches on them stay scalar.
__device__ __forceinline__ int2 uniform_raw(int2 r) {
  return make_int2(__builtin_amdgcn_readfirstlane(r.x), __builtin_amdgcn_readfirstlane(r.y));
}

// Called by every thread of the workgroup.  The last workgroup out resets the
// counters for the next execute.  Each ticket atomic has returned before the
// wave that took it goes on (its result is waited for), so after the barrier
// no ticket of this workgroup is in flight and its exit may be counted; the
// exit count orders nothing else, so there is no fence (the output stores
// drain on their own before the kernel ends).
__device__ __forceinline__ void leave_queue(AttnPlanHeader* hdr) {
  asm volatile("s_barrier" ::: "memory");
  if (threadIdx.x == 0) {
    const int done = atomicAdd(&hdr->exit_count, 1);
    if (done == static_cast<int>(gridDim.x) - 1) {
      for (int q = 0; q < kSubQueues; ++q) atomicExch(&hdr->queue[q].ticket, 0);
      atomicExch(&hdr->exit_count, 0);
    }
  }
}

// ------------------------- bf16 kernel helpers ------------------------------
//
// MFMA 16x16x32 operand layout (lane l, g = l / 16, c = l % 16):
//   A[16 x 32]: lane holds row c, k = 8g .. 8g+7
//   B[32 x 16]: lane holds column c, k = 8g .. 8g+7
//   D[16 x 16]: lane holds column c, rows 4g .. 4g+3
//
// LDS layout of a staged K or V block: up to 256 rows of 128 bytes (64 bf16),
// unpadded, with the eight 16-byte chunks of row r XOR-swizzled (chunk c at
// position c ^ (r & 7)), so the row reads of K and the transposing reads of V
// both spread over all banks.  Rows arrive by LDS DMA (global_load_lds_dwordx4):
// one wave instruction fills 1 KB = 8 consecutive rows, lane l writing
// position l & 7 of row l >> 3, so lane l fetches chunk (l & 7) ^ (l >> 3).
// Two such K/V buffers alternate: the DMA of the next stage fills one while
// the waves compute on the other.

constexpr int kRowBytes = kD * 2;
constexpr int kStageElems = kKRes * kD;

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) const char lds_cchar;

// Byte address of element (row0, head h, dim 0) of a packed [rows, H, 64]
// tensor.  Every argument is the same in all lanes, so this is scalar
// arithmetic and per-lane offsets can stay 32-bit.
__device__ __forceinline__ const char* head_base(const void* X, long long row0, long long row_elems, int h) {
  return static_cast<const char*>(X) + (row0 * row_elems + h * kD) * 2;
}

// Issues the DMA of rows [0, n) of one head's K and V (1 <= n <= 256) into
// Kd / Vd.  Rows up to the next multiple of 64 are filled as well: K with
// copies of row n-1 (their scores repeat a real score, so a block maximum
// taken over them is still a maximum over real keys) and V with zeros read
// from `zrow`, so those keys add nothing to the output; the denominators
// leave them out separately.
__device__ __forceinline__ void kv_dma(const char* kbase, const char* vbase, const char* zrow, int n,
                                       uint32_t row_bytes, uint16_t* Kd, uint16_t* Vd, int w0, int nw) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
  const uint32_t last = static_cast<uint32_t>(n - 1);
  const uint32_t chunk = static_cast<uint32_t>(((lane & 7) ^ (lane >> 3)) * 16);
  const int n8 = ((n + 63) & ~63) / 8;
  // Instruction pair i (8 rows of K, 8 of V) goes to wave w0 + i % nw.
  if (wave < w0) return;
  for (int i = wave - w0; i < n8; i += nw) {
    const int row0 = i * 8;
    const uint32_t row = static_cast<uint32_t>(row0 + (lane >> 3));
    const uint32_t off = min(row, last) * row_bytes + chunk;
    __builtin_amdgcn_global_load_lds(kbase + off, (lds_void*)(Kd + row0 * kD), 16, 0, 0);
    __builtin_amdgcn_global_load_lds(row <= last ? vbase + off : zrow + chunk, (lds_void*)(Vd + row0 * kD), 16,
                                     0, 0);
  }
}

// Per-lane byte offsets into a staged block (relative to the first row of a
// 16- or 32-key step; steps start at multiples of 8 rows, so the swizzle only
// depends on the lane).
struct LdsOffsets {
  uint32_t k0, k1;  // K row c16, dims 8g..8g+7 and 32+8g..32+8g+7
  uint32_t v[4];    // transposing V read for dims 16 dt .. 16 dt + 15
};

__device__ __forceinline__ LdsOffsets lds_offsets() {
  const int lane = threadIdx.x & 63;
  const int c16 = lane & 15, g = lane >> 4;
  LdsOffsets o;
  o.k0 = static_cast<uint32_t>(c16 * kRowBytes + ((g ^ (c16 & 7)) * 16));
  o.k1 = o.k0 ^ 64u;  // chunk g + 4 sits at position (g ^ (c16 & 7)) ^ 4
  // ds_read_b64_tr_b16: lane m = 4e + r of each 16-lane group points at
  // V[row 4g + e][16 dt + 4r .. +3], i.e. chunk 2 dt + r / 2, byte 8 (r & 1).
  const int e = c16 >> 2, r = c16 & 3;
  const int row = 4 * g + e;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
    o.v[dt] = static_cast<uint32_t>(row * kRowBytes + (((2 * dt + (r >> 1)) ^ (row & 7)) * 16) + 8 * (r & 1));
  return o;
}

// Per-lane read pointers into one staged K/V buffer, formed once per stage
// outside the key-block loop, so each read inside it carries only the block
// and step offsets as its immediate.
struct LanePtrs {
  lds_cchar* k0;
  lds_cchar* k1;
  const char* v[4];
};

// The K buffer's LDS address (past the 64 KB that the 16-bit offset field of
// an LDS instruction reaches) is hidden from the compiler, which would
// otherwise fold it into every K read and pay an add for each; this way it
// is added once per stage and each read carries its row offset as the
// immediate.  (The V buffers lie below 64 KB, so their reads need no such
// step; they keep their pointers' provenance, without which the compiler
// makes the transposing V reads wait for the LDS DMA in flight.)
__device__ __forceinline__ LanePtrs lane_ptrs(const char* Ks, const char* Vs, const LdsOffsets& lo) {
  uint32_t kbase = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_cchar*)Ks));
  asm volatile("" : "+s"(kbase));
  LanePtrs lp;
  lp.k0 = reinterpret_cast<lds_cchar*>(static_cast<uintptr_t>(kbase + lo.k0));
  lp.k1 = reinterpret_cast<lds_cchar*>(static_cast<uintptr_t>(kbase + lo.k1));
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) lp.v[dt] = Vs + lo.v[dt];
  return lp;
}

// Four V values of one dimension for four keys, read with the gfx950
// transposing LDS load.  In each group of 16 lanes, lane m = 4e + r points at
// V[row(e)][col0 + 4r .. +3]; lane j then receives V[row(e)][col0 + j] for
// e = 0..3 (the instruction hands lane j element j % 4 of the addresses of
// lanes 4e + j / 4).
__device__ __forceinline__ bf16x4 v_column4(const char* p) {
  typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(const_cast<char*>(p)));
}

// Query tile j of wave w is 16-query tile (w + 8 j) of the item's chunk, so
// the busy waves of a short sequence spread over all four SIMDs.
__device__ __forceinline__ int tile_q(int wave, int j) { return (wave + kWaves * j) * 16; }

// DMA of this wave's query tiles of an item's chunk (chunk rows [0, nq) at
// qbase, 1 <= nq <= kAttnQTile) into the query buffer, swizzled like K: the
// 16 rows of each tile the wave owns, rows past nq-1 filled with copies of row
// nq-1 so every row a tile reads is finite.  Each wave loads and reads only
// its own rows, so no barrier guards the buffer between items.
__device__ __forceinline__ void q_dma(const char* qbase, int nq, uint32_t row_bytes, uint16_t* Qd) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
  const uint32_t last = static_cast<uint32_t>(nq - 1);
  const uint32_t chunk = static_cast<uint32_t>(((lane & 7) ^ (lane >> 3)) * 16);
#pragma unroll
  for (int j = 0; j < kTilesPerWave; ++j) {
    const int t0 = tile_q(wave, j);
    if (t0 < nq) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int row0 = t0 + 8 * h;
        const uint32_t off = min(static_cast<uint32_t>(row0 + (lane >> 3)), last) * row_bytes + chunk;
        __builtin_amdgcn_global_load_lds(qbase + off, (lds_void*)(Qd + row0 * kD), 16, 0, 0);
      }
    }
  }
}

// The queries of an item's chunk into the query buffer (nothing for an empty item).
__device__ __forceinline__ void q_chunk_dma(const AttnParams& p, const Item& it, long long row_elems,
                                            uint32_t row_bytes, uint16_t* Qd) {
  const int cs = attn_chunk_size(it.len);
  const int q0 = it.chunk * cs;
  const int nq = min(cs, it.len - q0);
  if (nq > 0) q_dma(head_base(p.q, static_cast<long long>(it.seq0) + q0, row_elems, it.h), nq, row_bytes, Qd);
}

// B operands of the wave's query tiles from the query buffer: lane (c16, g)
// holds query tile_q + c16, dims 8g..8g+7 (ks = 0) and 32+8g..32+8g+7 (ks = 1).
__device__ __forceinline__ void q_read(const uint16_t* Qs, const LdsOffsets& lo, int nq, bf16x8 (&qf)[2][2]) {
  const int wave = threadIdx.x >> 6;
  const char* base = reinterpret_cast<const char*>(Qs);
#pragma unroll
  for (int j = 0; j < kTilesPerWave; ++j) {
    if (tile_q(wave, j) < nq) {
      const char* t = base + tile_q(wave, j) * kRowBytes;
      qf[j][0] = *reinterpret_cast<const bf16x8*>(t + lo.k0);
      qf[j][1] = *reinterpret_cast<const bf16x8*>(t + lo.k1);
    }
  }
}

// S^T[key][query] for keys kb .. kb+63 of the staged block (kb .. kb+31 for a
// HALF block, the last block of a sequence when at most 32 keys remain): 4 (2)
// key tiles of 16 against query tile 0 (and tile 1 when ACT1).
template <bool ACT1, bool HALF>
__device__ __forceinline__ void qk_block(const LanePtrs& lp, int kb, const bf16x8 (&qf)[2][2],
                                         floatx4 (&s)[2][4]) {
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kt = 0; kt < (HALF ? 2 : 4); ++kt) {
    const int off = (kb + kt * 16) * kRowBytes;
    typedef __attribute__((address_space(3))) const bf16x8 lds_bf16x8;
    const bf16x8 a0 = *reinterpret_cast<lds_bf16x8*>(lp.k0 + off);
    const bf16x8 a1 = *reinterpret_cast<lds_bf16x8*>(lp.k1 + off);
    s[0][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
        a1, qf[0][1], __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, qf[0][0], zero, 0, 0, 0), 0, 0, 0);
    if (ACT1)
      s[1][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
          a1, qf[1][1], __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, qf[1][0], zero, 0, 0, 0), 0, 0, 0);
  }
}

struct SoftmaxState {
  floatx4 o[2][4];  // O^T accumulators: dims dt*16 + 4g .. +3 of the lane's query
  floatx4 l[2];     // softmax denominators (every component holds the same sum)
  float m[2];       // running max, log2 units
};

// Maximum over the four 16-lane rows of the wave: lanes c, c+16, c+32 and
// c+48 hold different keys of the same query column.  Two row swaps
// (v_permlane16_swap, then v_permlane32_swap), no LDS round trip.
__device__ __forceinline__ float row_group_max(float m) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(m), __float_as_uint(m), false, false);
  m = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// Online softmax of one 64-key block (32 keys when HALF) followed by
// O^T += V^T P^T.  FIRST marks an item's first block: the running max starts
// at the block max and the accumulators start from zero.  In a partial block
// (kvalid < 64, or < 32 when HALF) the keys past the end are copies of the
// last key, with zero V rows: they leave every block maximum unchanged and add
// nothing to O, and the denominators skip them (their row of the ones operand
// is zero).
template <bool ACT1, bool FIRST, bool HALF>
__device__ __forceinline__ void softmax_pv_block(const LanePtrs& lp, int kb, int kvalid, float scale_log2,
                                                 const bf16x8& ones, floatx4 (&s)[2][4],
                                                 SoftmaxState& st) {
  constexpr int kTiles = ACT1 ? 2 : 1;
  constexpr int kKt = HALF ? 2 : 4;  // 16-key tiles in the block
  constexpr int kKs = HALF ? 1 : 2;  // 32-key P.V steps in the block
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4;
  // V^T operands of the block's P.V steps, read first (and kept first by a
  // scheduling barrier) so that the reads are in flight while the softmax
  // runs: the compiler otherwise issues them pairwise just before each P.V
  // product and waits out the LDS latency eight times per block.
  // A operand V^T: lane (c16, g) holds dim dt*16 + c16 at keys ks*32 + 4g + 0..3
  // and ks*32 + 16 + 4g + 0..3, the key order of P^T.
  bf16x8 va[kKs][4];
#pragma unroll
  for (int ks = 0; ks < kKs; ++ks)
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const char* lo_rows = lp.v[dt] + (kb + ks * 32) * kRowBytes;
      va[ks][dt] = __builtin_shufflevector(v_column4(lo_rows), v_column4(lo_rows + 16 * kRowBytes), 0, 1, 2, 3, 4, 5,
                                           6, 7);
    }
  __builtin_amdgcn_sched_barrier(0);
  // The lane's maximum over its 16 (8) scores (raw units; the scale is positive).
  float lm[2];
#pragma unroll
  for (int j = 0; j < kTiles; ++j) {
    float m = fmaxf(fmaxf(s[j][0][0], s[j][0][1]), s[j][0][2]);
    m = fmaxf(fmaxf(m, s[j][0][3]), s[j][1][0]);
#pragma unroll
    for (int kt = 1; kt < kKt; ++kt) {
      const int i0 = kt == 1 ? 1 : 0;
#pragma unroll
      for (int i = i0; i < 4; ++i) m = fmaxf(m, s[j][kt][i]);
    }
    lm[j] = m;
  }
  if (FIRST) {
#pragma unroll
    for (int j = 0; j < kTiles; ++j) st.m[j] = row_group_max(lm[j]) * scale_log2;
  } else {
    // Lazy rescaling: the running max only moves when a block exceeds it by
    // more than 2^8, so most blocks skip the rescale and the unnormalised
    // weights stay below 256.  Some lane's partial maximum exceeds the bound
    // exactly when some query's block maximum does, so the cross-lane
    // maximum is only taken on a rescale.
    bool grow = lm[0] * scale_log2 > st.m[0] + 8.0f;
    if (ACT1) grow = grow || lm[1] * scale_log2 > st.m[1] + 8.0f;
    if (__ballot(grow) != 0ull) {
#pragma unroll
      for (int j = 0; j < kTiles; ++j) {
        const float m_new = fmaxf(st.m[j], row_group_max(lm[j]) * scale_log2);
        const float alpha = __builtin_amdgcn_exp2f(st.m[j] - m_new);
        st.m[j] = m_new;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) st.o[j][dt] *= alpha;
        st.l[j] *= alpha;
      }
    }
  }
  bf16x8 pb[2][2];
#pragma unroll
  for (int j = 0; j < kTiles; ++j) {
    const float neg_m = -st.m[j];
#pragma unroll
    for (int kt = 0; kt < kKt; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) s[j][kt][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[j][kt][i], scale_log2, neg_m));
    // PV step ks, B operand k = 8g + e <-> key ks*32 + (e < 4 ? 4g + e : 16 + 4g + e - 4).
#pragma unroll
    for (int ks = 0; ks < kKs; ++ks)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        pb[j][ks][e] = static_cast<__bf16>(s[j][2 * ks][e]);
        pb[j][ks][4 + e] = static_cast<__bf16>(s[j][2 * ks + 1][e]);
      }
  }
  // O^T[dim][query] += V^T[dim][key] P^T[key][query]; a block of ones times
  // P^T accumulates the denominators (row sums of the bf16 weights).  In a
  // partial block the ones stop at the last key: element e of step ks in
  // lane group g stands for the key of P^T's element e.
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < kKs; ++ks) {
    const bool init = FIRST && ks == 0;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
      for (int j = 0; j < kTiles; ++j)
        st.o[j][dt] =
            __builtin_amdgcn_mfma_f32_16x16x32_bf16(va[ks][dt], pb[j][ks], init ? zero : st.o[j][dt], 0, 0, 0);
    }
  }
  if (kvalid < kKs * 32) {
    // Key of element e = ks*32 + 4g + (e < 4 ? e : 12 + e): compared as
    // 4g < kvalid - (the rest), one lane value against scalars.
    const int g4 = 4 * g;
#pragma unroll
    for (int ks = 0; ks < kKs; ++ks) {
      bf16x8 on;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int rest = ks * 32 + (e < 4 ? e : 12 + e);
        on[e] = g4 < kvalid - rest ? ones[e] : static_cast<__bf16>(0.0f);
      }
#pragma unroll
      for (int j = 0; j < kTiles; ++j)
        st.l[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(on, pb[j][ks], FIRST && ks == 0 ? zero : st.l[j], 0, 0, 0);
    }
  } else {
#pragma unroll
    for (int ks = 0; ks < kKs; ++ks)
#pragma unroll
      for (int j = 0; j < kTiles; ++j)
        st.l[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pb[j][ks], FIRST && ks == 0 ? zero : st.l[j], 0, 0, 0);
  }
}

// Wave priority by progress through a stage.  The three waves of a SIMD
// have the same work per stage, but the instruction arbiter favours the
// oldest wave, so left alone one wave finishes its blocks first, then the
// next, and the last runs alone on its SIMD (little to overlap its matrix
// and VALU work with) while the others wait at the stage barrier.  A stage
// starts every wave at priority 3 and each finished 64-key block lowers it
// by one, so the wave that is behind is served first and the three finish
// close together.
__device__ __forceinline__ void prio_after_block(int b) {
  if (b == 0) __builtin_amdgcn_s_setprio(2);
  else if (b == 1) __builtin_amdgcn_s_setprio(1);
  else __builtin_amdgcn_s_setprio(0);
}

// All key blocks of one stage (nk >= 1 keys in LDS): 64-key blocks, except
// that a last block of at most 32 keys runs as a 32-key half block after the
// others.  Two key blocks are in flight: the MFMAs of block kb+64 are issued
// before the softmax of block kb, so the matrix unit and the VALU overlap.
template <bool ACT1>
__device__ __forceinline__ void attend_stage(const LanePtrs& lp, int nk, bool first, float scale_log2,
                                             const bf16x8& ones, const bf16x8 (&qf)[2][2], SoftmaxState& sm) {
  const int tail = nk & 63;
  const int nm = tail != 0 && tail <= 32 ? nk - tail : nk;  // keys of the 64-key blocks
  if (nm > 0) {
    floatx4 sa[2][4], sbk[2][4];
    qk_block<ACT1, false>(lp, 0, qf, sa);
    if (nm > 64) qk_block<ACT1, false>(lp, 64, qf, sbk);
    if (first) softmax_pv_block<ACT1, true, false>(lp, 0, nm, scale_log2, ones, sa, sm);
    else softmax_pv_block<ACT1, false, false>(lp, 0, nm, scale_log2, ones, sa, sm);
    prio_after_block(0);
    // Unrolled over the stage (nm <= kKRes), so every block's LDS offsets are immediates.
#pragma unroll
    for (int kb = 64; kb < kKRes; kb += 128) {
      if (kb >= nm) break;
      if (kb + 64 < nm) qk_block<ACT1, false>(lp, kb + 64, qf, sa);
      softmax_pv_block<ACT1, false, false>(lp, kb, nm - kb, scale_log2, ones, sbk, sm);
      prio_after_block(kb >> 6);
      if (kb + 64 >= nm) break;
      if (kb + 128 < nm) qk_block<ACT1, false>(lp, kb + 128, qf, sbk);
      softmax_pv_block<ACT1, false, false>(lp, kb + 64, nm - kb - 64, scale_log2, ones, sa, sm);
      prio_after_block((kb >> 6) + 1);
    }
  }
  if (nm < nk) {
    floatx4 st[2][4];
    qk_block<ACT1, true>(lp, nm, qf, st);
    if (first && nm == 0) softmax_pv_block<ACT1, true, true>(lp, nm, nk - nm, scale_log2, ones, st, sm);
    else softmax_pv_block<ACT1, false, true>(lp, nm, nk - nm, scale_log2, ones, st, sm);
  }
}

// O = O^T / l rounded to bf16 for the wave's active query tiles (tile 1 when
// `act1`), obase = first row of the chunk.  Returns the number of store
// instructions issued (2 per tile): they are the last vector-memory
// instructions of the stage, which the next stage-start wait relies on.
//
// Lane (c16, g) holds dims 16 dt + 4g .. +3 of query c16.  One swap between
// 16-lane rows g and g^1 (v_permlane16_swap) per pair (dt, dt+1) leaves each
// lane with 8 consecutive dims, 8 * [0, 2, 1, 3][g] + 32 * pair .. +7, so a
// store instruction writes 64 contiguous bytes of each of 16 rows rather than
// 32 (half as many instructions, each touching half as many pieces of lines).
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ int store_out(char* obase, int nq, uint32_t row_bytes, const SoftmaxState& sm,
                                         bool act1) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4;
  const uint32_t chunk = static_cast<uint32_t>((((g & 1) << 1) | (g >> 1)) * 16);
  const __amdgpu_buffer_rsrc_t out = raw_buffer(obase);
#pragma unroll
  for (int j = 0; j < kTilesPerWave; ++j) {
    if (j == 1 && !act1) break;
    const float inv = __builtin_amdgcn_rcpf(sm.l[j][0]);
    uint32_t r[4][2];
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      bf16x4 x;
#pragma unroll
      for (int i = 0; i < 4; ++i) x[i] = static_cast<__bf16>(sm.o[j][dt][i] * inv);
      r[dt][0] = __builtin_bit_cast(u32x2, x)[0];
      r[dt][1] = __builtin_bit_cast(u32x2, x)[1];
    }
    u32x4 v[2];
#pragma unroll
    for (int pr = 0; pr < 2; ++pr) {
      const auto s0 = __builtin_amdgcn_permlane16_swap(r[2 * pr][0], r[2 * pr + 1][0], false, false);
      const auto s1 = __builtin_amdgcn_permlane16_swap(r[2 * pr][1], r[2 * pr + 1][1], false, false);
      v[pr] = u32x4{s0[0], s1[0], s0[1], s1[1]};
    }
    // Queries past the chunk's end get an offset past the resource: dropped.
    const int qi = tile_q(wave, j) + (lane & 15);
    const uint32_t off = qi < nq ? static_cast<uint32_t>(qi) * row_bytes + chunk : 0xFFFFFF00u;
    store_through(out, off, v[0]);
    store_through(out, off + 64, v[1]);
  }
  return act1 ? 4 : 2;
}

// Workgroup-uniform scheduling state of the execute loop.
struct Sched {
  Item cur, nx;    // item being computed, next item
  bool nx_valid;
  bool shift;      // the previous stage finished `cur`
  int sb;          // stage (256-key block) of `cur`
  int t_nn;        // queue thread: ticket of the item after `nx`
  int nst;         // output stores this wave issued at the end of the last stage
};

struct KernelCtx {
  const AttnParams& p;
  int n_items;
  int S, q, Gq;  // sub-queues, this workgroup's sub-queue, workgroups sharing it
  long long row_elems;
  uint32_t row_bytes;
  LdsOffsets lo;
  bf16x8 ones;
  const char* zrow;  // 128 zero bytes in the workspace header
};

// One stage: compute `cur`'s keys [sb*256, sb*256 + 256) from buffer Kc/Vc
// while the DMA of the next stage fills Kn/Vn.  Returns false after the last
// stage of the workgroup.
template <int B>
__device__ __forceinline__ bool attn_stage(const KernelCtx& c, Sched& s, const char* Kc, const char* Vc,
                                           uint16_t* Kn, uint16_t* Vn, uint16_t* Qs, int2* s_raw,
                                           bf16x8 (&qf)[2][2], SoftmaxState& sm) {
  const AttnParams& p = c.p;
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  // Stage start.  vmcnt counts in issue order and the previous stage's output
  // stores were this wave's last vector-memory instructions, so waiting until
  // only those remain outstanding waits for this wave's DMA (K/V of this
  // stage, queries of this item) without waiting for the stores.  After the
  // barrier every wave's DMA has landed, every wave is done with the other
  // buffer and the queue thread's descriptor write is visible.  (The barrier is
  // written out so that no LDS fence makes it wait for the DMA in flight.)
  const int nst = __builtin_amdgcn_readfirstlane(s.nst);
  if (nst == 4) asm volatile("s_waitcnt vmcnt(4) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  else if (nst == 2) asm volatile("s_waitcnt vmcnt(2) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  else asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  __builtin_amdgcn_s_setprio(3);
  if (s.shift) {
    const int2 raw = uniform_raw(s_raw[1 - B]);
    const bool nn_valid = raw.x != -1;
    const Item nn = nn_valid ? decode_item(p, raw) : Item{0, 0, 0, 0};
    s.cur = s.nx;
    s.nx = nn;
    s.nx_valid = nn_valid;
    s.sb = 0;
  }
  const Item cur = s.cur;
  const int kb0 = s.sb * kKRes;
  const int nk = min(kKRes, cur.len - kb0);
  const int cs = attn_chunk_size(cur.len);
  const int q0 = cur.chunk * cs;
  const int nq = min(cs, cur.len - q0);
  const bool act0 = tile_q(wave, 0) < nq;
  const bool act1 = kTilesPerWave > 1 && tile_q(wave, 1) < nq;
  if (s.sb == 0) {
    // The item's queries (this wave's rows), then, once they are in
    // registers, the next item's queries into the same rows.
    q_read(Qs, c.lo, nq, qf);
    if (s.nx_valid) {
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      q_chunk_dma(p, s.nx, c.row_elems, c.row_bytes, Qs);
    }
  }

  // Next stage: the rest of this item's keys, or the next item.  Its DMA is
  // issued by the waves with the fewest query tiles in this stage (waves
  // w >= T % kWaves for T tiles: with T > kWaves the waves below hold two
  // tiles, with T < kWaves the waves from T on hold none), so it stays off
  // the busiest waves' path.
  const int n_tiles = (nq + 15) / 16;
  const int w_dma = kTilesPerWave > 1 ? n_tiles % kWaves : (n_tiles < kWaves ? n_tiles : 0);
  const bool more_keys = kb0 + kKRes < cur.len;
  const bool have_next = more_keys || s.nx_valid;
  if (have_next) {
    const Item kv_item = more_keys ? cur : s.nx;
    const int kv_first = more_keys ? kb0 + kKRes : 0;
    const int kv_n = min(kKRes, kv_item.len - kv_first);
    if (kv_n > 0)
      kv_dma(head_base(p.k, static_cast<long long>(kv_item.seq0) + kv_first, c.row_elems, kv_item.h),
             head_base(p.v, static_cast<long long>(kv_item.seq0) + kv_first, c.row_elems, kv_item.h), c.zrow, kv_n,
             c.row_bytes, Kn, Vn, w_dma, kWaves - w_dma);
  }
  // Queue traffic goes out after the DMA; its results are consumed before
  // the output stores.
  int2 raw_next;
  raw_next.x = -1;
  raw_next.y = 0;
  int t_got = 0;
  if (tid == kQueueThread && !more_keys) {
    const int t = s.t_nn * c.S + c.q;
    if (t < c.n_items) raw_next = p.items[t];
    t_got = atomicAdd(&p.hdr->queue[c.q].ticket, 1);
  }

  if (act0) {
    const LanePtrs lp = lane_ptrs(Kc, Vc, c.lo);
    if constexpr (kTilesPerWave > 1) {
      if (act1) attend_stage<true>(lp, nk, s.sb == 0, p.scale_log2, c.ones, qf, sm);
      else attend_stage<false>(lp, nk, s.sb == 0, p.scale_log2, c.ones, qf, sm);
    } else {
      attend_stage<false>(lp, nk, s.sb == 0, p.scale_log2, c.ones, qf, sm);
    }
  }
  // Everything this stage loaded has arrived by now (the DMA went out before
  // the compute); an explicit wait says so, so that no later instruction
  // waits for it behind the output stores or the next DMA.
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  if (tid == kQueueThread && !more_keys) {
    s_raw[B] = raw_next;
    s.t_nn = t_got + 3 * c.Gq;
  }
  // The output goes last (nothing vector-memory may be issued after it).
  asm volatile("" ::: "memory");
  s.nst = 0;
  if (act0 && !more_keys) {
    char* obase = const_cast<char*>(head_base(p.out, static_cast<long long>(cur.seq0) + q0, c.row_elems, cur.h));
    s.nst = store_out(obase, nq, c.row_bytes, sm, act1);
  }
  s.shift = !more_keys;
  if (more_keys) ++s.sb;
  return have_next;
}

__global__ __launch_bounds__(kThreads) void attn_fwd_bf16_kernel(AttnParams p) {
  // Two K/V buffer pairs in one object, V first: the V buffers take the low
  // 64 KB of LDS, where the constant parts of the transposing V reads' addresses
  // (16 per key block) fit the instruction's offset field; the 8 K reads per
  // block pay the extra adds instead.
  struct StageLds {
    uint16_t v0[kStageElems], v1[kStageElems], k0[kStageElems], k1[kStageElems];
    uint16_t q[kAttnQTile * kD];  // queries of the current item, then of the next
  };
  __shared__ __attribute__((aligned(1024))) StageLds lds;
  uint16_t* const V0 = lds.v0;
  uint16_t* const V1 = lds.v1;
  uint16_t* const K0 = lds.k0;
  uint16_t* const K1 = lds.k1;
  __shared__ int2 s_init[2];  // the first two item descriptors
  __shared__ int2 s_raw[2];   // descriptor handed from the queue thread to the workgroup, by stage parity
  __shared__ int s_first;

  const int tid = threadIdx.x;
  // The first two descriptors are read before the plan header has arrived
  // (any slot below the workspace's capacity is in bounds) and dropped below
  // if they lie past the plan's item count.
  // Sub-queue q = w % S of workgroup w; its local tickets r, r + Gq, ...
  // (r = w / S, Gq workgroups share the sub-queue) name items lt * S + q.
  const int G = static_cast<int>(gridDim.x);
  const int S = min(kSubQueues, G);
  const int q = static_cast<int>(blockIdx.x) % S, r = static_cast<int>(blockIdx.x) / S;
  const int Gq = (G - q + S - 1) / S;
  const int t0 = r * S + q, t1 = (r + Gq) * S + q;
  int2 r0, r1;
  r0.x = -1;
  r0.y = 0;
  r1 = r0;
  if (tid == 0) {
    if (t0 < p.max_items) r0 = p.items[t0];
    if (t1 < p.max_items) r1 = p.items[t1];
  }
  if (!plan_matches(p)) {
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(p.status, DORA_DEV_PLAN);
    return;
  }
  KernelCtx c{p, min(p.hdr->n_items, p.max_items), S, q, Gq, static_cast<long long>(p.H) * kD,
              static_cast<uint32_t>(p.H) * kD * 2u, lds_offsets(), {},
              reinterpret_cast<const char*>(p.hdr->zero_row)};
#pragma unroll
  for (int e = 0; e < 8; ++e) c.ones[e] = static_cast<__bf16>(1.0f);

  // Queue.  Local tickets 0 .. 3Gq-1 of a sub-queue are dealt statically
  // (workgroup rank r takes r, r+Gq and r+2Gq, the longest items), the rest
  // come from the sub-queue's atomic counter, so the start of the kernel is
  // not a burst of atomics.  Eight counters on separate lines take eight
  // times the atomic rate of one: with one counter, the atomics alone bound
  // a DeiT-B execute to about 45 us.
  // One thread (kQueueThread) talks to the queue: it holds the local ticket
  // of the item after `nx`, loads that item's descriptor during a stage and
  // publishes it in LDS at the end of the stage, so no wave waits on the
  // queue mid-stage.
  Sched s;
  s.t_nn = 0;
  if (tid == kQueueThread) s.t_nn = r + 2 * Gq;
  if (tid == 0) {
    s_first = t0;
    if (t0 >= c.n_items) r0.x = -1;
    if (t1 >= c.n_items) r1.x = -1;
    s_init[0] = r0;
    s_init[1] = r1;
  }
  __syncthreads();
  if (s_first >= c.n_items) {
    leave_queue(p.hdr);
    return;
  }
  s.cur = decode_item(p, uniform_raw(s_init[0]));
  const int2 raw1 = uniform_raw(s_init[1]);
  s.nx_valid = raw1.x != -1;
  s.nx = s.nx_valid ? decode_item(p, raw1) : Item{0, 0, 0, 0};
  s.shift = false;
  s.sb = 0;
  s.nst = 0;

  bf16x8 qf[2][2];
  {
    const int nk = min(s.cur.len, kKRes);
    if (nk > 0)
      kv_dma(head_base(p.k, s.cur.seq0, c.row_elems, s.cur.h), head_base(p.v, s.cur.seq0, c.row_elems, s.cur.h),
             c.zrow, nk, c.row_bytes, K0, V0, 0, kWaves);
    q_chunk_dma(p, s.cur, c.row_elems, c.row_bytes, lds.q);
  }
  SoftmaxState sm;
  for (;;) {
    if (!attn_stage<0>(c, s, reinterpret_cast<const char*>(K0), reinterpret_cast<const char*>(V0), K1, V1, lds.q,
                       s_raw, qf, sm))
      break;
    if (!attn_stage<1>(c, s, reinterpret_cast<const char*>(K1), reinterpret_cast<const char*>(V1), K0, V0, lds.q,
                       s_raw, qf, sm))
      break;
  }
  leave_queue(p.hdr);
}

// ---------------------------------------------------------------------------
// fp32 inputs, v_mfma_f32_16x16x4_f32 (true fp32 products, fp32 accumulate).
// Same items, each taken as kF32Parts tickets of 64 queries; K/V streamed
// through LDS in blocks of 64 keys.
//
// MFMA 16x16x4 f32 operand layout (lane l, g = l / 16, c = l % 16):
//   A[16 x 4]: lane holds row c, k = g;  B[4 x 16]: lane holds column c, k = g
//   D[16 x 16]: lane holds column c, rows 4g .. 4g+3
// ---------------------------------------------------------------------------
constexpr int kBlockKeys = 64;
constexpr int kFStride = kD + 4;  // floats per K / V row in LDS

__global__ __launch_bounds__(kF32Threads) void attn_fwd_f32_kernel(AttnParams p) {
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

  // At most 8192 x 256 x 86 items (B, H, chunks of 16384 keys): the ticket
  // count stays below 2^31.
  const int n_tickets = n_items * kF32Parts;
  for (;;) {
    if (tid == 0) s_ticket = atomicAdd(&p.hdr->queue[0].ticket, 1);
    __syncthreads();
    const int ticket = s_ticket;
    __syncthreads();
    if (ticket >= n_tickets) break;
    const int part = ticket % kF32Parts;
    const Item it = decode_item(p, p.items[ticket / kF32Parts]);
    const long long seq0 = it.seq0;
    const int len = it.len;
    const int cs = attn_chunk_size(len);
    const int qbeg = it.chunk * cs + part * kF32PartQ;  // this part's queries start here
    const int qend = min(len, (it.chunk + 1) * cs);     // and the item's chunk ends here
    if (qbeg >= qend) continue;                          // workgroup-uniform: an empty part
    const int q0 = qbeg + wave * 16;
    const bool active = q0 < qend;

    float qf[16];
    {
      const int qi = q0 + c16;
#pragma unroll
      for (int ks = 0; ks < 16; ++ks)
        qf[ks] = qi < qend ? Q[(seq0 + qi) * row_elems + it.h * kD + 4 * ks + g] : 0.f;
    }
    floatx4 o[4];
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) o[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY;
    float l_run = 0.f;

    // K/V of the next 64-key block are loaded into registers while the
    // current block is computed, then stored to LDS between two barriers.
    constexpr int kU = kBlockKeys * 16 / kF32Threads;  // float4 of K (and of V) per thread per block
    float4 kn[kU], vn[kU];
    auto fetch = [&](int kb0) {
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int e = tid + u * kF32Threads;  // 64 keys x 16 float4
        const int key = e >> 4, dv = e & 15;
        kn[u] = make_float4(0.f, 0.f, 0.f, 0.f);
        vn[u] = kn[u];
        if (kb0 + key < len) {
          const long long off = (seq0 + kb0 + key) * row_elems + it.h * kD + dv * 4;
          kn[u] = *reinterpret_cast<const float4*>(K + off);
          vn[u] = *reinterpret_cast<const float4*>(V + off);
        }
      }
    };
    fetch(0);
    for (int kb0 = 0; kb0 < len; kb0 += kBlockKeys) {
      __syncthreads();
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int e = tid + u * kF32Threads;
        const int key = e >> 4, dv = e & 15;
        *reinterpret_cast<float4*>(&Ks[key * kFStride + dv * 4]) = kn[u];
        *reinterpret_cast<float4*>(&Vs[key * kFStride + dv * 4]) = vn[u];
      }
      __syncthreads();
      if (kb0 + kBlockKeys < len) fetch(kb0 + kBlockKeys);
      if (!active) continue;

      floatx4 s[4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        s[kt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < 16; ++ks)
          s[kt] = __builtin_amdgcn_mfma_f32_16x16x4f32(Ks[(kt * 16 + c16) * kFStride + 4 * ks + g], qf[ks], s[kt],
                                                      0, 0, 0);
      }
      // The running max stays in raw score units and is subtracted before
      // scaling, so the terms near the max carry only a small rounding error.
      const int kvalid = len - kb0;
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = kt * 16 + 4 * g + i;
          const float x = key < kvalid ? s[kt][i] : -INFINITY;
          s[kt][i] = x;
          mx = fmaxf(mx, x);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * p.scale_log2);
      m_run = m_new;
      float rs = 0.f;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float pv = __builtin_amdgcn_exp2f((s[kt][i] - m_new) * p.scale_log2);
          s[kt][i] = pv;
          rs += pv;
        }
      l_run = l_run * alpha + rs;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) o[dt] *= alpha;
      // O^T += V^T P^T, one 4-key step per (kt, i): MFMA k = g <-> key kt*16 + 4g + i.
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int dt = 0; dt < 4; ++dt)
            o[dt] = __builtin_amdgcn_mfma_f32_16x16x4f32(Vs[(kt * 16 + 4 * g + i) * kFStride + dt * 16 + c16],
                                                        s[kt][i], o[dt], 0, 0, 0);
    }

    if (active) {
      float l = l_run + __shfl_xor(l_run, 16, 64);
      l += __shfl_xor(l, 32, 64);
      const float inv = 1.0f / l;
      const int qi = q0 + c16;
      if (qi < qend) {
        float* dst = O + (seq0 + qi) * row_elems + it.h * kD + 4 * g;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
          *reinterpret_cast<float4*>(dst + dt * 16) =
              make_float4(o[dt][0] * inv, o[dt][1] * inv, o[dt][2] * inv, o[dt][3] * inv);
      }
    }
  }
  leave_queue(p.hdr);
}

// Persistent grid: every compute unit filled to the kernel's occupancy.
// The occupancy is queried once per device and kernel and cached; the cache
// entries are atomics, so concurrent first calls from several host threads
// store the same value without a data race.
template <typename KernelT>
int persistent_grid(KernelT kernel, int threads, int slot, int* grid) {
  static std::atomic<int> per_cu_cache[64][2];
  int dev = 0;
  const int cus = device_cu_count(&dev);
  if (cus <= 0 || dev >= 64) return DORA_ERR_HIP;
  int per_cu = per_cu_cache[dev][slot].load(std::memory_order_relaxed);
  if (per_cu == 0) {
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess ||
        per_cu < 1)
      per_cu = 1;
    per_cu_cache[dev][slot].store(per_cu, std::memory_order_relaxed);
  }
  *grid = cus * per_cu;
  return DORA_OK;
}

}  // namespace

int device_cu_count(int* device_out) {
  static std::atomic<int> cache[64];  // per device, written once (same value from any thread)
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -1;
  if (device_out) *device_out = dev;
  if (dev < 0 || dev >= 64) return -1;
  int n = cache[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -1;
    cache[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

int launch_attn_plan(const int32_t* cu, int32_t B, int32_t H, int32_t max_seqlen, int64_t total, int32_t min_len,
                     void* workspace, int32_t* dev_status, void* stream) {
  const AttnWorkspaceLayout L = attn_workspace_layout(B, H, max_seqlen);
  PlanParams p;
  p.cu = cu;
  p.B = B;
  p.H = H;
  p.max_seqlen = max_seqlen;
  p.min_len = min_len;
  p.total = total;
  p.status = dev_status;
  p.hdr = static_cast<AttnPlanHeader*>(workspace);
  p.items = reinterpret_cast<int2*>(static_cast<char*>(workspace) + L.items_off);
  hipLaunchKernelGGL(attn_plan_kernel, dim3(1), dim3(kPlanThreads), 0, static_cast<hipStream_t>(stream), p);
  return hipGetLastError() == hipSuccess ? DORA_OK : DORA_ERR_HIP;
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
  const AttnWorkspaceLayout L = attn_workspace_layout(B, H, max_seqlen);
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) || workspace_bytes < L.bytes)
    return DORA_ERR_WORKSPACE;
  return launch_attn_plan(cu_seqlens, B, H, max_seqlen, total, 0, workspace, dev_status, stream);
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
  const AttnWorkspaceLayout L = attn_workspace_layout(B, H, max_seqlen);
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) || workspace_bytes < L.bytes)
    return DORA_ERR_WORKSPACE;
  if (!(softmax_scale > 0.0f)) softmax_scale = 1.0f / sqrtf(static_cast<float>(D));

  AttnParams p;
  p.q = q;
  p.k = k;
  p.v = v;
  p.out = out;
  p.B = B;
  p.H = H;
  p.max_seqlen = max_seqlen;
  p.total = total;
  p.scale_log2 = softmax_scale * kLog2e;
  p.hdr = static_cast<AttnPlanHeader*>(workspace);
  p.items = reinterpret_cast<const int2*>(static_cast<char*>(workspace) + L.items_off);
  p.max_items = static_cast<int32_t>(L.max_items);
  p.status = dev_status;

  int grid = 0;
  const int rc = dtype == DORA_BF16 ? persistent_grid(attn_fwd_bf16_kernel, kThreads, 0, &grid)
                                    : persistent_grid(attn_fwd_f32_kernel, kF32Threads, 1, &grid);
  if (rc != DORA_OK) return rc;
  // No more workgroups than the plan can hold tickets: a small batch then
  // launches (and retires, each with its exit atomic) only what it can use.
  const int64_t max_tickets = L.max_items * (dtype == DORA_BF16 ? 1 : kF32Parts);
  if (max_tickets < grid) grid = static_cast<int>(max_tickets < 1 ? 1 : max_tickets);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (dtype == DORA_BF16)
    hipLaunchKernelGGL(attn_fwd_bf16_kernel, dim3(grid), dim3(kThreads), 0, st, p);
  else
    hipLaunchKernelGGL(attn_fwd_f32_kernel, dim3(grid), dim3(kF32Threads), 0, st, p);
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

// Workspace of dora_varlen_attn_noalloc: one per GPU, for the life of the
// process.  Host code never passes the array's name to a kernel (on the host
// it is a stand-in, not a device address); it uses the address that
// hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) uint8_t scratch[DORA_NOALLOC_WORKSPACE_BYTES];

namespace dora {
namespace {

// Device address of `scratch` on the current device, looked up on the first
// call there and kept (a per-device atomic: concurrent first calls store the
// same address).
int noalloc_workspace(void** out) {
  static std::atomic<void*> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return DORA_ERR_HIP;
  void* ptr = cache[dev].load(std::memory_order_acquire);
  if (ptr == nullptr) {
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return DORA_ERR_HIP;
    cache[dev].store(ptr, std::memory_order_release);
  }
  *out = ptr;
  return DORA_OK;
}

}  // namespace
}  // namespace dora

extern "C" int dora_varlen_attn_noalloc(const void* q, const void* k, const void* v,
                                        const int32_t* cu_seqlens, int32_t B, int32_t H, int32_t D,
                                        int32_t max_seqlen, int64_t total, float softmax_scale,
                                        dora_dtype dtype, void* out, int32_t* dev_status, void* stream) {
  using namespace dora;
  if (!q || !k || !v || !cu_seqlens || !out || !dev_status) return DORA_ERR_NULL;
  if (dtype != DORA_F32 && dtype != DORA_BF16) return DORA_ERR_DTYPE;
  if (D != DORA_HEAD_DIM) return DORA_ERR_SHAPE;
  const int sz = check_attn_sizes(B, H, max_seqlen, total);
  if (sz != DORA_OK) return sz;
  if ((reinterpret_cast<uintptr_t>(q) | reinterpret_cast<uintptr_t>(k) | reinterpret_cast<uintptr_t>(v) |
       reinterpret_cast<uintptr_t>(out)) & 15u)
    return DORA_ERR_ALIGN;
  const size_t need = attn_workspace_layout(B, H, max_seqlen).bytes;
  if (need > DORA_NOALLOC_WORKSPACE_BYTES) return DORA_ERR_STATIC_LIMIT;
  void* ws = nullptr;
  const int rc = noalloc_workspace(&ws);
  if (rc != DORA_OK) return rc;
  return dora_varlen_attn(q, k, v, cu_seqlens, B, H, D, max_seqlen, total, softmax_scale, dtype, out, ws,
                          DORA_NOALLOC_WORKSPACE_BYTES, dev_status, stream);
}

extern "C" const char* dora_status_string(int status) {
  switch (status) {
    case DORA_OK: return "DORA_OK";
    case DORA_ERR_NULL: return "DORA_ERR_NULL: a required pointer is NULL";
    case DORA_ERR_SHAPE: return "DORA_ERR_SHAPE: a size is out of range";
    case DORA_ERR_DTYPE: return "DORA_ERR_DTYPE: unknown dtype";
    case DORA_ERR_ALIGN: return "DORA_ERR_ALIGN: row data must be 16-byte aligned";
    case DORA_ERR_UNSUPPORTED: return "DORA_ERR_UNSUPPORTED: outside what this library implements";
    case DORA_ERR_CAPACITY: return "DORA_ERR_CAPACITY: output capacity out of range";
    case DORA_ERR_HIP: return "DORA_ERR_HIP: HIP runtime error at launch";
    case DORA_ERR_WORKSPACE: return "DORA_ERR_WORKSPACE: workspace missing, misaligned or too small";
    case DORA_ERR_STATIC_LIMIT: return "DORA_ERR_STATIC_LIMIT: sizes need more than the library's static workspace";
    default: return "unknown dora status";
  }
}
