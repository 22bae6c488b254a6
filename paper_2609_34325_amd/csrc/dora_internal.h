// Internal definitions shared by the HIP translation units of libdora.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dora.h"

namespace dora {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// Number of compute units of the current device (cached per device id).
int device_cu_count(int* device_out);

// Enqueues the attention plan kernel: items of the layout cu[0..B] into the
// workspace (sizes already checked by the caller).  Sequences shorter than
// min_len, longer than max_seqlen or past total make the plan empty and set
// DORA_DEV_CU_SEQLENS.
int launch_attn_plan(const int32_t* cu, int32_t B, int32_t H, int32_t max_seqlen, int64_t total, int32_t min_len,
                     void* workspace, int32_t* dev_status, void* stream);

// 16-byte stores at system scope (sc1), non-temporal (nt): written through
// the L2 and not kept there, so no line is left dirty (a bulk output written
// with plain stores leaves up to the L2's capacity dirty: several
// microseconds of write-back after the last workgroup ends) and the output
// does not push the inputs still to be read out of the caches.  Issued as
// buffer stores, the only global store form whose cache-policy bits a builtin
// sets; the compiler sees them as stores, so its hazard and wait bookkeeping
// covers them.  The resource spans [base, base + 2^31 - 1) with raw byte
// offsets; a store at an offset past that range is dropped by the hardware.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kStoreThrough = 16 | 2;  // cache policy: sc1 (system scope) | nt

__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_buffer(void* base) {
  // Word 3 of a raw gfx9-family buffer descriptor: 32-bit data format, no swizzle.
  return __builtin_amdgcn_make_buffer_rsrc(base, 0, 0x7FFFFFFF, 0x00020000);
}

__device__ __forceinline__ void store_through(__amdgpu_buffer_rsrc_t r, uint32_t off, u32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, kStoreThrough);
}

// Wave64 helpers.
__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

// ---------------------------------------------------------------------------
// Attention work-queue workspace layout (device memory owned by the caller).
//
//   [0, 2048)     AttnPlanHeader (plan sizes, exit counter, a row of zeros,
//                 one ticket counter per sub-queue, each on its own 128-byte
//                 line)
//   [2048, ...)   items[max_items]: int2 {x = first row of the sequence,
//                 y = len << 17 | head << 9 | query chunk}
//
// A work item is one (sequence, head, chunk of at most kAttnQTile queries);
// items are ordered by decreasing sequence length.  Item i belongs to
// sub-queue i % kSubQueues, so each sub-queue is itself longest-first and the
// sub-queues carry near-equal work.  Sequences with the same number of
// chunks form a contiguous class; inside it, full blocks of kSubQueues
// (sequence, head) groups place the chunks of group j at stride kSubQueues
// (attn_item_slot), so every chunk of a (sequence, head) is in one sub-queue,
// at consecutive tickets: the workgroups of one XCD take them together and
// read that head's K/V through one L2.
// ---------------------------------------------------------------------------
constexpr int32_t kPlanMagic = 0x444F5241;  // "DORA"
constexpr int kAttnQTile = 192;             // queries per work item (12 tiles of 16, one per wave)
constexpr int kPlanMaxB = 8192;             // sequences one plan can order
constexpr int kSubQueues = 8;               // ticket counters (one per XCD of an MI355X)

struct AttnQueueLine {
  int32_t ticket;  // next dynamic ticket of the sub-queue
  int32_t pad[31];
};

struct AttnPlanHeader {
  int32_t unused[2];
  int32_t n_items;     // items in this plan
  int32_t magic;       // kPlanMagic once planned
  int32_t B, H, max_seqlen, q_tile;
  int64_t total;
  int32_t reserved[22];
  uint32_t zero_row[32];  // one 128-byte row of zeros (bf16 V rows past a sequence's end)
  AttnQueueLine queue[kSubQueues];
  // Workgroups that have left the current execute.  On a line of its own:
  // every workgroup's exit atomic would otherwise queue behind, or hold up,
  // the loads of the plan fields that other workgroups make at their start.
  int32_t exit_count;
  int32_t reserved2[191];
};
static_assert(sizeof(AttnPlanHeader) == 2048, "header must fill its slot");
static_assert(__builtin_offsetof(AttnPlanHeader, exit_count) == 256 + kSubQueues * 128, "exit counter on its own line");
static_assert(__builtin_offsetof(AttnPlanHeader, zero_row) == 128, "zero row is the header's second line");
static_assert(__builtin_offsetof(AttnPlanHeader, queue) == 256, "queue counters start on a line of their own");

struct AttnWorkspaceLayout {
  size_t items_off, bytes;
  int64_t max_items;
};

inline AttnWorkspaceLayout attn_workspace_layout(int32_t B, int32_t H, int32_t max_seqlen) {
  AttnWorkspaceLayout L;
  const int64_t chunks = (static_cast<int64_t>(max_seqlen) + kAttnQTile - 1) / kAttnQTile;
  L.max_items = static_cast<int64_t>(B) * H * chunks;
  L.items_off = sizeof(AttnPlanHeader);
  L.bytes = L.items_off + static_cast<size_t>(L.max_items) * 8;
  L.bytes = (L.bytes + 255) & ~size_t(255);
  return L;
}

// Host-side range checks of the sizes a plan is made for.
inline int check_attn_sizes(int32_t B, int32_t H, int32_t max_seqlen, int64_t total) {
  if (B < 1 || B > kPlanMaxB || H < 1 || H > 256 || max_seqlen < 1 || max_seqlen > DORA_MAX_SEQLEN ||
      total < 0 || total > 0x7FFFFFFF)
    return DORA_ERR_SHAPE;
  if (attn_workspace_layout(B, H, max_seqlen).max_items > 0x7FFFFFFF) return DORA_ERR_UNSUPPORTED;
  return DORA_OK;
}

// Query chunks of a sequence of `len` tokens (len >= 0).
__host__ __device__ __forceinline__ int attn_chunks(int len) { return (len + kAttnQTile - 1) / kAttnQTile; }

// Queries per chunk: the chunks share the sequence evenly, rounded up to
// whole 16-query tiles (at most kAttnQTile; the last chunk takes the rest and
// is never empty).
__host__ __device__ __forceinline__ int attn_chunk_size(int len) {
  if (len <= kAttnQTile) return (len + 15) & ~15;  // one chunk: no division on the common path
  const int ch = attn_chunks(len);
  return ((len + ch - 1) / ch + 15) & ~15;
}

// Item slot of chunk c of group gi (the sequence's rank inside its class
// times H, plus the head) in a class of `groups` groups of ch chunks whose
// items start at slot `base`.  Full blocks of kSubQueues groups put group j's
// chunks at slots base + block * ch * kSubQueues + c * kSubQueues + j; the
// groups past the last full block follow chunk after chunk.
__host__ __device__ __forceinline__ long long attn_item_slot(long long base, int groups, int ch, int gi, int c) {
  const int full = groups / kSubQueues * kSubQueues;
  if (gi < full)
    return base + static_cast<long long>(ch) * (gi / kSubQueues) * kSubQueues +
           static_cast<long long>(c) * kSubQueues + gi % kSubQueues;
  return base + static_cast<long long>(ch) * full + static_cast<long long>(gi - full) * ch + c;
}

// Item descriptor of chunk c of head h of the sequence at rows [seq0, seq0 + len).
__device__ __forceinline__ int2 encode_item(int seq0, int len, int h, int c) {
  return make_int2(seq0, static_cast<int>((static_cast<uint32_t>(len) << 17) | (static_cast<uint32_t>(h) << 9) |
                                          static_cast<uint32_t>(c)));
}

// Header of a plan with n_items items (one thread); the zero row is written
// separately.
__device__ __forceinline__ void write_plan_header(AttnPlanHeader* hdr, int n_items, int32_t B, int32_t H,
                                                  int32_t max_seqlen, int64_t total) {
  hdr->n_items = n_items;
  for (int q = 0; q < kSubQueues; ++q) hdr->queue[q].ticket = 0;
  hdr->exit_count = 0;
  hdr->B = B;
  hdr->H = H;
  hdr->max_seqlen = max_seqlen;
  hdr->q_tile = kAttnQTile;
  hdr->total = total;
  hdr->magic = kPlanMagic;
}

}  // namespace dora
