/*
 * dora.h -- C ABI of the DORA deployment hot path on AMD Instinct MI355X (gfx950).
 *
 * DORA (arXiv 2609.34325) prunes Vision Transformer tokens per image.  At
 * deployment the actor keeps CLS, removes the visual tokens the selector
 * ranks highest for removal, and preserves the order of the survivors
 * (Sec. 3.1, Eq. (1); Sec. 3.2 "Sampling and deployment"; App. A.3).  The
 * survivors of all images are compacted into one packed buffer with
 * explicit sequence boundaries and processed by variable-length attention
 * that never attends across images (Sec. 3.5 "Inference"; App. E.5).
 *
 * This library implements that path as two calls:
 *   dora_select_pack  -- per-image top-k selection with CLS pinned, the
 *                        running total of keep counts (cu_seqlens) and the
 *                        gather of kept rows into the packed buffer;
 *   dora_varlen_attn  -- softmax attention inside each packed sequence
 *                        (split into _plan and _execute so one plan can
 *                        serve every layer that shares the same layout).
 *
 * Conventions shared by every entry point
 *   - All array arguments are DEVICE pointers allocated by the caller; the
 *     library never allocates device memory, never frees caller memory and
 *     keeps no state between calls other than a per-device cache of the
 *     compute-unit count and of the attention kernels' occupancy (atomics,
 *     safe to fill from several host threads at once).
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     Every call only enqueues work on that stream and returns without
 *     synchronising the host.
 *   - Argument errors that the host can see are returned as a negative
 *     dora_status before anything is enqueued.
 *   - Errors that depend on device data (keep counts, offsets) are reported
 *     by OR-ing DORA_DEV_* bits into *dev_status (an int32 in device memory
 *     that the caller zeroes beforehand and reads after synchronising).
 *     When a bit is set the affected outputs are unspecified, but no write
 *     ever lands outside the output buffers' stated extents.
 *   - Row-major layouts; int32 indices; element types per dora_dtype.
 */
#ifndef DORA_H_
#define DORA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { DORA_F32 = 0, DORA_BF16 = 1 } dora_dtype;

typedef enum {
  DORA_OK = 0,
  DORA_ERR_NULL = -1,        /* a required pointer is NULL                          */
  DORA_ERR_SHAPE = -2,       /* a size is out of range (B, N, C, H, D, max_seqlen)  */
  DORA_ERR_DTYPE = -3,       /* unknown dora_dtype                                  */
  DORA_ERR_ALIGN = -4,       /* a row-data pointer is not 16-byte aligned           */
  DORA_ERR_UNSUPPORTED = -5, /* valid request outside what this library implements  */
  DORA_ERR_CAPACITY = -6,    /* an output capacity cannot be represented            */
  DORA_ERR_HIP = -7,         /* the HIP runtime reported an error at launch         */
  DORA_ERR_WORKSPACE = -8,   /* workspace NULL, misaligned or smaller than required */
  DORA_ERR_STATIC_LIMIT = -9 /* sizes need more than the library's static workspace */
} dora_status;

/* Bits OR-ed into *dev_status by the kernels. */
#define DORA_DEV_KEEP_RANGE 0x1  /* some keep[b] < 1 or keep[b] > n_b; image b was skipped         */
#define DORA_DEV_CAPACITY 0x2    /* sum(keep) > cap_rows; rows at or past cap_rows were not written */
#define DORA_DEV_CU_IN 0x4       /* cu_in not a partition of [0,total_in) into segments of 1..N     */
#define DORA_DEV_CU_SEQLENS 0x8  /* attention offsets invalid (non-monotone, past total, or a
                                    sequence longer than max_seqlen); such sequences were skipped */
#define DORA_DEV_PLAN 0x10       /* execute called with a workspace not planned for these sizes    */
#define DORA_DEV_ACTOR 0x20      /* actor decode: a gate-on image without a legal budget or logit row;
                                    it was left unpruned                                           */

/* Limits of this library. */
#define DORA_MAX_ROW_TOKENS 2048     /* dora_select_pack: N (tokens per image, CLS included)  */
#define DORA_MAX_SEQLEN 16384        /* dora_varlen_attn: max_seqlen                          */
#define DORA_HEAD_DIM 64             /* dora_varlen_attn: D                                   */

/*
 * dora_select_pack -- hard deletion + packing (Sec. 3.1 Eq. (1); Sec. 3.2
 * "Sampling and deployment"; Sec. 3.5 "Inference"; App. A.3).
 *
 * For every image b with input segment of n_b tokens (position 0 is CLS):
 *   keep CLS and the keep[b]-1 visual positions with the highest score,
 *   comparing scores as FP32 values (App. E.5); equal scores go to the lower
 *   position, NaN ranks below every number, -0 equals +0.  The kept
 *   positions are written in ascending order, so CLS and the survivors'
 *   relative order are preserved.
 *
 * Scores are KEEP-scores (higher = keep).  The paper's selector scores
 * removal preference (higher = remove; Sec. 3.2, selector equation (2)), so a DORA caller
 * passes their negation; its removal budget k_l maps to keep = n_b - k_l
 * (n_b counts CLS).
 *
 *   scores     fp32.  Dense input (cu_in == NULL): [B, N], n_b = N.
 *              Packed input: [total_in], segment b = [cu_in[b], cu_in[b+1]).
 *   keep       int32 [B]   keep count of image b including CLS, 1..n_b.
 *   tokens     dtype [B, N, C] (dense) or [total_in, C] (packed); 16-byte aligned.
 *   cu_in      NULL or int32 [B+1] with cu_in[0] = 0, non-decreasing,
 *              1 <= cu_in[b+1]-cu_in[b] <= N, cu_in[B] <= total_in.
 *              Chaining rounds: pass the previous round's cu_out and packed_out.
 *   total_in   rows of the packed input (ignored for dense input).
 *   B          images, >= 1.
 *   N          dense: tokens per image; packed: an upper bound on n_b.
 *              1 <= N <= DORA_MAX_ROW_TOKENS.
 *   C          channels per token; C * sizeof(dtype) must be a multiple of 16.
 *   idx_out    int32 [cap_rows]: kept positions, local to each input segment,
 *              ascending within each image; idx_out[cu_out[b]] == 0 (CLS).
 *   cu_out     int32 [B+1]: cu_out[0] = 0, cu_out[b+1] = cu_out[b] + keep[b].
 *   packed_out dtype [cap_rows, C]: packed_out[cu_out[b] + r] is a bitwise copy
 *              of token row idx_out[cu_out[b] + r] of image b.  16-byte aligned.
 *   cap_rows   rows available in idx_out / packed_out, 1 .. 2^31-1.
 *   dev_status int32 device word, see DORA_DEV_*.
 *
 * cu_out is the running total of the keep counts.  Up to 2048 images each
 * workgroup sums the counts before its own image; past 2048 images one
 * workgroup first scans all counts into cu_out, in a launch of its own.
 *
 * Returns DORA_OK or a negative dora_status; enqueues one kernel (two past
 * 2048 images).
 */
int dora_select_pack(const float* scores, const int32_t* keep, const void* tokens,
                     const int32_t* cu_in, int64_t total_in, int32_t B, int32_t N, int32_t C,
                     dora_dtype dtype, int32_t* idx_out, int32_t* cu_out, void* packed_out,
                     int64_t cap_rows, int32_t* dev_status, void* stream);

/*
 * dora_varlen_attn_workspace_size -- bytes of device workspace that
 * dora_varlen_attn_plan / _execute / dora_varlen_attn need for B sequences,
 * H heads and sequences of at most max_seqlen tokens.  Returns 0 for sizes
 * out of range.
 */
size_t dora_varlen_attn_workspace_size(int32_t B, int32_t H, int32_t max_seqlen);

/*
 * dora_varlen_attn_plan -- build the attention work queue for one packed
 * layout (the sequence boundaries of Sec. 3.5 "Inference").
 *
 * Writes into `workspace` the list of (sequence, head, query-tile) items of
 * the layout, ordered by decreasing sequence length so that long sequences
 * start first and short ones fill the tail, and resets the queue counters.
 * A plan stays valid for any number of _execute calls with the same
 * cu_seqlens contents and sizes (e.g. every layer between two pruning steps).
 *
 *   cu_seqlens int32 [B+1]: 0 = cu[0] <= cu[1] <= ... <= cu[B] <= total and
 *              cu[b+1]-cu[b] <= max_seqlen; empty sequences are allowed.
 *   1 <= B <= 8192, 1 <= H <= 256, 1 <= max_seqlen <= DORA_MAX_SEQLEN,
 *              0 <= total <= 2^31-1.
 *   workspace  device, 256-byte aligned, >= dora_varlen_attn_workspace_size bytes.
 *   dev_status DORA_DEV_CU_SEQLENS when the offsets are invalid (the plan is
 *              then empty and _execute writes nothing).
 */
int dora_varlen_attn_plan(const int32_t* cu_seqlens, int32_t B, int32_t H, int32_t max_seqlen,
                          int64_t total, void* workspace, size_t workspace_bytes,
                          int32_t* dev_status, void* stream);

/*
 * dora_select_pack_plan -- dora_select_pack and, in the same launch, the
 * attention plan of its packed output (Sec. 3.5 "Inference": the packed
 * sequences are the kept tokens of each image, so sequence b has keep[b]
 * rows starting at cu_out[b]).
 *
 * The select/pack arguments and results are those of dora_select_pack.  The
 * plan written into `workspace` serves dora_varlen_attn_execute with
 * cu_seqlens = cu_out and the same B, H, max_seqlen and total, exactly as a
 * dora_varlen_attn_plan call on cu_out would.  Up to 2048 images it is built
 * in the select/pack launch while the rows are copied (it depends on the
 * keep counts only), its items ordered by decreasing keep count, then by
 * image.  Past 2048 images the keep counts are first scanned into cu_out by
 * a one-workgroup launch and the plan is made from cu_out as
 * dora_varlen_attn_plan makes it (decreasing length, equal lengths in an
 * unspecified order); attention results do not depend on that order.
 *
 *   H, max_seqlen, total  as for dora_varlen_attn_plan; total is the row
 *              count of the Q/K/V buffers that execute will read.
 *   workspace  device, 256-byte aligned, >= dora_varlen_attn_workspace_size
 *              (B, H, max_seqlen) bytes.
 *   dev_status the select/pack bits, plus DORA_DEV_CU_SEQLENS when some
 *              keep[b] is outside [1, max_seqlen] or sum(keep) > total (the
 *              plan is then empty and execute writes nothing).
 *
 * Returns DORA_OK or a negative dora_status; enqueues one kernel (three
 * past 2048 images).
 */
int dora_select_pack_plan(const float* scores, const int32_t* keep, const void* tokens,
                          const int32_t* cu_in, int64_t total_in, int32_t B, int32_t N, int32_t C,
                          dora_dtype dtype, int32_t* idx_out, int32_t* cu_out, void* packed_out,
                          int64_t cap_rows, int32_t H, int32_t max_seqlen, int64_t total,
                          void* workspace, size_t workspace_bytes, int32_t* dev_status, void* stream);

/*
 * dora_select_pack_residual -- deletion after the attention residual
 * (Sec. 3.1, Eq. (1): the removed rows still take part in the current
 * attention, and they are dropped from H + Attention(LayerNorm(H)) before
 * the MLP).  Equivalent to dora_select_pack on tokens = h + a, without
 * writing the full sum to memory: only the kept rows of the sum are formed.
 *
 *   h          dtype, the residual stream, laid out as `tokens` of
 *              dora_select_pack (dense [B, N, C] or packed [total_in, C]).
 *   a          dtype, the attention branch's output in h's layout (after the
 *              output projection); 16-byte aligned.
 *   packed_out packed_out[cu_out[b] + r] = h + a of token row
 *              idx_out[cu_out[b] + r] of image b, each element the exact sum
 *              of the two values rounded once to dtype, to nearest with ties
 *              to even (subnormals kept; a sum past the largest finite value
 *              is infinity).
 * Every other argument, result and dev_status bit is that of
 * dora_select_pack.  packed_out must not overlap h or a.
 *
 * Returns DORA_OK or a negative dora_status (DORA_ERR_NULL for a NULL a,
 * DORA_ERR_ALIGN for a misaligned one); enqueues one kernel (two past 2048
 * images, as dora_select_pack).
 */
int dora_select_pack_residual(const float* scores, const int32_t* keep, const void* h, const void* a,
                              const int32_t* cu_in, int64_t total_in, int32_t B, int32_t N, int32_t C,
                              dora_dtype dtype, int32_t* idx_out, int32_t* cu_out, void* packed_out,
                              int64_t cap_rows, int32_t* dev_status, void* stream);

/*
 * dora_actor_gate -- gate of the deterministic actor and compaction of the
 * gate-on images (Sec. 3.2 "Gate" and "Sampling and deployment"; App. A.2,
 * Eq. (legal budgets); App. A.3).
 *
 * Image b holds n_b tokens with CLS (N_l = n_b - 1 visual tokens).  The
 * budget grid is k = 2, 4, ..., 2M (M budget-head outputs, M = (N0 - 4) / 2
 * in the paper's Table 3) and a budget is legal when k <= N_l - 4, so that at
 * least four visual tokens survive.  The gate opens when p_gate[b] >= 0.5
 * (FP32 compare; NaN stays closed) and some budget is legal.  Gate-on images
 * are numbered in image order, so the controller (encoder, budget head,
 * selector) can run on them alone.
 *
 *   p_gate   fp32 [B], the gate probabilities.
 *   cu_in    NULL (every image has N tokens) or int32 [B+1] segment offsets
 *            of packed tokens (a later round); a segment with n_b outside
 *            [1, N] keeps its gate closed and sets DORA_DEV_CU_IN.
 *   B        1 .. 2^24 images; N 1 .. DORA_MAX_ROW_TOKENS; M >= 1.
 *   on_rank  int32 [B] out: b's number among the gate-on images, -1 if closed.
 *   on_list  int32 [B] out: on_list[r] = the gate-on image numbered r, for
 *            r < n_on; -1 after that.
 *   n_on     int32 [1] out (device): number of gate-on images.
 *
 * Returns DORA_OK or a negative dora_status; enqueues one single-workgroup
 * kernel.
 */
int dora_actor_gate(const float* p_gate, const int32_t* cu_in, int32_t B, int32_t N, int32_t M,
                    int32_t* on_rank, int32_t* on_list, int32_t* n_on, int32_t* dev_status, void* stream);

/*
 * dora_actor_decode -- budget and keep-scores of the deterministic actor
 * (App. A.3: the legal budget with the largest logit; the k highest removal
 * scores are deleted; Sec. 3.2, Eq. (2) for the scores).
 *
 *   budget_logits  fp32 [logit_rows, M]: row r holds the budget-head logits
 *            of gate-on image on_list[r] (the controller's sub-batch order).
 *            The budget of image b is k = 2(m + 1) for the m < (number of
 *            legal budgets) with the largest logit: the first such m on ties,
 *            a NaN logit above every number (the first NaN wins), as an
 *            argmax with the illegal budgets masked out.
 *   removal_scores, scores_out  fp32, both NULL or both given, in the score
 *            layout of dora_select_pack ([B, N] dense, [total_in] packed):
 *            scores_out = -removal_scores element by element (the keep-scores
 *            dora_select_pack takes).  They may be the same buffer.
 *   cu_in, total_in, B, N  as for dora_select_pack (cu_in NULL: dense).
 *   on_rank  int32 [B] from dora_actor_gate.
 *   keep_out int32 [B] out: n_b - k for a gate-on image, n_b for a gate-off
 *            one (nothing removed); 0 with DORA_DEV_CU_IN for an invalid
 *            segment; n_b with DORA_DEV_ACTOR for a gate-on image with no
 *            legal budget or with on_rank[b] >= logit_rows.
 *
 * Returns DORA_OK or a negative dora_status; enqueues one kernel.
 */
int dora_actor_decode(const float* budget_logits, int64_t logit_rows, int32_t M, const float* removal_scores,
                      const int32_t* cu_in, int64_t total_in, int32_t B, int32_t N, const int32_t* on_rank,
                      int32_t* keep_out, float* scores_out, int32_t* dev_status, void* stream);

/*
 * dora_pl_sample -- Plackett-Luce deletion by Gumbel-top-k, with the ordered
 * log-probability of the draw (Sec. 3.2 "Sampling and deployment": training
 * draws exactly k distinct tokens without replacement and keeps the order;
 * App. A.3, Eq. (app-actor-pl)).
 *
 * For image b (segment as in dora_select_pack; position 0 is CLS and is never
 * drawn): key_j = scores_j + gumbel_j in FP32 for the visual positions, and
 * the k[b] positions drawn are the first k[b] in decreasing key order (NaN
 * keys first, equal keys by higher position: the order in which
 * dora_select_pack with keep-scores -key and keep = n_b - k[b] deletes).
 * With gumbel i.i.d. standard Gumbel noise this is a Plackett-Luce sample
 * over exp(scores).  logprob_out[b] = sum_t [ s_{i_t} - log sum_{j in R_t}
 * exp(s_j) ] over the draws i_1..i_k, R_t the visual positions not drawn
 * before step t, in fp32 (each exp relative to the largest visual score).
 *
 *   scores     fp32 removal scores (higher = remove; Sec. 3.2, Eq. (2)),
 *              [B, N] dense (cu_in NULL) or [total_in] packed.  Finite.
 *   gumbel     fp32, the noise, same layout (the caller draws it).
 *   k          int32 [B], 0 .. n_b - 1.
 *   order_out  int32 [cap]: the draws of image b, in drawing order, at
 *              [cu_order_out[b], cu_order_out[b+1]); positions local to the
 *              segment (1 .. n_b - 1).
 *   cu_order_out  int32 [B+1]: running total of k.
 *   logprob_out   fp32 [B].
 *   B 1 .. 8192; N 1 .. DORA_MAX_ROW_TOKENS; cap 1 .. 2^31-1.
 *   dev_status DORA_DEV_KEEP_RANGE for a k[b] outside [0, n_b - 1] (its
 *              slots are left unwritten, logprob NaN), DORA_DEV_CU_IN for an
 *              invalid segment, DORA_DEV_CAPACITY when sum k > cap (draws at
 *              or past cap are not written).
 *
 * Returns DORA_OK or a negative dora_status; enqueues one kernel.
 */
int dora_pl_sample(const float* scores, const float* gumbel, const int32_t* k, const int32_t* cu_in,
                   int64_t total_in, int32_t B, int32_t N, int32_t* order_out, int32_t* cu_order_out,
                   float* logprob_out, int64_t cap, int32_t* dev_status, void* stream);

/*
 * dora_pl_logprob -- the ordered log-probability of given draws under
 * (other) scores (App. A.3: the same action is scored under the old and the
 * new policy), as in dora_pl_sample.
 *
 *   order, cu_order  as written by dora_pl_sample (order holds cu_order[B]
 *              entries; cu_order[0] = 0, non-decreasing): distinct visual
 *              positions per image.  An image whose offsets break this gets
 *              NaN and DORA_DEV_KEEP_RANGE, and none of its entries is read.
 *   logprob_out fp32 [B]; NaN with DORA_DEV_KEEP_RANGE when an image's list
 *              is longer than n_b - 1, repeats a position or holds one outside
 *              1 .. n_b - 1.
 * Other arguments as for dora_pl_sample.  Returns DORA_OK or a negative
 * dora_status; enqueues one kernel.
 */
int dora_pl_logprob(const float* scores, const int32_t* order, const int32_t* cu_order, const int32_t* cu_in,
                    int64_t total_in, int32_t B, int32_t N, float* logprob_out, int32_t* dev_status,
                    void* stream);

/*
 * dora_lc1_readout -- readout input of a DINOv2 linear classifier on the
 * packed, pruned tokens (App. E.3 "Baseline implementations": the LC1 readout
 * joins the normalised CLS token with the mean of the normalised surviving
 * visual tokens), fused with the backbone's final LayerNorm.  For sequence b
 * (rows [cu_seqlens[b], cu_seqlens[b+1]) of x; the first is CLS):
 *   LN(x_j)        = (x_j - mean(x_j)) / sqrt(var(x_j) + eps) * gamma + beta
 *                    (mean and biased variance over the C channels)
 *   out[b, 0:C]    = LN(x_CLS)
 *   out[b, C:2C]   = mean of LN(x_j) over the sequence's other rows
 *                    (NaN when only CLS survives).
 * Arithmetic in fp32 from the exact input values; 1 / sqrt(var + eps) comes
 * from the hardware reciprocal square root (within about 1 ulp).
 *
 *   x          dtype [total, C], 16-byte aligned; C * sizeof(dtype) a multiple
 *              of 16 and at most 4096 bytes (else DORA_ERR_UNSUPPORTED).
 *   cu_seqlens int32 [B+1]; a sequence that is empty or reaches past total
 *              sets DORA_DEV_CU_SEQLENS and gets a NaN output row.
 *   gamma, beta fp32 [C]; eps >= 0 (DINOv2: 1e-6).
 *   out        fp32 [B, 2C].
 *   B          1 .. 2^24.
 *   workspace  NULL: one workgroup per sequence.  Otherwise device memory of
 *              at least dora_lc1_readout_workspace_size(B, C) bytes, 256-byte
 *              aligned (else DORA_ERR_WORKSPACE / DORA_ERR_ALIGN), with no
 *              required contents: when the batch is small against the GPU,
 *              the rows of a sequence are split over up to 8 workgroups,
 *              which write their sums there, and a second kernel adds them in
 *              a fixed order (the result does not depend on timing).  Calls
 *              that share a workspace must not overlap in time.
 *
 * Returns DORA_OK or a negative dora_status; enqueues one kernel, or two when
 * the rows are split.
 */
size_t dora_lc1_readout_workspace_size(int32_t B, int32_t C);  /* 0 when B or C is out of range */
int dora_lc1_readout(const void* x, const int32_t* cu_seqlens, int64_t total, int32_t B, int32_t C,
                     dora_dtype dtype, const float* gamma, const float* beta, float eps, float* out,
                     void* workspace, size_t workspace_bytes, int32_t* dev_status, void* stream);

/* Backbone shape for dora_trajectory_flops (Table 3; DINOv2's LC1 readout has
 * head_inputs = 2).  actor: 1 to count DORA's actor, 0 for the bare backbone. */
typedef struct {
  int32_t d;           /* token width                                        */
  int32_t L;           /* blocks                                             */
  int32_t N0;          /* visual tokens at the input (patches)               */
  int32_t patch;       /* patch side; the embedding is in_chans*patch^2 -> d */
  int32_t in_chans;    /* image channels (3)                                 */
  int32_t classes;     /* classifier outputs (1000)                          */
  int32_t head_inputs; /* classifier input width in units of d               */
  int32_t mlp_ratio;   /* MLP hidden width in units of d (4)                 */
  int32_t M;           /* budget-head outputs, (N0 - 4) / 2                  */
  int32_t actor;       /* 0 or 1                                             */
} dora_flops_config;

/*
 * dora_trajectory_flops -- FLOPs of the complete forward of each image along
 * its realised token trajectory (App. E.4, Eq. (app-experiments-flops) before
 * averaging): two per multiply-accumulate of the patch embedding, every
 * linear layer, the two attention products and the classifier.  At block l
 * the attention runs over tokens[l] tokens and the MLP over tokens[l+1]
 * (CLS included).  With actor = 1 (App. A.1): the gate (d + 19 -> 64 -> 1)
 * at every block whose visual tokens allow a budget (N_l >= 6), and where
 * tokens were removed the controller: d -> 128 projection of every key,
 * 3 -> 128 history projection, a width-128 Transformer block (4 heads, FFN
 * 128 -> 256 -> 128), budget head 128 -> 128 -> M, the 1 -> 128 projection of
 * k / N and the selector 128 -> 64 -> 1 on the visual tokens.  LayerNorm,
 * softmax, activations and additions are not counted.
 *
 *   tokens     device int32 [L+1, B]: tokens[0][b] = N0 + 1 and
 *              1 <= tokens[l+1][b] <= tokens[l][b].  An image that breaks
 *              this gets flops_out = -1, is left out of the total and sets
 *              DORA_DEV_KEEP_RANGE.
 *   config     host pointer, read during the call.
 *   flops_out  device int64 [B]; total_out device int64 [1]: the sum over the
 *              valid images.
 *   B 1 .. 2^24.
 * Returns DORA_OK or a negative dora_status (DORA_ERR_SHAPE for a config
 * field out of range); enqueues one single-workgroup kernel.
 */
int dora_trajectory_flops(const int32_t* tokens, int32_t B, const dora_flops_config* config, int64_t* flops_out,
                          int64_t* total_out, int32_t* dev_status, void* stream);

/*
 * dora_varlen_attn_execute -- exact softmax attention inside each packed
 * sequence (Sec. 3.5 "Inference"; App. E.5): for every sequence b and head h
 *   O_b,h = softmax(softmax_scale * Q_b,h K_b,h^T) V_b,h
 * with no causal mask, no bias and no attention across sequence boundaries.
 *
 *   q, k, v    dtype [total, H, D] contiguous, 16-byte aligned.
 *   out        dtype [total, H, D]; rows outside every sequence are not written.
 *   D          must be DORA_HEAD_DIM (64).
 *   softmax_scale  <= 0 selects 1/sqrt(D).
 *   dtype      DORA_BF16: bf16 inputs, fp32 accumulation and softmax, P rounded
 *              to bf16 for the P.V product, output rounded once to bf16.
 *              DORA_F32: fp32 throughout.
 *   workspace  as filled by dora_varlen_attn_plan (or dora_select_pack_plan)
 *              with the same cu_seqlens, B, H, max_seqlen and total; otherwise
 *              DORA_DEV_PLAN is set and nothing is written.
 * Execute calls that share one workspace must not overlap in time.
 */
int dora_varlen_attn_execute(const void* q, const void* k, const void* v,
                             const int32_t* cu_seqlens, int32_t B, int32_t H, int32_t D,
                             int32_t max_seqlen, int64_t total, float softmax_scale,
                             dora_dtype dtype, void* out, void* workspace,
                             size_t workspace_bytes, int32_t* dev_status, void* stream);

/* dora_varlen_attn -- dora_varlen_attn_plan followed by dora_varlen_attn_execute. */
int dora_varlen_attn(const void* q, const void* k, const void* v, const int32_t* cu_seqlens,
                     int32_t B, int32_t H, int32_t D, int32_t max_seqlen, int64_t total,
                     float softmax_scale, dora_dtype dtype, void* out, void* workspace,
                     size_t workspace_bytes, int32_t* dev_status, void* stream);

/*
 * dora_varlen_attn_noalloc -- dora_varlen_attn for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops or
 * harnesses that forbid allocation).  The plan and work queue live in a
 * library-owned static device array of DORA_NOALLOC_WORKSPACE_BYTES instead
 * of a caller workspace; every GPU the library runs on holds its own copy
 * until the process ends.  The call allocates nothing (no hipMalloc, no
 * allocating library routine); the caller still passes inputs and outputs.
 *
 * Arguments, results and dev_status bits are those of dora_varlen_attn
 * without workspace / workspace_bytes.  Outputs are bit-identical to
 * dora_varlen_attn's (the same two kernels run; the plan kernel rewrites
 * the whole header, counters included, on every call, so nothing of an
 * earlier call's contents is used).
 *
 * Limit: dora_varlen_attn_workspace_size(B, H, max_seqlen) must not exceed
 * DORA_NOALLOC_WORKSPACE_BYTES (4 MiB: about 524,000 (sequence, head,
 * query chunk) items), else DORA_ERR_STATIC_LIMIT before anything is
 * enqueued.
 * Concurrency: every call on one GPU shares that GPU's array, so calls that
 * overlap in time on one GPU (several streams or host threads) race and
 * give undefined results; calls must be serialised, e.g. on one stream.
 * The first call on each device looks up the array's device address
 * (hipGetSymbolAddress) and keeps it; DORA_ERR_HIP if that fails.
 */
#define DORA_NOALLOC_WORKSPACE_BYTES (4u << 20)
int dora_varlen_attn_noalloc(const void* q, const void* k, const void* v, const int32_t* cu_seqlens,
                             int32_t B, int32_t H, int32_t D, int32_t max_seqlen, int64_t total,
                             float softmax_scale, dora_dtype dtype, void* out, int32_t* dev_status,
                             void* stream);

/* Human-readable name of a dora_status value (static string). */
const char* dora_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* DORA_H_ */
