/*
 * Plain CPU oracle for the DORA deployment hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or constant with the GPU path.
 *
 * What it computes (DORA, arXiv 2609.34325):
 *   - Deployment keep rule (Sec. 3.2 "Sampling and deployment", App. A.3):
 *     the selector removes the highest-scoring visual tokens and CLS is never
 *     removed; deletion preserves CLS and the relative order of survivors
 *     (Sec. 3.1, pruning operator, Eq. (1)).  Here scores are keep-scores
 *     (higher = keep), so an image keeps CLS plus its keep-1 highest-scoring
 *     visual tokens.  Score comparisons are FP32 values (App. E.5).
 *   - Packing (Sec. 3.5 "Inference"): survivors of all images are compacted
 *     into one buffer with explicit sequence boundaries.
 *   - Attention (Sec. 3.5, App. E.5): exact softmax attention inside each
 *     sequence boundary, with no attention between images, no bias term and
 *     no token-size correction.
 *
 * Readings where the paper is silent (listed with the tests that pin them):
 *   - Ties: equal scores are broken by the lower position (a stable order).
 *   - NaN ranks below every number; NaNs tie with each other.  -0 == +0.
 *   - Softmax scale is a parameter (1/sqrt(64) for ViT heads of width 64).
 *   - Residual before deletion (Sec. 3.1, Eq. (1): the rows are removed from
 *     H + Attention(...), not from H): each element of the sum is the exact
 *     sum of the two stored values rounded once, to nearest with ties to
 *     even, into the storage format (bf16 or fp32); subnormals are kept and
 *     a sum past the largest finite value becomes infinity.
 *
 * Everything is computed the slow, direct way: a full sort per image and a
 * dense fp64 score matrix per (image, head).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Return codes of oracle_select_pack (bit set). */
#define ORACLE_BAD_KEEP 1      /* some keep[b] outside [1, n_b]                 */
#define ORACLE_OVERFLOW 2      /* sum of keep exceeds the output capacity        */
#define ORACLE_BAD_SEGMENTS 4  /* packed input offsets are not a valid partition */

typedef struct {
  float score;
  int32_t pos;
} candidate;

/* Total order on candidates: "a before b" when a is preferred for keeping.
 * Non-NaN before NaN; larger score first (IEEE compare, so -0 == +0);
 * equal scores and NaN-vs-NaN by ascending position. */
static int candidate_order(const void* pa, const void* pb) {
  const candidate* a = (const candidate*)pa;
  const candidate* b = (const candidate*)pb;
  int an = isnan(a->score), bn = isnan(b->score);
  if (an != bn) return an ? 1 : -1;
  if (!an) {
    double x = (double)a->score, y = (double)b->score;
    if (x > y) return -1;
    if (x < y) return 1;
  }
  return (a->pos < b->pos) ? -1 : (a->pos > b->pos) ? 1 : 0;
}

static int ascending_int(const void* pa, const void* pb) {
  int32_t a = *(const int32_t*)pa, b = *(const int32_t*)pb;
  return (a < b) ? -1 : (a > b) ? 1 : 0;
}

/*
 * Select + pack.
 *   scores  : dense [B*N] (cu_in == NULL) or packed [total_in] fp32
 *   keep    : [B], keep count including CLS
 *   tokens  : rows of row_bytes bytes, dense [B*N] rows or packed [total_in] rows
 *   cu_in   : NULL (dense, every segment has N rows) or [B+1] segment offsets
 *   idx_out : [sum keep] kept positions, local to each segment, ascending
 *   cu_out  : [B+1] output sequence boundaries
 *   packed  : [sum keep] rows
 * Returns 0 or a bitwise OR of ORACLE_* codes; on error nothing is written.
 */
int oracle_select_pack(const float* scores, const int32_t* keep, const uint8_t* tokens,
                       const int32_t* cu_in, int64_t total_in, int32_t B, int32_t N,
                       int64_t row_bytes,
                       int32_t* idx_out, int32_t* cu_out, uint8_t* packed, int64_t cap_rows) {
  int status = 0;
  int64_t* off_in = (int64_t*)malloc(sizeof(int64_t) * (size_t)(B > 0 ? B : 1));
  int64_t* n_in = (int64_t*)malloc(sizeof(int64_t) * (size_t)(B > 0 ? B : 1));
  int64_t total = 0;
  for (int32_t b = 0; b < B; ++b) {
    if (cu_in) {
      off_in[b] = cu_in[b];
      n_in[b] = (int64_t)cu_in[b + 1] - cu_in[b];
      if ((b == 0 && cu_in[0] != 0) || cu_in[b] < 0 || n_in[b] < 1 || n_in[b] > N ||
          cu_in[b + 1] > total_in)
        status |= ORACLE_BAD_SEGMENTS;
    } else {
      off_in[b] = (int64_t)b * N;
      n_in[b] = N;
    }
    if (keep[b] < 1 || keep[b] > n_in[b]) status |= ORACLE_BAD_KEEP;
    total += keep[b];
  }
  if (total > cap_rows) status |= ORACLE_OVERFLOW;
  if (status) {
    free(off_in);
    free(n_in);
    return status;
  }

  /* Sequence boundaries: running total of keep counts. */
  cu_out[0] = 0;
  for (int32_t b = 0; b < B; ++b) cu_out[b + 1] = cu_out[b] + keep[b];

#pragma omp parallel for schedule(dynamic)
  for (int32_t b = 0; b < B; ++b) {
    const int64_t n = n_in[b];
    const float* s = scores + off_in[b];
    candidate* cand = (candidate*)malloc(sizeof(candidate) * (size_t)n);
    int32_t* kept = idx_out + cu_out[b];
    /* Visual tokens are positions 1..n-1; CLS (position 0) is not a candidate. */
    for (int64_t j = 1; j < n; ++j) {
      cand[j - 1].score = s[j];
      cand[j - 1].pos = (int32_t)j;
    }
    qsort(cand, (size_t)(n - 1), sizeof(candidate), candidate_order);
    kept[0] = 0;
    for (int32_t r = 0; r < keep[b] - 1; ++r) kept[r + 1] = cand[r].pos;
    /* Survivors keep their original relative order. */
    qsort(kept, (size_t)keep[b], sizeof(int32_t), ascending_int);
    for (int32_t r = 0; r < keep[b]; ++r)
      memcpy(packed + (size_t)(cu_out[b] + r) * (size_t)row_bytes,
             tokens + (size_t)(off_in[b] + kept[r]) * (size_t)row_bytes, (size_t)row_bytes);
    free(cand);
  }
  free(off_in);
  free(n_in);
  return 0;
}

/*
 * Dense softmax attention per sequence and head, fp64.
 *   q, k, v, out : [total, H, D] row-major, already widened to double
 *   cu           : [B+1] sequence boundaries
 * O_b = softmax(scale * Q_b K_b^T) V_b for every sequence b and head h.
 */
/* Output of query row i (head h) of the sequence at rows [start, start + len):
 * a dense fp64 logit row, its softmax, and the weighted sum of V. */
static void attend_row(const double* q, const double* k, const double* v, int64_t start, int64_t len, int64_t i,
                       int32_t H, int32_t h, int32_t D, double scale, double* logits, double* oi) {
  const double* qi = q + (i * H + h) * D;
  double mx = -INFINITY;
  for (int64_t j = 0; j < len; ++j) {
    const double* kj = k + ((start + j) * H + h) * D;
    double dot = 0.0;
    for (int32_t d = 0; d < D; ++d) dot += qi[d] * kj[d];
    logits[j] = scale * dot;
    if (logits[j] > mx) mx = logits[j];
  }
  double z = 0.0;
  for (int64_t j = 0; j < len; ++j) {
    logits[j] = exp(logits[j] - mx);
    z += logits[j];
  }
  for (int32_t d = 0; d < D; ++d) oi[d] = 0.0;
  for (int64_t j = 0; j < len; ++j) {
    const double* vj = v + ((start + j) * H + h) * D;
    const double p = logits[j] / z;
    for (int32_t d = 0; d < D; ++d) oi[d] += p * vj[d];
  }
}

void oracle_varlen_attn(const double* q, const double* k, const double* v, const int32_t* cu,
                        int32_t B, int32_t H, int32_t D, double scale, double* out,
                        int32_t nthreads) {
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int32_t b = 0; b < B; ++b) {
    for (int32_t h = 0; h < H; ++h) {
      const int64_t start = cu[b];
      const int64_t len = (int64_t)cu[b + 1] - cu[b];
      if (len <= 0) continue;
      double* logits = (double*)malloc(sizeof(double) * (size_t)len);
      for (int64_t i = 0; i < len; ++i)
        attend_row(q, k, v, start, len, start + i, H, h, D, scale, logits, out + ((start + i) * H + h) * D);
      free(logits);
    }
  }
}

/* Round x to the nearest value of a binary floating-point format with p
 * significand bits (hidden bit included), smallest normal exponent emin and
 * largest exponent emax; a tie goes to the even significand.  A result at or
 * past 2^(emax+1) is infinity.  NaN, infinities and zeros pass through. */
static double round_nearest_even(double x, int p, int emin, int emax) {
  if (!isfinite(x) || x == 0.0) return x;
  int e;
  frexp(fabs(x), &e);                           /* |x| = m 2^e, 1/2 <= m < 1 */
  const int lead = (e - 1 < emin) ? emin : e - 1; /* exponent of the leading bit, subnormals at emin */
  const double quantum = ldexp(1.0, lead - (p - 1));
  const double k = fabs(x) / quantum;           /* exact: power-of-two scaling */
  double n = floor(k);
  const double frac = k - n;
  if (frac > 0.5 || (frac == 0.5 && fmod(n, 2.0) != 0.0)) n += 1.0;
  double r = n * quantum;
  if (r >= ldexp(1.0, emax + 1)) r = INFINITY;
  return copysign(r, x);
}

/* x rounded to bf16 (is_bf16 != 0) or fp32, written as its bit pattern
 * (uint16 or uint32) into out[i]. */
void oracle_round_to_format(const double* x, int64_t n, int32_t is_bf16, void* out) {
  for (int64_t i = 0; i < n; ++i) {
    const float f = (float)round_nearest_even(x[i], is_bf16 ? 8 : 24, -126, 127); /* exact */
    uint32_t bits;
    memcpy(&bits, &f, sizeof bits);
    if (is_bf16) ((uint16_t*)out)[i] = (uint16_t)(bits >> 16);
    else ((uint32_t*)out)[i] = bits;
  }
}

static double stored_value(const void* v, int64_t i, int32_t is_bf16) {
  uint32_t bits;
  float f;
  if (is_bf16) bits = (uint32_t)((const uint16_t*)v)[i] << 16;
  else bits = ((const uint32_t*)v)[i];
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

/* out = h + a elementwise over n values of bf16 (is_bf16 != 0) or fp32 bit
 * patterns.  The sum of two such values in fp64 is either exact or rounded
 * with at least 2p+2 significand bits to spare, so rounding it once more to
 * the storage format gives the correctly rounded sum. */
void oracle_residual_add(const void* h, const void* a, int64_t n, int32_t is_bf16, void* out) {
  for (int64_t i = 0; i < n; ++i) {
    const double s = stored_value(h, i, is_bf16) + stored_value(a, i, is_bf16);
    oracle_round_to_format(&s, 1, is_bf16, is_bf16 ? (void*)((uint16_t*)out + i) : (void*)((uint32_t*)out + i));
  }
}

/* Number of legal budgets of an image of n_tok tokens (CLS included), by
 * enumerating the grid 2, 4, ..., 2M. */
static int32_t legal_budget_count(int32_t n_tok, int32_t M) {
  int32_t count = 0;
  for (int32_t m = 0; m < M; ++m)
    if (2 * (m + 1) <= (n_tok - 1) - 4) ++count;
  return count;
}

/* Deterministic actor decode, gate (Sec. 3.2 "Sampling and deployment";
 * Sec. 3.2 "Gate"; App. A.2, Eq. (legal budgets); App. A.3).  Image b holds
 * n_tok[b] tokens with CLS, so N_l = n_tok[b] - 1 visual tokens.  The legal
 * budgets are the even counts k = 2, 4, ..., 2M with k <= N_l - 4; the gate
 * opens when p_gate[b] >= 0.5 and at least one budget is legal.  Gate-on
 * images are numbered in image order: on_rank[b] is b's number (-1 when the
 * gate is off), on_list[r] the image numbered r (-1 past the last), *n_on the
 * count. */
void oracle_actor_gate(const float* p_gate, const int32_t* n_tok, int32_t B, int32_t M, int32_t* on_rank,
                       int32_t* on_list, int32_t* n_on) {
  int32_t r = 0;
  for (int32_t b = 0; b < B; ++b) on_list[b] = -1;
  for (int32_t b = 0; b < B; ++b) {
    const int open = p_gate[b] >= 0.5f && legal_budget_count(n_tok[b], M) > 0;
    on_rank[b] = open ? r : -1;
    if (open) on_list[r++] = b;
  }
  *n_on = r;
}

/* Deterministic actor decode, budget and keep counts (App. A.3: the highest
 * legal budget logit, then the k highest removal scores are deleted).  Row
 * on_rank[b] of logits [rows, M] belongs to gate-on image b; the budget is
 * the legal k = 2(m+1) of the largest logit, the first on ties, NaN above
 * every number (so the first NaN wins), as an argmax over the logits with the
 * illegal budgets masked out.  keep[b] = n_tok[b] - k (CLS is never removed);
 * a gate-off image keeps all n_tok[b] tokens. */
void oracle_actor_budget(const float* logits, int32_t M, const int32_t* n_tok, const int32_t* on_rank,
                         int32_t B, int32_t* keep) {
  for (int32_t b = 0; b < B; ++b) {
    if (on_rank[b] < 0) {
      keep[b] = n_tok[b];
      continue;
    }
    const float* row = logits + (int64_t)on_rank[b] * M;
    const int32_t legal = legal_budget_count(n_tok[b], M);
    int32_t best = 0;
    for (int32_t m = 1; m < legal; ++m) {
      const float x = row[m], y = row[best];
      if (isnan(y)) break;
      if (isnan(x) || x > y) best = m;
    }
    keep[b] = n_tok[b] - 2 * (best + 1);
  }
}

/* Keep-scores from the selector's removal scores (Sec. 3.2, Eq. (2): higher
 * = remove): out = -s, elementwise. */
void oracle_negate(const float* s, int64_t n, float* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = -s[i];
}

/* Removal order of the Plackett-Luce sample: "a before b" when a is drawn
 * (removed) earlier.  This is the keep order of candidate_order on the
 * keep-score -key, reversed, so that the drawn set is exactly what select +
 * pack deletes with keep-scores -key: NaN keys first, then larger keys, equal
 * keys (and NaN vs NaN) by descending position. */
static int removal_order(const void* pa, const void* pb) {
  const candidate* a = (const candidate*)pa;
  const candidate* b = (const candidate*)pb;
  int an = isnan(a->score), bn = isnan(b->score);
  if (an != bn) return an ? -1 : 1;
  if (!an) {
    double x = (double)a->score, y = (double)b->score;
    if (x > y) return -1;
    if (x < y) return 1;
  }
  return (a->pos > b->pos) ? -1 : (a->pos < b->pos) ? 1 : 0;
}

/* Segment geometry shared by the Plackett-Luce functions; returns nonzero
 * when cu_in is not a valid partition. */
static int segments(const int32_t* cu_in, int64_t total_in, int32_t B, int32_t N, int64_t* off, int64_t* n) {
  int bad = 0;
  for (int32_t b = 0; b < B; ++b) {
    if (cu_in) {
      off[b] = cu_in[b];
      n[b] = (int64_t)cu_in[b + 1] - cu_in[b];
      if ((b == 0 && cu_in[0] != 0) || cu_in[b] < 0 || n[b] < 1 || n[b] > N || cu_in[b + 1] > total_in) bad = 1;
    } else {
      off[b] = (int64_t)b * N;
      n[b] = N;
    }
  }
  return bad;
}

/* Ordered Plackett-Luce log-probability (App. A.3, Eq. (app-actor-pl)) of
 * drawing the visual positions order[0..k) in that order from one image's
 * removal scores s[1..n) (position 0, CLS, never drawn):
 *   sum_t [ s_{i_t} - log sum_{j in R_t} exp(s_j) ],
 *   R_t = visual positions not drawn before step t,
 * in fp64, each exp taken relative to the largest visual score (the same
 * value, without overflow).  Scores are expected finite. */
static double pl_logprob_one(const float* s, int64_t n, const int32_t* order, int32_t k) {
  char* drawn = (char*)calloc((size_t)n, 1);
  double m = -INFINITY;
  for (int64_t j = 1; j < n; ++j) m = fmax(m, (double)s[j]);
  double lp = 0.0;
  for (int32_t t = 0; t < k; ++t) {
    double z = 0.0;
    for (int64_t j = 1; j < n; ++j)
      if (!drawn[j]) z += exp((double)s[j] - m);
    lp += ((double)s[order[t]] - m) - log(z);
    drawn[order[t]] = 1;
  }
  free(drawn);
  return lp;
}

/*
 * Plackett-Luce deletion by Gumbel-top-k (Sec. 3.2 "Sampling and deployment";
 * App. A.3, Eq. (app-actor-pl)).  For image b with removal scores s and
 * Gumbel noise g (same layout as the scores of oracle_select_pack; position 0
 * is CLS and is never drawn), key_j = s_j + g_j in FP32, and the k[b] visual
 * positions drawn are the first k[b] in removal_order of the keys: a
 * Plackett-Luce sample without replacement over exp(s).
 *   order_out : [sum k] drawn positions, image after image, in drawing order
 *   cu_order  : [B+1] offsets of each image's list
 *   logprob   : [B] ordered log-probability of the list under s (fp64)
 * k[b] must lie in [0, n_b - 1].  Returns 0 or ORACLE_* bits (nothing written).
 */
int oracle_pl_sample(const float* s, const float* g, const int32_t* k, const int32_t* cu_in, int64_t total_in,
                     int32_t B, int32_t N, int32_t* order_out, int32_t* cu_order, double* logprob, int64_t cap) {
  int64_t* off = (int64_t*)malloc(sizeof(int64_t) * (size_t)(B > 0 ? B : 1));
  int64_t* n = (int64_t*)malloc(sizeof(int64_t) * (size_t)(B > 0 ? B : 1));
  int status = segments(cu_in, total_in, B, N, off, n) ? ORACLE_BAD_SEGMENTS : 0;
  int64_t total = 0;
  for (int32_t b = 0; b < B; ++b) {
    if (k[b] < 0 || k[b] > n[b] - 1) status |= ORACLE_BAD_KEEP;
    total += k[b];
  }
  if (total > cap) status |= ORACLE_OVERFLOW;
  if (status) {
    free(off);
    free(n);
    return status;
  }
  cu_order[0] = 0;
  for (int32_t b = 0; b < B; ++b) cu_order[b + 1] = cu_order[b] + k[b];
  candidate* cand = (candidate*)malloc(sizeof(candidate) * (size_t)(N > 0 ? N : 1));
  for (int32_t b = 0; b < B; ++b) {
    const float* sb = s + off[b];
    const float* gb = g + off[b];
    for (int64_t j = 1; j < n[b]; ++j) {
      const float key = sb[j] + gb[j]; /* FP32 sum */
      cand[j - 1].score = key;
      cand[j - 1].pos = (int32_t)j;
    }
    qsort(cand, (size_t)(n[b] - 1), sizeof(candidate), removal_order);
    int32_t* ob = order_out + cu_order[b];
    for (int32_t t = 0; t < k[b]; ++t) ob[t] = cand[t].pos;
    logprob[b] = pl_logprob_one(sb, n[b], ob, k[b]);
  }
  free(cand);
  free(off);
  free(n);
  return 0;
}

/* Ordered log-probability of given drawing orders (the same action scored
 * under another policy's scores): order/cu_order as written by
 * oracle_pl_sample. */
int oracle_pl_logprob(const float* s, const int32_t* order, const int32_t* cu_order, const int32_t* cu_in,
                      int64_t total_in, int32_t B, int32_t N, double* logprob) {
  int64_t* off = (int64_t*)malloc(sizeof(int64_t) * (size_t)(B > 0 ? B : 1));
  int64_t* n = (int64_t*)malloc(sizeof(int64_t) * (size_t)(B > 0 ? B : 1));
  int status = segments(cu_in, total_in, B, N, off, n) ? ORACLE_BAD_SEGMENTS : 0;
  for (int32_t b = 0; b < B && !status; ++b) {
    const int32_t kb = cu_order[b + 1] - cu_order[b];
    if (kb < 0 || kb > n[b] - 1) status |= ORACLE_BAD_KEEP;
    for (int32_t t = 0; t < kb && !status; ++t) {
      const int32_t j = order[cu_order[b] + t];
      if (j < 1 || j >= n[b]) status |= ORACLE_BAD_KEEP;
    }
  }
  if (!status)
    for (int32_t b = 0; b < B; ++b)
      logprob[b] = pl_logprob_one(s + off[b], n[b], order + cu_order[b], cu_order[b + 1] - cu_order[b]);
  free(off);
  free(n);
  return status;
}

/* LayerNorm of one row of C values (biased variance, eps inside the square
 * root, then the affine gamma, beta), in fp64. */
static void layer_norm_row(const double* x, int32_t C, const double* gamma, const double* beta, double eps,
                           double* y) {
  double mu = 0.0, var = 0.0;
  for (int32_t c = 0; c < C; ++c) mu += x[c];
  mu /= C;
  for (int32_t c = 0; c < C; ++c) var += (x[c] - mu) * (x[c] - mu);
  var /= C;
  const double r = 1.0 / sqrt(var + eps);
  for (int32_t c = 0; c < C; ++c) y[c] = (x[c] - mu) * r * gamma[c] + beta[c];
}

/*
 * Readout input of a DINOv2 linear classifier on pruned tokens (App. E.3
 * "Baseline implementations": the LC1 readout joins the normalised CLS token
 * with the mean of the normalised surviving visual tokens).  For image b with
 * packed rows [cu[b], cu[b+1]) (the first row is CLS):
 *   out[b, 0:C]  = LayerNorm(x_CLS)
 *   out[b, C:2C] = mean over the other rows of LayerNorm(x_j)
 * (0/0 = NaN when only CLS survives).  x holds the exact values, fp64.
 */
void oracle_lc1_readout(const double* x, const int32_t* cu, int32_t B, int32_t C, const double* gamma,
                        const double* beta, double eps, double* out) {
  double* y = (double*)malloc(sizeof(double) * (size_t)C);
  for (int32_t b = 0; b < B; ++b) {
    double* ob = out + (int64_t)b * 2 * C;
    const int64_t r0 = cu[b], r1 = cu[b + 1];
    layer_norm_row(x + r0 * C, C, gamma, beta, eps, ob);
    for (int32_t c = 0; c < C; ++c) ob[C + c] = 0.0;
    for (int64_t r = r0 + 1; r < r1; ++r) {
      layer_norm_row(x + r * C, C, gamma, beta, eps, y);
      for (int32_t c = 0; c < C; ++c) ob[C + c] += y[c];
    }
    for (int32_t c = 0; c < C; ++c) ob[C + c] /= (double)(r1 - r0 - 1);
  }
  free(y);
}

/* The same attention for selected query rows only: out[r] = the output of
 * packed row rows[r] (all heads), which attends to every key of its own
 * sequence.  Rows are found in their sequence by the offsets cu. */
void oracle_varlen_attn_rows(const double* q, const double* k, const double* v, const int32_t* cu,
                             int32_t B, int32_t H, int32_t D, double scale, const int64_t* rows, int64_t nrows,
                             double* out) {
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int64_t r = 0; r < nrows; ++r) {
    for (int32_t h = 0; h < H; ++h) {
      const int64_t i = rows[r];
      int32_t b = 0;
      while (b < B && cu[b + 1] <= i) ++b;
      const int64_t start = cu[b], len = (int64_t)cu[b + 1] - cu[b];
      double* logits = (double*)malloc(sizeof(double) * (size_t)len);
      attend_row(q, k, v, start, len, i, H, h, D, scale, logits, out + (r * H + h) * D);
      free(logits);
    }
  }
}

int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
