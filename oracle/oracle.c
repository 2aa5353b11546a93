/*
 * Reference oracle for sparse absorbed-MLA partial attention and the
 * log-sum-exp merge of partials.  TEST INFRASTRUCTURE ONLY: the tests, the
 * smoke check and the benchmark's CPU-baseline leg may load this library;
 * the product path never does.  It shares no code, header or table with the
 * GPU library.
 *
 * Plain, slow and written to be checked by eye against the paper
 * ("Move the Query, Not the Cache", arXiv 2606.01502):
 *   - Introduction and Section 3.2 (wire format): a token's key and value
 *     are one compressed latent vector; a routed query row is d_qk = 576
 *     wide (a 512-wide latent part and a 64-wide decoupled-RoPE part) and
 *     the partial output row is d_v = 512 wide.  Reading: key = [ckv ; kpe]
 *     (576), value = ckv (512); the up/down projections are absorbed outside.
 *   - Section 3.2: the holder sends back the softmax-weighted latent row for
 *     the keys it holds together with the two softmax statistics (maximum
 *     logit, denominator) that make an exact recombination possible.  Here
 *     those statistics are folded into lse = max + ln(denominator), natural
 *     log, next to the normalised output row.
 *   - Section 3.2: any positional rotation of the query happens at the
 *     requester, and Section 3.3: a selected cache entry keeps the position
 *     it was cached at.  So the holder applies no mask and no rotation.
 *   - Section 3.3 and Section 6.3: the selection-regime holder attends only
 *     the indexer's selected entries: here either 64-token blocks, or single
 *     tokens (an indexer's top-k tokens, the selection budgets that Section
 *     6.3 sweeps).
 *   - Section 2.2 and Section 3.3: partials are recombined by online softmax;
 *     the merge is commutative and has a zero-weight identity.
 *
 * Arithmetic: every input bit pattern is decoded exactly to double; all
 * sums are two-pass (all scores, then the max, then the sums) in natural
 * index order; exp/log are the C library's double routines.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_DLAT 512  /* latent width, d_v (Section 3.2)                 */
#define ORACLE_DPE 64    /* decoupled-RoPE width, d_qk - d_v (Section 3.2)   */
#define ORACLE_BLOCK 64  /* tokens per selectable cache block               */

/* bfloat16 -> double.  A bf16 value is the upper half of an IEEE binary32
 * bit pattern, so the decode is exact. */
double oracle_bf16_to_f64(uint16_t bits) {
  uint32_t u = ((uint32_t)bits) << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* OCP 8-bit float E4M3FN -> double, by the format's definition:
 * 1 sign bit, 4 exponent bits (bias 7), 3 mantissa bits; exponent field 0
 * encodes subnormals m * 2^-9; there are no infinities; S.1111.111 is NaN. */
double oracle_e4m3fn_to_f64(uint8_t code) {
  int sign = (code >> 7) & 1;
  int e = (code >> 3) & 0xF;
  int m = code & 0x7;
  double mag;
  if (e == 0xF && m == 0x7) return NAN;
  if (e == 0)
    mag = ldexp((double)m, -9);             /* (m / 8) * 2^(1 - 7) */
  else
    mag = ldexp(1.0 + (double)m / 8.0, e - 7);
  return sign ? -mag : mag;
}

/* kv_kind values */
#define ORACLE_KV_BF16 0
#define ORACLE_KV_E4M3FN 1

typedef struct {
  int kind;
  const void* ckv;        /* [P][64][512] */
  const void* kpe;        /* [P][64][64]  */
  const float* ckv_scale; /* [P], e4m3 only */
  const float* kpe_scale; /* [P], e4m3 only */
} kv_view;

/* Exact value of the cache entry ckv[b][t][d]. */
static double ckv_at(const kv_view* kv, int64_t b, int t, int d) {
  int64_t i = (b * ORACLE_BLOCK + t) * ORACLE_DLAT + d;
  if (kv->kind == ORACLE_KV_BF16) return oracle_bf16_to_f64(((const uint16_t*)kv->ckv)[i]);
  return oracle_e4m3fn_to_f64(((const uint8_t*)kv->ckv)[i]) * (double)kv->ckv_scale[b];
}

/* Exact value of the cache entry kpe[b][t][d]. */
static double kpe_at(const kv_view* kv, int64_t b, int t, int d) {
  int64_t i = (b * ORACLE_BLOCK + t) * ORACLE_DPE + d;
  if (kv->kind == ORACLE_KV_BF16) return oracle_bf16_to_f64(((const uint16_t*)kv->kpe)[i]);
  return oracle_e4m3fn_to_f64(((const uint8_t*)kv->kpe)[i]) * (double)kv->kpe_scale[b];
}

/*
 * Partial attention of every query row of every job over that job's
 * selected blocks.
 *
 *   q_lat [R][Mq][H][512], q_pe [R][Mq][H][64]  bf16 bit patterns
 *   ckv [P][64][512], kpe [P][64][64]           bf16 bits, or e4m3fn codes
 *                                               with per-block scales
 *   table [R][NB]  logical block of the job's chunk -> pool block
 *   sel            selected logical blocks, -1 = empty slot; a block listed
 *                  twice is attended twice (multiset).  sel_per_row = 0:
 *                  [R][K], one selection for all rows of a job; 1:
 *                  [R][Mq][K], a selection per query row (one holder serving
 *                  several routed requesters on one chunk, Section 6.3)
 *   sel_tokens     0: a slot names a logical block, all 64 of its tokens;
 *                  1: a slot names one logical token s of the chunk, token
 *                  s % 64 of logical block s / 64
 *   out   [R][Mq][H][512], lse [R][Mq][H]        double, written
 *   max_out, denom_out [R][Mq][H]                double, written unless NULL:
 *                  the two softmax statistics of Section 3.2's wire partial,
 *                  the largest score M and the denominator l = sum_T exp(s - M)
 *                  (so lse = M + ln l); an empty T gives M = -inf, l = 0
 *
 * For job r and row (i, h), with T the multiset of tokens (b, t) selected
 * for the row (by the job, or by query row i):
 *   s(b,t) = scale * (q_lat . ckv[b][t] + q_pe . kpe[b][t])
 *   lse    = ln sum_T exp(s)                    (via its maximum M)
 *   out    = sum_T exp(s - lse) * ckv[b][t]
 * and for an empty T: out = 0, lse = -inf.
 *
 * Returns 0, or -1 if a selected id or a table entry is out of range
 * (nothing is then guaranteed about out/lse).
 */
int oracle_partial(int R, int Mq, int H, int64_t P, int NB, int K,
                   const uint16_t* q_lat, const uint16_t* q_pe, int kv_kind,
                   const void* ckv, const void* kpe, const float* ckv_scale,
                   const float* kpe_scale, const int32_t* table, const int32_t* sel,
                   int sel_per_row, int sel_tokens, double scale, double* out, double* lse,
                   double* max_out, double* denom_out, int n_threads) {
  kv_view kv = {kv_kind, ckv, kpe, ckv_scale, kpe_scale};
  int bad = 0;
  if (kv_kind != ORACLE_KV_BF16 && kv_kind != ORACLE_KV_E4M3FN) return -1;
  if (kv_kind == ORACLE_KV_E4M3FN && (!ckv_scale || !kpe_scale)) return -1;

  /* Row i of job r reads its selection at sel + r * sel_s0 + i * sel_s1. */
  const int64_t sel_s1 = sel_per_row ? K : 0;
  const int64_t sel_s0 = sel_per_row ? (int64_t)Mq * K : K;
  const int n_sel = sel_per_row ? Mq : 1;
  /* A slot covers `per_slot` tokens; logical ids run below NB * per_slot. */
  const int per_slot = sel_tokens ? 1 : ORACLE_BLOCK;
  const int64_t n_ids = sel_tokens ? (int64_t)NB * ORACLE_BLOCK : NB;

  /* Check every selected id and table entry before computing anything. */
  for (int r = 0; r < R; ++r)
    for (int64_t jj = 0; jj < (int64_t)n_sel * K; ++jj) {
      int32_t s = sel[(int64_t)r * sel_s0 + jj];
      if (s == -1) continue;
      if (s < 0 || s >= n_ids) return -1;
      int32_t b = table[(int64_t)r * NB + (sel_tokens ? s / ORACLE_BLOCK : s)];
      if (b < 0 || (int64_t)b >= P) return -1;
    }

  int64_t n_rows = (int64_t)R * Mq * H;
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads) reduction(| : bad)
  for (int64_t row = 0; row < n_rows; ++row) {
    int r = (int)(row / ((int64_t)Mq * H));
    int i = (int)((row / H) % Mq);
    const int32_t* row_sel = sel + (int64_t)r * sel_s0 + (int64_t)i * sel_s1;
    const uint16_t* ql = q_lat + row * ORACLE_DLAT;
    const uint16_t* qp = q_pe + row * ORACLE_DPE;
    double* o = out + row * ORACLE_DLAT;

    /* The token multiset of this row, in slot order. */
    int n_tok = 0;
    for (int j = 0; j < K; ++j)
      if (row_sel[j] != -1) n_tok += per_slot;
    for (int d = 0; d < ORACLE_DLAT; ++d) o[d] = 0.0;
    if (n_tok == 0) {
      lse[row] = -INFINITY;
      if (max_out) max_out[row] = -INFINITY;
      if (denom_out) denom_out[row] = 0.0;
      continue;
    }
    double* score = (double*)malloc(sizeof(double) * (size_t)n_tok);
    int64_t* blk = (int64_t*)malloc(sizeof(int64_t) * (size_t)n_tok);
    int* tok = (int*)malloc(sizeof(int) * (size_t)n_tok);
    if (!score || !blk || !tok) {
      bad = 1;
      free(score); free(blk); free(tok);
      continue;
    }

    /* Pass 1: every score. */
    int n = 0;
    for (int j = 0; j < K; ++j) {
      int32_t s = row_sel[j];
      if (s == -1) continue;
      int64_t b = table[(int64_t)r * NB + (sel_tokens ? s / ORACLE_BLOCK : s)];
      int t0 = sel_tokens ? s % ORACLE_BLOCK : 0;
      for (int t = t0; t < t0 + per_slot; ++t) {
        double dot = 0.0;
        for (int d = 0; d < ORACLE_DLAT; ++d)
          dot += oracle_bf16_to_f64(ql[d]) * ckv_at(&kv, b, t, d);
        for (int d = 0; d < ORACLE_DPE; ++d)
          dot += oracle_bf16_to_f64(qp[d]) * kpe_at(&kv, b, t, d);
        score[n] = scale * dot;
        blk[n] = b;
        tok[n] = t;
        ++n;
      }
    }

    /* Pass 2: the maximum, then the normaliser, then the weighted values. */
    double M = score[0];
    for (int k = 1; k < n; ++k)
      if (score[k] > M) M = score[k];
    double l = 0.0;
    for (int k = 0; k < n; ++k) l += exp(score[k] - M);
    double L = M + log(l);
    lse[row] = L;
    if (max_out) max_out[row] = M;
    if (denom_out) denom_out[row] = l;
    for (int k = 0; k < n; ++k) {
      double w = exp(score[k] - L);
      for (int d = 0; d < ORACLE_DLAT; ++d) o[d] += w * ckv_at(&kv, blk[k], tok[k], d);
    }
    free(score); free(blk); free(tok);
  }
  return bad ? -1 : 0;
}

/*
 * Merge of n_parts partials of the same rows (Section 2.2, Section 3.3):
 *   o   [n_parts][n_rows][dv]   normalised partial outputs
 *   lam [n_parts][n_rows]       their log-sum-exps (natural log)
 * Per row, with live = { j : lam_j != -inf }:
 *   Lam = max_live lam_j,  lse = Lam + ln sum_live exp(lam_j - Lam),
 *   out = sum_live exp(lam_j - lse) * o_j;
 * an empty live set gives out = 0, lse = -inf.  A part with lam = -inf
 * contributes nothing, whatever its o holds (the zero-weight identity).
 */
int oracle_merge(int n_parts, int64_t n_rows, int dv, const double* o, const double* lam,
                 double* out, double* lse_out, int n_threads) {
  if (n_parts < 1 || dv < 1) return -1;
#pragma omp parallel for schedule(static) num_threads(n_threads)
  for (int64_t row = 0; row < n_rows; ++row) {
    double* y = out + row * dv;
    for (int d = 0; d < dv; ++d) y[d] = 0.0;
    int any = 0;
    double Lam = -INFINITY;
    for (int j = 0; j < n_parts; ++j) {
      double v = lam[(int64_t)j * n_rows + row];
      if (v == -INFINITY) continue;
      if (!any || v > Lam) Lam = v;
      any = 1;
    }
    if (!any) {
      if (lse_out) lse_out[row] = -INFINITY;
      continue;
    }
    double l = 0.0;
    for (int j = 0; j < n_parts; ++j) {
      double v = lam[(int64_t)j * n_rows + row];
      if (v == -INFINITY) continue;
      l += exp(v - Lam);
    }
    double L = Lam + log(l);
    if (lse_out) lse_out[row] = L;
    for (int j = 0; j < n_parts; ++j) {
      double v = lam[(int64_t)j * n_rows + row];
      if (v == -INFINITY) continue;
      double w = exp(v - L);
      const double* x = o + ((int64_t)j * n_rows + row) * dv;
      for (int d = 0; d < dv; ++d) y[d] += w * x[d];
    }
  }
  return 0;
}
