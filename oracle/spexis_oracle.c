/*
 * spexis_oracle.c -- plain, slow CPU reference of the speculative verification step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or load this
 * file or the library built from it; only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark do.  It shares no code, header, table or helper
 * with the HIP implementation: the cache layout, the softmax and the acceptance rule are
 * written out here again from their definitions.
 *
 * What it computes (Spexis, "Speculative-Parallel Execution" and Related Work, which cite
 * speculative decoding [sd]: the draft proposes k tokens, the full model verifies them in
 * one pass):
 *   oracle_append_kv   -- write the k+1 new K/V rows of every sequence into the paged cache
 *                         (the cache is shared by speculative and normal execution, Sec. 4).
 *   oracle_attention   -- causal, grouped-query attention of the k+1 query tokens of each
 *                         sequence over its paged KV, in fp64, straight from the definition.
 *   oracle_softmax     -- temperature softmax of fp32 logits, in fp64, rounded to fp32.
 *   oracle_lm_head     -- the output projection in front of acceptance (logits = h W^T over
 *                         bf16 inputs, in fp64) and each row's softmax statistics.
 *   oracle_linear      -- a linear layer of the drafting adapter (y = x W^T + residual, fp64).
 *   oracle_select_drafts -- acceptance-guided selective speculation: drop the alpha fraction of
 *                         the batch's draft tokens with the lowest confidence (Sec. 5).
 *   oracle_accept      -- speculative-sampling acceptance (accept x_i with probability
 *                         min(1, p_i(x_i)/q_i(x_i)); on the first rejection sample from the
 *                         normalised residual max(0, p - q); otherwise sample the bonus token
 *                         from p_k), with every decision taken in exact arithmetic so that any
 *                         correct implementation reaches the same integers.
 *   oracle_lookahead   -- the look-ahead KV-memory estimate of Algorithm 1 (Sec. 5).
 *
 * Cache layout (the library's documented format, restated here independently):
 *   K pool: bf16 [num_blocks][Hkv][D/8][bs][8]
 *           element (blk, h, slot, d) at ((((blk*Hkv + h)*(D/8) + d/8)*bs + slot)*8 + d%8)
 *   V pool: bf16 [num_blocks][Hkv][D][bs], the slot index stored with bits 2 and 3 swapped
 *           element (blk, h, slot, d) at (((blk*Hkv + h)*D + d)*bs + swap23(slot))
 *
 * Build: gcc -O2 -std=c11 -fopenmp -ffp-contract=off -shared -fPIC (no fast-math).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ---------------------------------------------------------------- helpers */

/* bf16 bit pattern -> double (exact: bf16 is the top half of an fp32). */
static double bf16_to_double(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

static int64_t swap23(int64_t slot) {
  int64_t b2 = (slot >> 2) & 1, b3 = (slot >> 3) & 1;
  return (slot & ~(int64_t)12) | (b2 << 3) | (b3 << 2);
}

static int64_t k_index(int64_t blk, int64_t h, int64_t slot, int64_t d, int64_t hkv, int64_t bs,
                       int64_t D) {
  return (((blk * hkv + h) * (D / 8) + d / 8) * bs + slot) * 8 + d % 8;
}

static int64_t v_index(int64_t blk, int64_t h, int64_t slot, int64_t d, int64_t hkv, int64_t bs,
                       int64_t D) {
  return ((blk * hkv + h) * D + d) * bs + swap23(slot);
}

/* ------------------------------------------------------------- append KV */

/*
 * For sequence b with n_b = qsl[b+1]-qsl[b] new tokens and post-append length S_b,
 * new token j sits at position L_b + j with L_b = S_b - n_b; its row goes to block
 * block_tables[b][pos/bs], slot pos%bs.  Returns 0, or -1 if an index is out of range
 * (a sequence with inconsistent lengths, or a token whose block id is out of range, is
 * skipped).
 */
int oracle_append_kv(uint16_t* k_pool, uint16_t* v_pool, int32_t num_blocks, int32_t hkv,
                     int32_t bs, int32_t D, int32_t B, const int32_t* qsl,
                     const int32_t* seq_lens, const int32_t* block_tables,
                     int32_t max_blocks_per_seq, const uint16_t* new_k, const uint16_t* new_v) {
  int rc = 0;
  for (int32_t b = 0; b < B; ++b) {
    int32_t n = qsl[b + 1] - qsl[b];
    int32_t L = seq_lens[b] - n;
    if (n < 1 || L < 0 || (seq_lens[b] + bs - 1) / bs > max_blocks_per_seq) { rc = -1; continue; }
    for (int32_t j = 0; j < n; ++j) {
      int64_t pos = (int64_t)L + j;
      int32_t blk = block_tables[(int64_t)b * max_blocks_per_seq + pos / bs];
      if (blk < 0 || blk >= num_blocks) { rc = -1; continue; }
      int64_t slot = pos % bs;
      int64_t row = (int64_t)qsl[b] + j;
      for (int32_t h = 0; h < hkv; ++h)
        for (int32_t d = 0; d < D; ++d) {
          int64_t src = (row * hkv + h) * D + d;
          k_pool[k_index(blk, h, slot, d, hkv, bs, D)] = new_k[src];
          v_pool[v_index(blk, h, slot, d, hkv, bs, D)] = new_v[src];
        }
    }
  }
  return rc;
}

/* ------------------------------------------------------------- attention */

/*
 * out[(qsl[b]+j)*Hq + h][d] = sum_t softmax_t(s) v[b,t,g][d], fp64, for every sequence b
 * listed in seqs[0..nseqs), query token j < n_b and query head h, where
 *   g = h / (Hq/Hkv)                     (contiguous query-head groups share a KV head)
 *   t ranges over 0 .. L_b + j           (a query sees the cache and itself, not later drafts)
 *   s_t = scale * <q[qsl[b]+j][h], k[b,t,g]>
 * Rows of sequences not listed are left untouched.  Returns -1 on an index out of range.
 */
int oracle_attention(const uint16_t* k_pool, const uint16_t* v_pool, int32_t num_blocks,
                     int32_t hkv, int32_t bs, int32_t D, int32_t B, const int32_t* qsl,
                     const int32_t* seq_lens, const int32_t* block_tables,
                     int32_t max_blocks_per_seq, const uint16_t* q, int32_t hq, float scale,
                     const int32_t* seqs, int32_t nseqs, double* out) {
  if (hkv <= 0 || hq % hkv != 0) return -1;
  int32_t G = hq / hkv;
  int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
  for (int32_t si = 0; si < nseqs; ++si) {
    int32_t b = seqs[si];
    if (b < 0 || b >= B) { bad |= 1; continue; }
    int32_t n = qsl[b + 1] - qsl[b];
    int32_t S = seq_lens[b];
    int32_t L = S - n;
    if (n < 1 || L < 0 || (S + bs - 1) / bs > max_blocks_per_seq) { bad |= 1; continue; }
    double* s = (double*)malloc(sizeof(double) * (size_t)S);
    for (int32_t j = 0; j < n; ++j) {
      for (int32_t h = 0; h < hq; ++h) {
        int32_t g = h / G;
        const uint16_t* qrow = q + ((int64_t)(qsl[b] + j) * hq + h) * D;
        int32_t last = L + j; /* keys 0..last are visible */
        double m = -INFINITY;
        for (int32_t t = 0; t <= last; ++t) {
          int32_t blk = block_tables[(int64_t)b * max_blocks_per_seq + t / bs];
          if (blk < 0 || blk >= num_blocks) { bad |= 1; blk = 0; }
          double dot = 0.0;
          for (int32_t d = 0; d < D; ++d)
            dot += bf16_to_double(qrow[d]) * bf16_to_double(k_pool[k_index(blk, g, t % bs, d, hkv, bs, D)]);
          s[t] = (double)scale * dot;
          if (s[t] > m) m = s[t];
        }
        double z = 0.0;
        for (int32_t t = 0; t <= last; ++t) { s[t] = exp(s[t] - m); z += s[t]; }
        double* o = out + ((int64_t)(qsl[b] + j) * hq + h) * D;
        for (int32_t d = 0; d < D; ++d) o[d] = 0.0;
        for (int32_t t = 0; t <= last; ++t) {
          int32_t blk = block_tables[(int64_t)b * max_blocks_per_seq + t / bs];
          if (blk < 0 || blk >= num_blocks) blk = 0;
          double w = s[t] / z;
          for (int32_t d = 0; d < D; ++d)
            o[d] += w * bf16_to_double(v_pool[v_index(blk, g, t % bs, d, hkv, bs, D)]);
        }
      }
    }
    free(s);
  }
  return bad ? -1 : 0;
}

/* --------------------------------------------------------------- softmax */

/*
 * probs[r][v] = exp((l_v - max l)/T) / sum_u exp((l_u - max l)/T), evaluated in fp64 from
 * the fp32 logits and fp32 temperature, then rounded to fp32.  Temperature divides the
 * logits of both the target and the draft rows before the softmax.
 */
void oracle_softmax(const float* logits, int64_t rows, int32_t V, float temperature, float* probs) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) {
    const float* x = logits + r * V;
    double m = -INFINITY;
    for (int32_t v = 0; v < V; ++v) if ((double)x[v] > m) m = (double)x[v];
    double* e = (double*)malloc(sizeof(double) * (size_t)V);
    double z = 0.0;
    for (int32_t v = 0; v < V; ++v) { e[v] = exp(((double)x[v] - m) / (double)temperature); z += e[v]; }
    for (int32_t v = 0; v < V; ++v) probs[r * V + v] = (float)(e[v] / z);
    free(e);
  }
}

/* --------------------------------------------------------------- LM head */

/*
 * The output projection that produces the rows acceptance reads (the verifying stage owns an
 * LM head, Implementation): for bf16 hidden states h [rows][d] and LM-head weights W [V][d],
 *   logits[r][v] = sum_j h[r][j] * W[v][j]                       (fp64, exact products)
 * and each row's softmax statistics at temperature T (the same convention as oracle_softmax):
 *   mx[r] = max_v logits[r][v] / T,   z[r] = sum_v exp(logits[r][v] / T - mx[r]).
 * `logits` (fp64 [rows][V]) may be NULL; mx and z are fp64 [rows].
 */
void oracle_lm_head(const uint16_t* h, const uint16_t* W, int64_t rows, int32_t V, int32_t d, float temperature,
                    double* logits, double* mx, double* z) {
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < rows; ++r) {
    double* hr = (double*)malloc(sizeof(double) * (size_t)d);
    double* lr = (double*)malloc(sizeof(double) * (size_t)V);
    for (int32_t j = 0; j < d; ++j) hr[j] = bf16_to_double(h[r * d + j]);
    for (int32_t v = 0; v < V; ++v) {
      double acc = 0.0;
      const uint16_t* wv = W + (int64_t)v * d;
      for (int32_t j = 0; j < d; ++j) acc += hr[j] * bf16_to_double(wv[j]);
      lr[v] = acc;
    }
    double m = -INFINITY;
    for (int32_t v = 0; v < V; ++v) if (lr[v] / (double)temperature > m) m = lr[v] / (double)temperature;
    double zz = 0.0;
    for (int32_t v = 0; v < V; ++v) zz += exp(lr[v] / (double)temperature - m);
    mx[r] = m;
    z[r] = zz;
    if (logits) memcpy(logits + r * V, lr, sizeof(double) * (size_t)V);
    free(hr);
    free(lr);
  }
}

/* ------------------------------------------------------------ linear layer */

/*
 * A linear layer of the drafting adapter (Implementation: a linear layer and an attention
 * layer, then the LM head): for bf16 inputs x [rows][in] and weights W [out][in], and an
 * optional bf16 residual R [rows][out],
 *   y[r][o] = sum_j x[r][j] * W[o][j]  (+ R[r][o])             (fp64, exact products)
 * y is fp64 [rows][out]; residual may be NULL.
 */
void oracle_linear(const uint16_t* x, const uint16_t* W, const uint16_t* residual, int64_t rows, int32_t out,
                   int32_t in, double* y) {
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < rows; ++r) {
    double* xr = (double*)malloc(sizeof(double) * (size_t)in);
    for (int32_t j = 0; j < in; ++j) xr[j] = bf16_to_double(x[r * in + j]);
    for (int32_t o = 0; o < out; ++o) {
      double acc = 0.0;
      const uint16_t* wo = W + (int64_t)o * in;
      for (int32_t j = 0; j < in; ++j) acc += xr[j] * bf16_to_double(wo[j]);
      if (residual) acc += bf16_to_double(residual[r * out + o]);
      y[r * out + o] = acc;
    }
    free(xr);
  }
}

/* ------------------------------------------------------ selective speculation */

/*
 * Acceptance-guided selective speculation (Sec. 5, "Acceptance-Guided Selective Speculation"):
 * the draft tokens of a batch are ranked by confidence and a fixed fraction alpha of them, the
 * lowest ranked, is dropped; speculation continues on the rest.
 *   - sequence b has k_b = qsl[b+1]-qsl[b]-1 drafts, draft i at index qsl[b]-b+i, with
 *     confidence conf[...] (the draft model's probability of the token it drafted; NaN or
 *     values outside [0, 1] are clamped into [0, 1], NaN to 0);
 *   - a draft's score is the confidence of its whole prefix, the fp32 product
 *     s_i = s_{i-1} * conf_i taken in order (s_{-1} = 1): a later draft is verified only if
 *     every earlier one is kept, so the product is what survives;
 *   - the N = sum k_b drafts are ordered by score, higher first, equal scores by lower index
 *     first; the last m = floor(alpha * N) of that order are dropped (alpha in [0, 1));
 *   - each sequence keeps the drafts before its first dropped one: kept_k[b], keep[i] = 1 for
 *     the kept drafts, and kept_qsl is the query_start_loc of the reduced batch.
 * Returns 0, or -1 on bad sizes.
 */
typedef struct {
  float score;
  int32_t idx;
} oracle_ranked;

static int ranked_order(const void* pa, const void* pb) {
  const oracle_ranked* a = (const oracle_ranked*)pa;
  const oracle_ranked* b = (const oracle_ranked*)pb;
  if (a->score != b->score) return a->score > b->score ? -1 : 1;
  return a->idx < b->idx ? -1 : (a->idx > b->idx ? 1 : 0);
}

int oracle_select_drafts(int32_t B, const int32_t* qsl, const float* conf, float alpha, int32_t* kept_k,
                         int32_t* kept_qsl, int32_t* keep) {
  if (B < 0 || !(alpha >= 0.0f) || !(alpha < 1.0f)) return -1;
  const int32_t N = qsl[B] - B;
  if (N < 0) return -1;
  oracle_ranked* r = (oracle_ranked*)malloc(sizeof(oracle_ranked) * (size_t)(N > 0 ? N : 1));
  for (int32_t b = 0; b < B; ++b) {
    const int32_t k = qsl[b + 1] - qsl[b] - 1, d0 = qsl[b] - b;
    float s = 1.0f;
    for (int32_t i = 0; i < k; ++i) {
      float c = conf[d0 + i];
      c = isnan(c) ? 0.0f : (c < 0.0f ? 0.0f : (c > 1.0f ? 1.0f : c));
      s = s * c; /* fp32 product, round to nearest */
      r[d0 + i].score = s;
      r[d0 + i].idx = d0 + i;
    }
  }
  qsort(r, (size_t)N, sizeof(oracle_ranked), ranked_order);
  const int64_t m = (int64_t)floor((double)alpha * (double)N);
  for (int32_t i = 0; i < N; ++i) keep[i] = 0;
  for (int64_t j = 0; j < N - m; ++j) keep[r[j].idx] = 1;
  kept_qsl[0] = 0;
  for (int32_t b = 0; b < B; ++b) {
    const int32_t k = qsl[b + 1] - qsl[b] - 1, d0 = qsl[b] - b;
    int32_t kk = 0;
    while (kk < k && keep[d0 + kk]) ++kk;
    for (int32_t i = kk; i < k; ++i) keep[d0 + i] = 0;
    kept_k[b] = kk;
    kept_qsl[b + 1] = kept_qsl[b] + kk + 1;
  }
  free(r);
  return 0;
}

/* ---------------------------------------------------------------- accept */

/* row_status codes */
#define ORACLE_OK 0
#define ORACLE_EMPTY_ROW 1   /* sampled row had no positive weight, even after the fallback */
#define ORACLE_BAD_ROW 2     /* sampled row held a NaN, an infinity or a negative value */
#define ORACLE_BAD_TOKEN 3   /* a draft token id outside [0, V) */

static int bad_value(float x) { return isnan(x) || isinf(x) || x < 0.0f; }

/*
 * Exact threshold t = floor(u * S) for an fp32 uniform u and an integer S < 2^63.
 * u = f * 2^e with f in [0.5, 1) (frexp); f * 2^24 is an integer m < 2^24, so
 * u * S = m * S / 2^(24 - e) and the floor is a right shift of the 128-bit product.
 * u <= 0 or NaN gives 0; u >= 1 gives S - 1; the result is clamped to S - 1.
 */
static uint64_t exact_threshold(float u, uint64_t S) {
  if (!(u > 0.0f)) return 0;
  if (u >= 1.0f) return S - 1;
  int e;
  float f = frexpf(u, &e);
  uint64_t m = (uint64_t)ldexpf(f, 24);
  int shift = 24 - e; /* >= 25 */
  unsigned __int128 prod = (unsigned __int128)m * (unsigned __int128)S;
  uint64_t t = shift >= 128 ? 0 : (uint64_t)(prod >> shift);
  return t < S ? t : S - 1;
}

/*
 * Inverse-CDF sample in fixed point.  The scale is that of the target row p: M = max p, and
 * e such that M in [2^e, 2^(e+1)); s = 40 - e.  For the weight row w (w <= p entrywise):
 *   W_v = floor(w_v * 2^s)  (exact: a power-of-two scaling of an fp32 value, then floor);
 *   S = sum W_v; if S == 0 and a fallback row is given, the weights become the fallback's;
 *   t = floor(u * S) exactly;
 *   token = the smallest m with W_0 + ... + W_m > t.
 * Returns -1 if M == 0 (then every weight is 0).
 */
static uint64_t fixed_sum(const float* w, int32_t V, int s) {
  uint64_t S = 0;
  for (int32_t v = 0; v < V; ++v) S += (uint64_t)floor(ldexp((double)w[v], s));
  return S;
}

static int32_t sample_fixed_point(const float* w, const float* fallback, int32_t V, float M, float u) {
  if (M == 0.0f) return -1;
  int E;
  frexp((double)M, &E); /* M = f * 2^E, f in [0.5,1)  =>  M in [2^(E-1), 2^E) */
  int s = 40 - (E - 1);
  uint64_t S = fixed_sum(w, V, s);
  if (S == 0 && fallback) {
    w = fallback;
    S = fixed_sum(w, V, s);
  }
  uint64_t t = exact_threshold(u, S);
  uint64_t prefix = 0;
  for (int32_t v = 0; v < V; ++v) {
    prefix += (uint64_t)floor(ldexp((double)w[v], s));
    if (prefix > t) return v;
  }
  return V - 1; /* unreachable: prefix reaches S > t (S >= 2^40 once the weights are p's) */
}

/*
 * Speculative-sampling acceptance on fp32 probability rows.
 *   Sequence b has k_b = qsl[b+1]-qsl[b]-1 drafts x_i = draft_ids[qsl[b]-b+i].
 *   Target row i of b is target[(qsl[b]+i)*V ...] (i = 0..k_b); draft row i is
 *   draft[(qsl[b]-b+i)*V ...] (i = 0..k_b-1).
 * Steps, for each b:
 *   1. any x_i outside [0, V): status 3, a_b = 0, every token -1.
 *   2. for i = 0..k_b-1: accept iff (double)u_i * (double)q_i(x_i) < (double)p_i(x_i)
 *      (exact: a product of two fp32 values is exact in fp64, so this is u < p/q, i.e. the
 *      test u < min(1, p/q) for u in [0,1)); a_b = the number of leading accepts.
 *   3. a_b < k_b: weights w_v = max(0, fp32(p_a(v) - q_a(v))), with p_a as the fallback when
 *      every fixed-point weight is 0.  a_b = k_b: w = p_k (bonus token).
 *      The row(s) read here must be finite and non-negative, else status 2.
 *   4. token = sample_fixed_point(w, fallback, max p_a, u_sample[b]) (the scale of the target
 *      row); if p_a has no positive entry, status 1.
 *   Outputs: accepted_len[b] = a_b; out_tokens[b][0..a_b) = x_0..x_{a_b-1};
 *   out_tokens[b][a_b] = token (-1 on status 1/2); later positions -1.
 *   If seq_lens_inout is not NULL, seq_lens_inout[b] = S_b - k_b + a_b (the rows of
 *   rejected drafts become stale) unless status is 3.
 */
void oracle_accept(int32_t B, int32_t V, int32_t max_k, const int32_t* qsl, const float* target,
                   const float* draft, const int32_t* draft_ids, const float* u_accept,
                   const float* u_sample, int32_t* accepted_len, int32_t* out_tokens,
                   int32_t* row_status, int32_t* seq_lens_inout) {
#pragma omp parallel for schedule(dynamic, 16)
  for (int32_t b = 0; b < B; ++b) {
    int32_t k = qsl[b + 1] - qsl[b] - 1;
    int64_t t0 = qsl[b];       /* first target row of b */
    int64_t d0 = qsl[b] - b;   /* first draft row of b */
    int32_t* tok = out_tokens + (int64_t)b * (max_k + 1);
    for (int32_t i = 0; i <= max_k; ++i) tok[i] = -1;
    accepted_len[b] = 0;
    row_status[b] = ORACLE_OK;

    int ids_ok = 1;
    for (int32_t i = 0; i < k; ++i)
      if (draft_ids[d0 + i] < 0 || draft_ids[d0 + i] >= V) ids_ok = 0;
    if (!ids_ok) { row_status[b] = ORACLE_BAD_TOKEN; continue; }

    int32_t a = 0;
    while (a < k) {
      int32_t x = draft_ids[d0 + a];
      double p = (double)target[(t0 + a) * V + x];
      double q = (double)draft[(d0 + a) * V + x];
      double u = (double)u_accept[d0 + a];
      if (u * q < p) ++a; else break;
    }
    accepted_len[b] = a;
    for (int32_t i = 0; i < a; ++i) tok[i] = draft_ids[d0 + i];
    if (seq_lens_inout) seq_lens_inout[b] = seq_lens_inout[b] - k + a;

    const float* P = target + (t0 + a) * V;
    const float* Q = a < k ? draft + (d0 + a) * V : NULL;
    int bad = 0;
    for (int32_t v = 0; v < V; ++v) {
      if (bad_value(P[v])) bad = 1;
      if (Q && bad_value(Q[v])) bad = 1;
    }
    if (bad) { row_status[b] = ORACLE_BAD_ROW; continue; }

    float* w = (float*)malloc(sizeof(float) * (size_t)V);
    float M = 0.0f;
    for (int32_t v = 0; v < V; ++v) {
      if (P[v] > M) M = P[v];
      if (Q) {
        float diff = P[v] - Q[v]; /* one IEEE fp32 subtraction, round to nearest */
        w[v] = diff > 0.0f ? diff : 0.0f;
      } else {
        w[v] = P[v];
      }
    }
    int32_t token = sample_fixed_point(w, Q ? P : NULL, V, M, u_sample[b]);
    free(w);
    if (token < 0) row_status[b] = ORACLE_EMPTY_ROW;
    tok[a] = token;
  }
}

/*
 * Look-ahead memory estimate (Sec. 5, Remaining-Length-Aware Scheduling; Algorithm 1): the
 * expected KV-cache tokens held by the running requests over the next `iters` decoding
 * iterations of a pipeline of depth pp whose speculation is accepted with probability theta.
 *
 * Derived here from the process the estimate models, not from the printed listing.  Each
 * request runs a string of speculation outcomes: an accepted token advances it by one
 * iteration, a rejection stalls it for pp iterations, and either way one token is generated.
 * Let mass(c, w) be the probability weight of reaching exactly c iterations with w rejections.
 * Its last outcome was an acceptance (from c-1, w) or a rejection (from c-pp, w-1):
 *   mass(0, 0) = 1,  mass(c, w) = theta * mass(c-1, w) + (1 - theta) * mass(c-pp, w-1),
 * i.e. the sum over every ordering of t = c - pp*w acceptances and w rejections of
 * theta^t (1 - theta)^w (the paper's p(i, w); it does not sum to 1 over w when pp > 1, since
 * a rejection can step over iteration i).  At iteration i such a string has generated
 * k = t + w tokens.  The estimate then weighs the running requests by these masses:
 *   E_gen(i)  = sum_w k mass(i, w)                      tokens a request is expected to add
 *   Pfin_r(i) = prec[r] * (mass of the strings with k >= remaining[r])
 *   mem(i)    = sum_r cur_len[r] + (n - sum_r Pfin_r) E_gen - sum_r cur_len[r] Pfin_r:
 *     the current lengths, plus the expected growth of the requests still running, minus the
 *     lengths that finished requests release.
 * prec[r] is the precision of the prediction of request r's remaining length (the paper's
 * E(tau)).  All arithmetic in fp64.  e_gen, e_nfin and e_lfin may be NULL; otherwise they
 * receive E_gen, sum_r Pfin_r and sum_r cur_len[r] Pfin_r per iteration.  Returns 0, or -1 on
 * bad arguments or a failed allocation.
 */
int oracle_lookahead(int32_t n, const int64_t* cur_len, const int32_t* remaining, const double* prec,
                     int32_t pp, double theta, int32_t iters, double* mem, double* e_gen, double* e_nfin,
                     double* e_lfin) {
  if (n < 0 || pp < 1 || iters < 1 || !(theta >= 0.0 && theta <= 1.0) || !mem) return -1;
  if (n > 0 && (!cur_len || !remaining || !prec)) return -1;
  const int64_t W = iters / pp + 1;            /* rejections possible within the horizon */
  double* m = calloc((size_t)(iters + 1) * (size_t)W, sizeof *m);   /* m[c*W + w] = mass(c, w) */
  if (!m) return -1;
  m[0] = 1.0;
  for (int32_t c = 1; c <= iters; ++c)
    for (int64_t w = 0; w < W; ++w) {
      double v = theta * m[(int64_t)(c - 1) * W + w];
      if (w > 0 && c >= pp) v += (1.0 - theta) * m[(int64_t)(c - pp) * W + (w - 1)];
      m[(int64_t)c * W + w] = v;
    }
  double held = 0.0;                           /* tokens the requests hold now */
  for (int32_t r = 0; r < n; ++r) held += (double)cur_len[r];
  for (int32_t i = 1; i <= iters; ++i) {
    const double* row = m + (int64_t)i * W;
    double grow = 0.0;
    for (int64_t w = 0; w * pp <= i; ++w) grow += (double)(i - pp * w + w) * row[w];
    double fin = 0.0, released = 0.0;
    for (int32_t r = 0; r < n; ++r) {
      double tail = 0.0;                       /* mass of the strings that generated >= remaining[r] */
      for (int64_t w = 0; w * pp <= i; ++w)
        if (i - pp * w + w >= (int64_t)remaining[r]) tail += row[w];
      const double pfin = prec[r] * tail;
      fin += pfin;
      released += (double)cur_len[r] * pfin;
    }
    mem[i - 1] = held + ((double)n - fin) * grow - released;
    if (e_gen) e_gen[i - 1] = grow;
    if (e_nfin) e_nfin[i - 1] = fin;
    if (e_lfin) e_lfin[i - 1] = released;
  }
  free(m);
  return 0;
}

/* Threads of the parallel loops above from now on (n >= 1; no effect without OpenMP). */
void oracle_set_num_threads(int n) {
#ifdef _OPENMP
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* Number of OpenMP threads the parallel loops above use (for reporting). */
int oracle_num_threads(void) {
  int n = 1;
#ifdef _OPENMP
#pragma omp parallel
  {
#pragma omp single
    n = omp_get_num_threads();
  }
#endif
  return n;
}
