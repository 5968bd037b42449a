/*
 * oracle.c -- plain double-precision CPU reference of the span-merging
 * (UMIM) inference hot path.  TEST INFRASTRUCTURE ONLY: it is loaded by the
 * tests, the smoke check and the benchmark's CPU-baseline leg, never by the
 * product path, and it shares no code with the GPU library.
 *
 * Each function follows the passage of the paper it cites, with no blocking,
 * fusion or reordering beyond what that passage states.  Paper: "Distilling
 * Sequential Computation in Transformer Language Models" (arXiv 2609.27233).
 *
 * Readings where the paper is silent (each is listed with its reason in the
 * design notes of the repository):
 *   - M_phi takes the appendix form (Linear -> GELU -> LayerNorm on both
 *     sides); the main text's Eq. 1 is the special case selected by flag 1.
 *   - GELU is the exact erf form; LayerNorm uses the biased variance and an
 *     affine gain/bias over all d features; Linear is y = W x + b, W [out][in].
 *   - Heads are contiguous blocks of d_h = d / h features, concatenated in
 *     head order; the pooling scale is 1 / sqrt(d_h) of M_phi.
 *   - A merged span keeps its last position; compressed positions are
 *     contiguous.
 *   - The paged cache frees blocks onto a LIFO stack: rollback pushes in
 *     reverse request order, highest logical block first; append pops in
 *     request order, lowest logical block first.
 *   - Decode attention: scale given by the caller (1/sqrt(head_dim) in the
 *     workloads), grouped-query head g = h / (Hq / Hkv), no soft-cap, no
 *     window; the query attends over every cached entry (it has been
 *     appended first).
 *   - Prefill attention: the same scores, causal over cache positions; a
 *     request's query rows are its last m cached positions (the prompt's
 *     K/V are appended before the pass).
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int orc_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Threads for the following parallel loops (timing only; results do not
   depend on it: every loop writes disjoint outputs). */
void orc_set_num_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* ------------------------------------------------------------------------ */
/* element access of raw pool storage                                       */

static double load_elem(const void *base, int64_t idx, int is_bf16) {
  if (is_bf16) {
    uint16_t h = ((const uint16_t *)base)[idx];
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
  }
  return (double)((const float *)base)[idx];
}

static void copy_elem(void *dst, int64_t di, const void *src, int64_t si,
                      int elem_bytes) {
  memcpy((char *)dst + di * elem_bytes, (const char *)src + si * elem_bytes,
         (size_t)elem_bytes);
}

/* ------------------------------------------------------------------------ */
/* Merge module M_phi                                                       */
/* Appendix "Module Architecture and Integration", subsection               */
/* "Attention-based Pooling Architecture":                                  */
/*   P   = LN_kv(GELU(Linear_kv(E_s)))                                       */
/*   a_i = softmax(P_i q_i / sqrt(d_h)),  o_i = a_i^T P_i                     */
/*   z_s = LN_o(GELU(Linear_o([o_1; ...; o_h])))                              */
/* The main text's Eq. 1 is the same pooling without GELU, LN and biases.   */

static double gelu_erf(double x) { return 0.5 * x * (1.0 + erf(x / sqrt(2.0))); }

/* y = W x + b, W row-major [d_out][d_in] */
static void linear(const double *W, const double *b, const double *x, int d_in,
                   int d_out, double *y) {
  for (int o = 0; o < d_out; ++o) {
    double s = b ? b[o] : 0.0;
    const double *w = W + (int64_t)o * d_in;
    for (int i = 0; i < d_in; ++i) s += w[i] * x[i];
    y[o] = s;
  }
}

/* LayerNorm over all d features: biased variance, affine gain and bias. */
static void layer_norm(double *v, int d, const double *g, const double *b,
                       double eps) {
  double mean = 0.0;
  for (int i = 0; i < d; ++i) mean += v[i];
  mean /= d;
  double var = 0.0;
  for (int i = 0; i < d; ++i) var += (v[i] - mean) * (v[i] - mean);
  var /= d;
  double inv = 1.0 / sqrt(var + eps);
  for (int i = 0; i < d; ++i) v[i] = g[i] * (v[i] - mean) * inv + b[i];
}

int orc_merge_spans(int d, int h, double ln_eps, const double *emb,
                    int64_t emb_rows, const int32_t *row_idx,
                    const int32_t *span_offsets, int num_spans,
                    const double *Q, const double *W_kv, const double *b_kv,
                    const double *g_kv, const double *beta_kv,
                    const double *W_o, const double *b_o, const double *g_o,
                    const double *beta_o, int flags, double *out,
                    double *pool_weights, int pool_weights_stride) {
  if (d <= 0 || h <= 0 || d % h != 0 || num_spans < 0) return ORC_EINVAL;
  if (num_spans > 0 && span_offsets[0] != 0) return ORC_EINVAL;
  for (int s = 0; s < num_spans; ++s)
    if (span_offsets[s + 1] - span_offsets[s] < 1) return ORC_EINVAL;
  int64_t total = num_spans > 0 ? span_offsets[num_spans] : 0;
  for (int64_t r = 0; r < total; ++r)
    if (row_idx[r] < 0 || row_idx[r] >= emb_rows) return ORC_EINVAL;

  const int bare = flags & 1;
  const int dh = d / h;
  const double inv_sqrt_dh = 1.0 / sqrt((double)dh);

#pragma omp parallel for schedule(dynamic, 1)
  for (int s = 0; s < num_spans; ++s) {
    const int n = span_offsets[s + 1] - span_offsets[s];
    double *P = (double *)malloc(sizeof(double) * (size_t)n * d);
    double *scores = (double *)malloc(sizeof(double) * (size_t)n);
    double *c = (double *)malloc(sizeof(double) * (size_t)d);
    double *y = (double *)malloc(sizeof(double) * (size_t)d);

    /* token processor: P_j = LN_kv(GELU(W_kv e_j + b_kv)) */
    for (int j = 0; j < n; ++j) {
      const double *e = emb + (int64_t)row_idx[span_offsets[s] + j] * d;
      double *Pj = P + (int64_t)j * d;
      linear(W_kv, bare ? NULL : b_kv, e, d, d, Pj);
      if (!bare) {
        for (int i = 0; i < d; ++i) Pj[i] = gelu_erf(Pj[i]);
        layer_norm(Pj, d, g_kv, beta_kv, ln_eps);
      }
    }

    /* per-head learned-query pooling; P_i is both key and value */
    for (int i = 0; i < h; ++i) {
      const double *qi = Q + (int64_t)i * dh;
      double m = -INFINITY;
      for (int j = 0; j < n; ++j) {
        const double *Pij = P + (int64_t)j * d + (int64_t)i * dh;
        double sc = 0.0;
        for (int t = 0; t < dh; ++t) sc += Pij[t] * qi[t];
        scores[j] = sc * inv_sqrt_dh;
        if (scores[j] > m) m = scores[j];
      }
      double Z = 0.0;
      for (int j = 0; j < n; ++j) {
        scores[j] = exp(scores[j] - m);
        Z += scores[j];
      }
      for (int j = 0; j < n; ++j) scores[j] /= Z; /* alpha_i[j] */
      if (pool_weights)
        for (int j = 0; j < n; ++j)
          pool_weights[((int64_t)s * h + i) * pool_weights_stride + j] =
              scores[j];
      for (int t = 0; t < dh; ++t) {
        double acc = 0.0;
        for (int j = 0; j < n; ++j)
          acc += scores[j] * P[(int64_t)j * d + (int64_t)i * dh + t];
        c[(int64_t)i * dh + t] = acc; /* concat in head order */
      }
    }

    /* output processor: z = LN_o(GELU(W_o c + b_o)) */
    linear(W_o, bare ? NULL : b_o, c, d, d, y);
    if (!bare) {
      for (int i = 0; i < d; ++i) y[i] = gelu_erf(y[i]);
      layer_norm(y, d, g_o, beta_o, ln_eps);
    }
    memcpy(out + (int64_t)s * d, y, sizeof(double) * (size_t)d);

    free(P);
    free(scores);
    free(c);
    free(y);
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Prompt packing                                                           */
/* "Prompt-time Integration" (contiguous compressed positions), "Prompt     */
/* Merging" (L~_p = L_p - sum (j - i - 1)), "Mask Construction and Sequence */
/* Alignment" (the surrogate is aligned with the final position of its      */
/* span), "Positional Encoding under Token-Span Merging" (pi(t) = t - r(t)).*/

int orc_pack_spans(int B, const int32_t *seq_offsets, int num_spans,
                   const int32_t *span_start, const int32_t *span_len,
                   const int32_t *seq_span_offsets, int32_t *pi,
                   int32_t *packed_offsets, int32_t *packed_src,
                   const int32_t *token_ids, const void *emb,
                   int64_t emb_rows, const void *surrogates, int d,
                   int elem_bytes, void *packed) {
  if (B < 0 || num_spans < 0) return ORC_EINVAL;
  if (seq_offsets[0] != 0 || seq_span_offsets[0] != 0 ||
      seq_span_offsets[B] != num_spans)
    return ORC_EINVAL;
  for (int b = 0; b < B; ++b) {
    if (seq_offsets[b + 1] < seq_offsets[b]) return ORC_EINVAL;
    if (seq_span_offsets[b + 1] < seq_span_offsets[b]) return ORC_EINVAL;
    for (int s = seq_span_offsets[b]; s < seq_span_offsets[b + 1]; ++s) {
      if (span_len[s] < 1) return ORC_EINVAL;
      if (span_start[s] < seq_offsets[b]) return ORC_EINVAL;
      if ((int64_t)span_start[s] + span_len[s] > seq_offsets[b + 1])
        return ORC_EINVAL;
      if (s > seq_span_offsets[b] &&
          span_start[s] < span_start[s - 1] + span_len[s - 1])
        return ORC_EINVAL;
    }
  }
  const int total = seq_offsets[B];

  /* which span (if any) covers each token */
  int32_t *span_of = (int32_t *)malloc(sizeof(int32_t) * (size_t)(total + 1));
  for (int t = 0; t < total; ++t) span_of[t] = -1;
  for (int s = 0; s < num_spans; ++s)
    for (int t = span_start[s]; t < span_start[s] + span_len[s]; ++t)
      span_of[t] = s;

  if (packed)
    for (int t = 0; t < total; ++t)
      if (span_of[t] < 0 && (token_ids[t] < 0 || token_ids[t] >= emb_rows)) {
        free(span_of);
        return ORC_EINVAL;
      }

  int32_t running = 0;
  for (int b = 0; b < B; ++b) {
    packed_offsets[b] = running;
    int32_t pos = 0; /* exclusive scan of the keep mask */
    for (int t = seq_offsets[b]; t < seq_offsets[b + 1]; ++t) {
      const int s = span_of[t];
      const int is_last = s >= 0 && t == span_start[s] + span_len[s] - 1;
      const int keep = (s < 0) || is_last;
      pi[t] = pos;
      if (keep) {
        packed_src[running + pos] = (s < 0) ? t : -1 - s;
        ++pos;
      }
    }
    running += pos;
  }
  packed_offsets[B] = running;

  if (packed) {
    for (int32_t r = 0; r < running; ++r) {
      const int32_t src = packed_src[r];
      for (int i = 0; i < d; ++i) {
        if (src >= 0)
          copy_elem(packed, (int64_t)r * d + i, emb,
                    (int64_t)token_ids[src] * d + i, elem_bytes);
        else
          copy_elem(packed, (int64_t)r * d + i, surrogates,
                    (int64_t)(-1 - src) * d + i, elem_bytes);
      }
    }
  }
  free(span_of);
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Paged KV cache: rollback and append                                      */
/* "Decoding-time Integration" and "Decoding-Time Merging and KV-Cache      */
/* Update": crop the n-1 cached entries of the matched span, forward the    */
/* surrogate to produce one new K/V state; L_C' = L_C - (n-1) + 1.          */

static int64_t k_index(const orc_cache *c, int blk, int g, int slot, int t) {
  return (((int64_t)blk * c->num_kv_heads + g) * c->block_size + slot) *
             c->head_dim + t;
}

static int64_t v_index(const orc_cache *c, int blk, int g, int slot, int t) {
  return (((int64_t)blk * c->num_kv_heads + g) * c->head_dim + t) *
             c->block_size + slot;
}

static int blocks_for(int64_t len, int bs) { return (int)((len + bs - 1) / bs); }

static int ids_valid(const orc_cache *c, const int32_t *seq_ids, int n) {
  for (int i = 0; i < n; ++i) {
    if (seq_ids[i] < 0 || seq_ids[i] >= c->max_seqs) return 0;
    for (int j = 0; j < i; ++j)
      if (seq_ids[j] == seq_ids[i]) return 0;
  }
  return 1;
}

int orc_kv_rollback(orc_cache *c, const int32_t *seq_ids, const int32_t *k,
                    int n) {
  const int bs = c->block_size;
  const int64_t cap = (int64_t)c->max_blocks_per_seq * bs;
  if (n < 0 || !ids_valid(c, seq_ids, n)) return ORC_EINVAL;
  for (int i = 0; i < n; ++i)
    if (k[i] < 0) return ORC_EINVAL;
  int64_t freed = 0;
  for (int i = 0; i < n; ++i) {
    const int32_t L = c->lengths[seq_ids[i]];
    if (L < 0 || L > cap || k[i] > L) return ORC_ERANGE;
    freed += blocks_for(L, bs) - blocks_for(L - k[i], bs);
  }
  if (*c->free_top < 0 || *c->free_top + freed > c->num_blocks)
    return ORC_ERANGE;

  for (int i = n - 1; i >= 0; --i) { /* reverse request order */
    const int s = seq_ids[i];
    int32_t *row = c->block_table + (int64_t)s * c->max_blocks_per_seq;
    const int32_t L = c->lengths[s];
    const int nb_old = blocks_for(L, bs);
    const int nb_new = blocks_for(L - k[i], bs);
    for (int j = nb_old - 1; j >= nb_new; --j) { /* highest block first */
      c->free_stack[(*c->free_top)++] = row[j];
      row[j] = -1;
    }
    c->lengths[s] = L - k[i];
  }
  return ORC_OK;
}

int orc_kv_append(orc_cache *c, const int32_t *seq_ids,
                  const int32_t *row_offsets, int n, const void *K,
                  const void *V) {
  const int bs = c->block_size, H = c->num_kv_heads, D = c->head_dim;
  const int eb = c->is_bf16 ? 2 : 4;
  const int64_t cap = (int64_t)c->max_blocks_per_seq * bs;
  if (n < 0 || !ids_valid(c, seq_ids, n)) return ORC_EINVAL;
  if (n > 0 && row_offsets[0] != 0) return ORC_EINVAL;
  for (int i = 0; i < n; ++i)
    if (row_offsets[i + 1] < row_offsets[i]) return ORC_EINVAL;
  int64_t need = 0;
  for (int i = 0; i < n; ++i) {
    const int32_t L = c->lengths[seq_ids[i]];
    const int32_t m = row_offsets[i + 1] - row_offsets[i];
    if (L < 0 || (int64_t)L + m > cap) return ORC_ERANGE;
    need += blocks_for((int64_t)L + m, bs) - blocks_for(L, bs);
  }
  if (need > *c->free_top) return ORC_ENOMEM;
  for (int64_t j = 0; j < need; ++j) {
    const int32_t blk = c->free_stack[*c->free_top - 1 - j];
    if (blk < 0 || blk >= c->num_blocks) return ORC_EINVAL;
  }

  for (int i = 0; i < n; ++i) { /* request order */
    const int s = seq_ids[i];
    int32_t *row = c->block_table + (int64_t)s * c->max_blocks_per_seq;
    for (int32_t r = row_offsets[i]; r < row_offsets[i + 1]; ++r) {
      const int32_t pos = c->lengths[s];
      if (pos % bs == 0) row[pos / bs] = c->free_stack[--(*c->free_top)];
      const int blk = row[pos / bs], slot = pos % bs;
      for (int g = 0; g < H; ++g)
        for (int t = 0; t < D; ++t) {
          const int64_t src = ((int64_t)r * H + g) * D + t;
          copy_elem(c->k_pool, k_index(c, blk, g, slot, t), K, src, eb);
          copy_elem(c->v_pool, v_index(c, blk, g, slot, t), V, src, eb);
        }
      c->lengths[s] = pos + 1;
    }
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Decode attention over the cache ("Efficiency Analysis": each decode step */
/* attends to the accumulated KV cache; the backbone itself is unchanged).  */
/* out = sum_j softmax_j(scale * q . K_j) V_j over all cached entries.      */

int orc_decode_attention(const orc_cache *c, const int32_t *seq_ids, int n,
                         const double *q, int num_q_heads, double scale,
                         double *out, double *probs, int probs_stride) {
  const int H = c->num_kv_heads, D = c->head_dim, bs = c->block_size;
  if (n < 0 || num_q_heads <= 0 || num_q_heads % H != 0) return ORC_EINVAL;
  const int G = num_q_heads / H;
  int status = ORC_OK;

#pragma omp parallel for collapse(2) schedule(dynamic, 1)
  for (int i = 0; i < n; ++i) {
    for (int hq = 0; hq < num_q_heads; ++hq) {
      double *o = out + ((int64_t)i * num_q_heads + hq) * D;
      for (int t = 0; t < D; ++t) o[t] = 0.0;
      const int s = seq_ids[i];
      int bad = s < 0 || s >= c->max_seqs;
      const int32_t L = bad ? 0 : c->lengths[s];
      if (!bad && (L < 0 || L > (int64_t)c->max_blocks_per_seq * bs)) bad = 1;
      const int32_t *row =
          bad ? NULL : c->block_table + (int64_t)s * c->max_blocks_per_seq;
      for (int j = 0; !bad && j < L; j += bs)
        if (row[j / bs] < 0 || row[j / bs] >= c->num_blocks) bad = 1;
      if (bad) {
#pragma omp atomic write
        status = ORC_EINVAL;
        continue;
      }
      if (L == 0) continue;
      const int g = hq / G;
      const double *qv = q + ((int64_t)i * num_q_heads + hq) * D;
      double *sc = (double *)malloc(sizeof(double) * (size_t)L);
      double m = -INFINITY;
      for (int j = 0; j < L; ++j) {
        const int blk = row[j / bs], slot = j % bs;
        double dot = 0.0;
        for (int t = 0; t < D; ++t)
          dot += qv[t] * load_elem(c->k_pool, k_index(c, blk, g, slot, t),
                                   c->is_bf16);
        sc[j] = dot * scale;
        if (sc[j] > m) m = sc[j];
      }
      double Z = 0.0;
      for (int j = 0; j < L; ++j) {
        sc[j] = exp(sc[j] - m);
        Z += sc[j];
      }
      for (int j = 0; j < L; ++j) {
        sc[j] /= Z;
        if (probs) probs[((int64_t)i * num_q_heads + hq) * probs_stride + j] = sc[j];
      }
      for (int j = 0; j < L; ++j) {
        const int blk = row[j / bs], slot = j % bs;
        for (int t = 0; t < D; ++t)
          o[t] += sc[j] * load_elem(c->v_pool, v_index(c, blk, g, slot, t),
                                    c->is_bf16);
      }
      free(sc);
    }
  }
  return status;
}

/* ------------------------------------------------------------------------ */
/* Prefill attention over the cache ("Efficiency Analysis": prompt merging  */
/* shortens the sequence before the backbone runs, so every layer's         */
/* attention runs over the compressed positions).  Causal: the query at     */
/* cache position p sees entries 0..p.                                      */

int orc_prefill_attention(const orc_cache *c, const int32_t *seq_ids, int n,
                          const int32_t *q_offsets, const double *q,
                          int num_q_heads, double scale, double *out) {
  const int H = c->num_kv_heads, D = c->head_dim, bs = c->block_size;
  if (n < 0 || num_q_heads <= 0 || num_q_heads % H != 0) return ORC_EINVAL;
  if (n > 0 && q_offsets[0] != 0) return ORC_EINVAL;
  for (int i = 0; i < n; ++i) {
    const int s = seq_ids[i];
    if (s < 0 || s >= c->max_seqs) return ORC_EINVAL;
    const int32_t L = c->lengths[s];
    const int32_t m = q_offsets[i + 1] - q_offsets[i];
    if (L < 0 || L > (int64_t)c->max_blocks_per_seq * bs || m < 0 || m > L) return ORC_EINVAL;
    const int32_t *row = c->block_table + (int64_t)s * c->max_blocks_per_seq;
    for (int j = 0; j < L; j += bs)
      if (row[j / bs] < 0 || row[j / bs] >= c->num_blocks) return ORC_EINVAL;
  }
  const int G = num_q_heads / H;
  const int64_t rows = n > 0 ? q_offsets[n] : 0;
  for (int64_t e = 0; e < rows * num_q_heads * D; ++e) out[e] = 0.0;

  for (int i = 0; i < n; ++i) {
    const int s = seq_ids[i];
    const int32_t L = c->lengths[s];
    const int32_t m = q_offsets[i + 1] - q_offsets[i];
    const int32_t *row = c->block_table + (int64_t)s * c->max_blocks_per_seq;
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int r = 0; r < m; ++r) {
      for (int hq = 0; hq < num_q_heads; ++hq) {
        const int p = L - m + r;  /* this query's position */
        const int g = hq / G;
        const int64_t qi = ((int64_t)(q_offsets[i] + r) * num_q_heads + hq) * D;
        const double *qv = q + qi;
        double *o = out + qi;
        double *sc = (double *)malloc(sizeof(double) * (size_t)(p + 1));
        double mx = -INFINITY;
        for (int j = 0; j <= p; ++j) {
          const int blk = row[j / bs], slot = j % bs;
          double dot = 0.0;
          for (int t = 0; t < D; ++t)
            dot += qv[t] * load_elem(c->k_pool, k_index(c, blk, g, slot, t), c->is_bf16);
          sc[j] = dot * scale;
          if (sc[j] > mx) mx = sc[j];
        }
        double Z = 0.0;
        for (int j = 0; j <= p; ++j) {
          sc[j] = exp(sc[j] - mx);
          Z += sc[j];
        }
        for (int j = 0; j <= p; ++j) {
          const int blk = row[j / bs], slot = j % bs;
          const double w = sc[j] / Z;
          for (int t = 0; t < D; ++t)
            o[t] += w * load_elem(c->v_pool, v_index(c, blk, g, slot, t), c->is_bf16);
        }
        free(sc);
      }
    }
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Test-only layer input side: how a frozen backbone turns an input         */
/* embedding at a (compressed) position into q, k, v.  Used to build K/V   */
/* for the end-to-end invariants; it is not part of the merged path.        */

static void rope_rotate_half(double *v, int D, double pos, double theta) {
  const int half = D / 2;
  for (int i = 0; i < half; ++i) {
    const double inv_freq = pow(theta, -2.0 * i / D);
    const double ang = pos * inv_freq;
    const double cs = cos(ang), sn = sin(ang);
    const double x1 = v[i], x2 = v[i + half];
    v[i] = x1 * cs - x2 * sn;
    v[i + half] = x2 * cs + x1 * sn;
  }
}

void orc_layer_qkv(int T, int d, const double *x, const int32_t *pos,
                   int num_q_heads, int num_kv_heads, int head_dim,
                   double rope_theta, double rms_eps, const double *W_q,
                   const double *W_k, const double *W_v, double *q, double *k,
                   double *v) {
  double *xn = (double *)malloc(sizeof(double) * (size_t)d);
  for (int t = 0; t < T; ++t) {
    const double *xt = x + (int64_t)t * d;
    double ms = 0.0;
    for (int i = 0; i < d; ++i) ms += xt[i] * xt[i];
    const double inv = 1.0 / sqrt(ms / d + rms_eps);
    for (int i = 0; i < d; ++i) xn[i] = xt[i] * inv;
    double *qt = q + (int64_t)t * num_q_heads * head_dim;
    double *kt = k + (int64_t)t * num_kv_heads * head_dim;
    double *vt = v + (int64_t)t * num_kv_heads * head_dim;
    linear(W_q, NULL, xn, d, num_q_heads * head_dim, qt);
    linear(W_k, NULL, xn, d, num_kv_heads * head_dim, kt);
    linear(W_v, NULL, xn, d, num_kv_heads * head_dim, vt);
    for (int hh = 0; hh < num_q_heads; ++hh)
      rope_rotate_half(qt + (int64_t)hh * head_dim, head_dim, pos[t], rope_theta);
    for (int hh = 0; hh < num_kv_heads; ++hh)
      rope_rotate_half(kt + (int64_t)hh * head_dim, head_dim, pos[t], rope_theta);
  }
  free(xn);
}

/* ------------------------------------------------------------------------ */
/* Merge rules and their matching (appendix "Non-overlapping Assignment in  */
/* a Sequence", "Rule Matching", "Decoding-time Integration").              */

static int key_cmp(const int32_t *a, const int32_t *b) {
  for (int i = 0; i < 4; ++i)
    if (a[i] != b[i]) return a[i] < b[i] ? -1 : 1;
  return 0;
}

static int rule_len(const int32_t *k) { /* n >= 2 leading ids >= 0, then -1; else 0 */
  int n = 0;
  while (n < 4 && k[n] >= 0) ++n;
  for (int i = n; i < 4; ++i)
    if (k[i] != -1) return 0;
  return n >= 2 ? n : 0;
}

static const int32_t *g_sort_keys; /* qsort context: input rules */
static int idx_cmp(const void *pa, const void *pb) {
  const int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
  const int c = key_cmp(g_sort_keys + 4 * (int64_t)a, g_sort_keys + 4 * (int64_t)b);
  return c != 0 ? c : (a < b ? -1 : a > b);
}

int orc_rules_init(orc_rules *r, const int32_t *rules, int count) {
  r->count = 0;
  r->keys = NULL;
  r->ids = NULL;
  if (count < 0) return ORC_EINVAL;
  for (int i = 0; i < count; ++i)
    if (!rule_len(rules + 4 * (int64_t)i)) return ORC_EINVAL;
  int32_t *order = (int32_t *)malloc(sizeof(int32_t) * (size_t)(count > 0 ? count : 1));
  for (int i = 0; i < count; ++i) order[i] = i;
  g_sort_keys = rules;
  qsort(order, (size_t)count, sizeof(int32_t), idx_cmp);
  r->keys = (int32_t *)malloc(sizeof(int32_t) * 4 * (size_t)(count > 0 ? count : 1));
  r->ids = (int32_t *)malloc(sizeof(int32_t) * (size_t)(count > 0 ? count : 1));
  for (int i = 0; i < count; ++i) {
    const int32_t *k = rules + 4 * (int64_t)order[i];
    /* equal keys are adjacent, smallest index first: keep that one */
    if (r->count > 0 && key_cmp(r->keys + 4 * (int64_t)(r->count - 1), k) == 0) continue;
    for (int j = 0; j < 4; ++j) r->keys[4 * (int64_t)r->count + j] = k[j];
    r->ids[r->count++] = order[i];
  }
  free(order);
  return ORC_OK;
}

void orc_rules_free(orc_rules *r) {
  free(r->keys);
  free(r->ids);
  r->keys = NULL;
  r->ids = NULL;
  r->count = 0;
}

int orc_rules_find(const orc_rules *r, const int32_t *gram, int n) {
  if (n < 2 || n > 4) return -1;
  int32_t k[4] = {-1, -1, -1, -1};
  for (int i = 0; i < n; ++i) {
    if (gram[i] < 0) return -1;
    k[i] = gram[i];
  }
  int lo = 0, hi = r->count - 1;
  while (lo <= hi) {
    const int mid = lo + (hi - lo) / 2;
    const int c = key_cmp(r->keys + 4 * (int64_t)mid, k);
    if (c == 0) return r->ids[mid];
    if (c < 0) lo = mid + 1;
    else hi = mid - 1;
  }
  return -1;
}

int orc_match_prompt(const orc_rules *r, int B, const int32_t *seq_offsets,
                     const int32_t *token_ids, int32_t *span_start,
                     int32_t *span_len, int32_t *span_rule,
                     int32_t *seq_span_offsets) {
  if (B < 0 || seq_offsets[0] != 0) return ORC_EINVAL;
  for (int b = 0; b < B; ++b)
    if (seq_offsets[b + 1] < seq_offsets[b]) return ORC_EINVAL;
  int S = 0;
  for (int b = 0; b < B; ++b) {
    seq_span_offsets[b] = S;
    const int32_t *x = token_ids + seq_offsets[b];
    const int T = seq_offsets[b + 1] - seq_offsets[b];
    int i = 0;
    while (i < T) {
      int taken = 0;
      for (int n = 4; n >= 2 && !taken; --n) {
        if (i + n > T) continue;
        const int id = orc_rules_find(r, x + i, n);
        if (id >= 0) {
          span_start[S] = seq_offsets[b] + i;
          span_len[S] = n;
          span_rule[S] = id;
          ++S;
          i += n;
          taken = 1;
        }
      }
      if (!taken) i += 1;
    }
  }
  seq_span_offsets[B] = S;
  return ORC_OK;
}

void orc_match_decode_step(const orc_rules *r, int32_t *state, int *state_len,
                           int32_t token, int32_t *k_out, int32_t *rule_out) {
  state[(*state_len)++] = token;
  *k_out = 0;
  *rule_out = -1;
  for (int n = 4; n >= 2; --n) {
    if (*state_len < n) continue;
    const int32_t *tail = state + *state_len - n;
    int raw = 1;
    for (int j = 0; j < n; ++j)
      if (tail[j] == ORC_MERGED) raw = 0;
    if (!raw) continue;
    const int id = orc_rules_find(r, tail, n);
    if (id < 0) continue;
    *state_len -= n;
    state[(*state_len)++] = ORC_MERGED;
    *k_out = n - 1;
    *rule_out = id;
    return;
  }
}

/* ------------------------------------------------------------------------ */
/* Surrogate lookup and span dedupe ("Computational Scope").                */

int orc_gather_surrogates(const void *emb, int64_t emb_rows, const void *lut,
                          int64_t lut_rows, const int32_t *token_ids,
                          const int32_t *rule_ids, int n, int d,
                          int elem_bytes, void *out) {
  int st = ORC_OK;
  for (int i = 0; i < n; ++i) {
    const char *src = NULL;
    if (rule_ids[i] >= 0) {
      if (rule_ids[i] < lut_rows) src = (const char *)lut + (int64_t)rule_ids[i] * d * elem_bytes;
    } else if (token_ids && token_ids[i] >= 0 && token_ids[i] < emb_rows) {
      src = (const char *)emb + (int64_t)token_ids[i] * d * elem_bytes;
    }
    char *dst = (char *)out + (int64_t)i * d * elem_bytes;
    if (src) {
      for (int64_t b = 0; b < (int64_t)d * elem_bytes; ++b) dst[b] = src[b];
    } else {
      for (int64_t b = 0; b < (int64_t)d * elem_bytes; ++b) dst[b] = 0;
      st = ORC_EINVAL;
    }
  }
  return st;
}

int orc_span_dedupe(const int32_t *span_rule, const int32_t *span_start,
                    const int32_t *span_len, int S, int num_rules,
                    const int32_t *token_ids, int32_t *uniq_span,
                    int32_t *span_slot, int32_t *uniq_row_idx,
                    int32_t *uniq_span_offsets) {
  for (int s = 0; s < S; ++s)
    if (span_rule[s] < 0 || span_rule[s] >= num_rules) return -1;
  int U = 0;
  uniq_span_offsets[0] = 0;
  for (int s = 0; s < S; ++s) {
    int first = -1; /* an earlier span with the same rule */
    for (int p = 0; p < s && first < 0; ++p)
      if (span_rule[p] == span_rule[s]) first = p;
    if (first < 0) {
      span_slot[s] = U;
      uniq_span[U] = s;
      const int off = uniq_span_offsets[U];
      for (int j = 0; j < span_len[s]; ++j) uniq_row_idx[off + j] = token_ids[span_start[s] + j];
      uniq_span_offsets[U + 1] = off + span_len[s];
      ++U;
    } else {
      span_slot[s] = span_slot[first];
    }
  }
  return U;
}

/* ------------------------------------------------------------------------ */
/* The surrogate's K/V state at its compressed position.                    */

int orc_kv_project(const orc_cache *c, const int32_t *seq_ids, int n,
                   const double *x, int d, const double *W_k,
                   const double *W_v, double rope_theta, double rms_eps,
                   double *K, double *V) {
  const int H = c->num_kv_heads, D = c->head_dim;
  for (int i = 0; i < n; ++i)
    if (seq_ids[i] < 0 || seq_ids[i] >= c->max_seqs) return ORC_EINVAL;
  double *xn = (double *)malloc(sizeof(double) * (size_t)d);
  for (int i = 0; i < n; ++i) {
    const double *xi = x + (int64_t)i * d;
    double ms = 0.0;
    for (int j = 0; j < d; ++j) ms += xi[j] * xi[j];
    const double inv = 1.0 / sqrt(ms / d + rms_eps);
    for (int j = 0; j < d; ++j) xn[j] = xi[j] * inv;
    double *ki = K + (int64_t)i * H * D, *vi = V + (int64_t)i * H * D;
    linear(W_k, NULL, xn, d, H * D, ki);
    linear(W_v, NULL, xn, d, H * D, vi);
    const double pos = c->lengths[seq_ids[i]];
    for (int h = 0; h < H; ++h) rope_rotate_half(ki + (int64_t)h * D, D, pos, rope_theta);
  }
  free(xn);
  return ORC_OK;
}
