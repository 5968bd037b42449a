/*
 * oracle.h -- plain, slow, obviously-correct CPU reference of the
 * span-merging inference hot path, in double precision.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or helper with the GPU library; the two meet only through
 * the seeded inputs the tests hand to both.
 *
 * Floating inputs arrive as double (bf16 / fp32 values widen exactly);
 * floating outputs stay double.  Paged-cache pools hold the raw storage
 * elements (2-byte bf16 or 4-byte fp32 bit patterns) so that copies can be
 * compared bit for bit.
 *
 * Status codes: 0 ok, 1 invalid argument, 2 out of range, 3 out of blocks.
 * Every cache call validates the whole request list first and changes
 * nothing when it fails.  Checks run in the order invalid -> range -> memory
 * and the first class that fails is returned.
 */
#ifndef SPANMERGE_ORACLE_H
#define SPANMERGE_ORACLE_H

#include <stdint.h>

#define ORC_OK 0
#define ORC_EINVAL 1
#define ORC_ERANGE 2
#define ORC_ENOMEM 3

/* Paged cache (element storage: elem_bytes = 2 for bf16, 4 for fp32).
 *   K page: [num_blocks][num_kv_heads][block_size][head_dim]
 *   V page: [num_blocks][num_kv_heads][head_dim][block_size]
 * Cached entry j of sequence s sits in physical block
 * block_table[s * max_blocks_per_seq + j / block_size], slot j % block_size. */
typedef struct {
  int is_bf16;
  int num_kv_heads, head_dim, block_size, num_blocks, max_seqs,
      max_blocks_per_seq;
  void *k_pool, *v_pool;
  int32_t *block_table, *lengths, *free_stack, *free_top;
} orc_cache;

/* M_phi over num_spans spans (double everywhere).  flags bit 0: drop GELU,
 * LayerNorm and biases, which gives the bare form of the main text's Eq. 1. */
int orc_merge_spans(int d, int h, double ln_eps, const double *emb,
                    int64_t emb_rows, const int32_t *row_idx,
                    const int32_t *span_offsets, int num_spans,
                    const double *Q, const double *W_kv, const double *b_kv,
                    const double *g_kv, const double *beta_kv,
                    const double *W_o, const double *b_o, const double *g_o,
                    const double *beta_o, int flags, double *out,
                    double *pool_weights /* nullable [num_spans][h][max n] */,
                    int pool_weights_stride);

int orc_pack_spans(int B, const int32_t *seq_offsets, int num_spans,
                   const int32_t *span_start, const int32_t *span_len,
                   const int32_t *seq_span_offsets, int32_t *pi,
                   int32_t *packed_offsets, int32_t *packed_src,
                   const int32_t *token_ids, const void *emb,
                   int64_t emb_rows, const void *surrogates, int d,
                   int elem_bytes, void *packed /* nullable */);

int orc_kv_rollback(orc_cache *c, const int32_t *seq_ids, const int32_t *k,
                    int n);

int orc_kv_append(orc_cache *c, const int32_t *seq_ids,
                  const int32_t *row_offsets, int n, const void *K,
                  const void *V);

int orc_decode_attention(const orc_cache *c, const int32_t *seq_ids, int n,
                         const double *q, int num_q_heads, double scale,
                         double *out, double *probs /* nullable, see .c */,
                         int probs_stride);

/* Prefill attention over the cache ("Efficiency Analysis": the prefill
 * pass runs over the compressed sequence).  Request i's m_i query rows
 * q[q_offsets[i] .. q_offsets[i+1]) are the last m_i cached positions of
 * sequence seq_ids[i] (full prefill: m_i = length; chunked: fewer); row r
 * sits at position p = L - m_i + r and attends causally to entries 0..p.
 * q: [rows][num_q_heads][head_dim]; out: same shape. */
int orc_prefill_attention(const orc_cache *c, const int32_t *seq_ids, int n,
                          const int32_t *q_offsets, const double *q,
                          int num_q_heads, double scale, double *out);

/* Test-only attention-layer input side (not part of the merged path): unit
 * RMSNorm, then q/k/v projections, rotate-half RoPE at the given positions. */
void orc_layer_qkv(int T, int d, const double *x, const int32_t *pos,
                   int num_q_heads, int num_kv_heads, int head_dim,
                   double rope_theta, double rms_eps, const double *W_q,
                   const double *W_k, const double *W_v, double *q, double *k,
                   double *v);

/* Merge rules (appendix "Non-overlapping Assignment in a Sequence" and
 * "Rule Matching").  A rule is an n-gram of token ids, n = 2..4, given as 4
 * int32 with the unused tail set to -1.  The rule set R is a set: a rule
 * listed twice keeps its first index as its id.  The oracle holds R as a
 * sorted array searched by bisection. */
typedef struct {
  int count;      /* distinct rules */
  int32_t *keys;  /* [count][4], sorted lexicographically */
  int32_t *ids;   /* [count] smallest input index of each key */
} orc_rules;

/* Validates every rule (n >= 2 leading ids >= 0, then -1) and builds R;
 * EINVAL (and an empty set) if any rule is malformed. */
int orc_rules_init(orc_rules *r, const int32_t *rules, int count);
void orc_rules_free(orc_rules *r);
/* id of the n-gram gram[0..n) in R, or -1 (any negative token: -1). */
int orc_rules_find(const orc_rules *r, const int32_t *gram, int n);

/* Prompt-time assignment: for each sequence b (tokens seq_offsets[b] ..
 * seq_offsets[b+1]) scan left to right; at position i try n = 4, 3, 2 and
 * take the first n whose full window is a rule, then jump past it, else
 * step one token.  Spans come out in order: global start, length, rule id;
 * seq_span_offsets [B+1] gives each sequence's range.  Capacity of the span
 * arrays: seq_offsets[B] / 2. */
int orc_match_prompt(const orc_rules *r, int B, const int32_t *seq_offsets,
                     const int32_t *token_ids, int32_t *span_start,
                     int32_t *span_len, int32_t *span_rule,
                     int32_t *seq_span_offsets);

/* Decode-time check after one generated token (appendix "Decoding-time
 * Integration"): state[0..*state_len) is the generated-state list, raw
 * token ids >= 0 and ORC_MERGED for a surrogate.  The token is appended,
 * then the longest n in 4, 3, 2 whose last n entries are all raw and form a
 * rule is merged: those n entries become one ORC_MERGED.  *k_out = n - 1
 * entries to crop from the cache (0 without a match), *rule_out = rule id
 * or -1.  The list needs room for one more entry. */
#define ORC_MERGED (-2)
void orc_match_decode_step(const orc_rules *r, int32_t *state, int *state_len,
                           int32_t token, int32_t *k_out, int32_t *rule_out);

/* Surrogate lookup ("Computational Scope": a span's surrogate depends on
 * its tokens only, so surrogates can be precomputed per rule and looked
 * up).  out[i] = lut[rule_ids[i]] when rule_ids[i] >= 0, else
 * emb[token_ids[i]]: the step input of a decode step (surrogate or plain
 * token) and the surrogates of a prompt's spans.  Rows are raw elements of
 * elem_bytes; an index out of range gives EINVAL and a zero row. */
int orc_gather_surrogates(const void *emb, int64_t emb_rows, const void *lut,
                          int64_t lut_rows, const int32_t *token_ids,
                          const int32_t *rule_ids, int n, int d,
                          int elem_bytes, void *out);

/* Span dedupe within one merge batch: spans with the same rule share one
 * surrogate.  uniq_span[u] = the u-th span (in order) whose rule has not
 * occurred before it; span_slot[s] = u of the first span with s's rule;
 * returns the number of unique spans (or -1 for a rule id outside
 * [0, num_rules)).  The unique spans' rows for the merge module come out
 * as CSR: uniq_row_idx (token ids) and uniq_span_offsets [U + 1]. */
int orc_span_dedupe(const int32_t *span_rule, const int32_t *span_start,
                    const int32_t *span_len, int S, int num_rules,
                    const int32_t *token_ids, int32_t *uniq_span,
                    int32_t *span_slot, int32_t *uniq_row_idx,
                    int32_t *uniq_span_offsets);

/* The surrogate's single K/V state (appendix "Decoding-time Integration":
 * the frozen backbone processes z_s as one input embedding; the K/V
 * append): for request i, the input row x[i] (a surrogate or a plain
 * token embedding) at the compressed position p = lengths[seq_ids[i]] (the
 * slot it will take) gives, per kv head, K = RoPE_p(W_k RMSNorm(x)) and
 * V = W_v RMSNorm(x), the first layer's input side with the norm's gain
 * folded into W_k, W_v.  K, V: [n][num_kv_heads][head_dim]. */
int orc_kv_project(const orc_cache *c, const int32_t *seq_ids, int n,
                   const double *x, int d, const double *W_k,
                   const double *W_v, double rope_theta, double rms_eps,
                   double *K, double *V);

/* Number of OpenMP threads the oracle's parallel loops use. */
int orc_num_threads(void);
void orc_set_num_threads(int n);

#endif
