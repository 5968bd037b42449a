/*
 * spanmerge.h -- C ABI of the span-merging (UMIM) inference hot path on
 * AMD Instinct MI355X (gfx950).
 *
 * The method ("Distilling Sequential Computation in Transformer Language
 * Models", arXiv 2609.27233) replaces a span of n input tokens by one
 * surrogate embedding produced by a small attention-pooling merge module
 * M_phi (Sec. 3.2 Eq. 1; appendix "Module Architecture and Integration").
 * At inference it compresses prompts before prefill and, during decoding,
 * rolls back the n-1 cached entries of a freshly completed span and appends
 * the surrogate's single K/V state (appendix "Inference with UMIM: Prompt and
 * Decoding-Time Merging").  Every later decode step then attends over the
 * shorter cache.  The calls below are the device-side steps of that
 * path:
 *
 *   sm_merge_spans      z_s = M_phi(e(x_span))            for every span s
 *   sm_pack_spans       keep mask -> compressed positions -> packed rows
 *   sm_kv_rollback      crop k entries from the tail of each listed sequence
 *   sm_kv_append        append K/V rows (one surrogate state, or a prompt)
 *   sm_decode_attention one query per sequence over its whole paged cache
 *   sm_prefill_attention causal attention of a prompt's positions over the
 *                       paged cache (the prefill pass over the compressed
 *                       sequence)
 *   sm_rules_build      the merge-rule set R as a device hash table
 *   sm_match_prompt     left-to-right, longest-first, non-overlapping spans
 *                       of a prompt batch
 *   sm_match_decode     the raw-suffix check after one generated token, with
 *                       the cache crop it implies
 *   sm_gather_surrogates surrogates looked up per rule (or plain token rows)
 *   sm_span_dedupe      one surrogate per distinct rule in a merge batch
 *   sm_kv_project       the K/V state of an input row (surrogate or token) at
 *                       its compressed position; sm_kv_append_projected
 *                       appends it
 *
 * General rules for every call
 * ----------------------------
 *  - Every pointer is a DEVICE pointer unless its comment says (host).
 *  - The caller owns every buffer (tables, pools, workspaces, outputs); the
 *    library allocates nothing and never synchronizes.  Its only state: the
 *    per-device scratch array of sm_decode_step_noalloc and the test-only
 *    bound of sm_set_commit_wait_limit.
 *    Work is enqueued on `stream` (0 = the null stream); pointers must stay
 *    valid until that work has completed.  Calls are safe to capture in a
 *    HIP graph.
 *  - Synchronous status: SM_EINVAL for arguments the host can check (null
 *    pointers, unsupported shapes, a workspace that is too small); SM_EHIP if
 *    a kernel launch fails.  Nothing is enqueued when a call returns non-OK.
 *  - Asynchronous status: problems only visible to the device (indices read
 *    from device memory) OR a bit into a device error word `err`
 *    (SM_ERR_EINVAL / SM_ERR_ERANGE / SM_ERR_ENOMEM).  The word is sticky: a
 *    mutating cache call (rollback, append) that finds `*err != 0` when it
 *    starts does nothing, so a failed call leaves the cache exactly as it
 *    was (all-or-nothing) and the cache stays frozen until the caller has
 *    read and cleared the word.  Exactly one bit is set per failing call,
 *    checked in the order EINVAL, ERANGE, ENOMEM.  No index read from device
 *    memory is ever used to address memory before it has been range-checked.
 *
 * Dtypes: SM_F32 (fp32 storage, fp32 arithmetic) and SM_BF16 (bf16 storage,
 * fp32 accumulation, outputs rounded to nearest-even bf16).
 */
#ifndef SPANMERGE_H
#define SPANMERGE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { SM_F32 = 0, SM_BF16 = 1 } sm_dtype;

typedef enum {
  SM_OK = 0,
  SM_EINVAL = 1, /* bad argument */
  SM_ERANGE = 2, /* length / capacity out of range */
  SM_ENOMEM = 3, /* not enough free KV blocks */
  SM_EHIP = 4    /* a HIP launch failed */
} sm_status;

/* bits of the device error word */
enum { SM_ERR_EINVAL = 1, SM_ERR_ERANGE = 2, SM_ERR_ENOMEM = 4 };

/* Largest number of requests (sequences) in one rollback / append call. */
#define SM_MAX_REQUESTS 1024

/*
 * Parameters phi of the merge module M_phi (appendix "Attention-based Pooling
 * Architecture" and "Parameter Count": |phi| = 2d^2 + 7d).  Storage dtype is
 * the call's dtype.  Linear layers compute y = W x + b with W stored
 * row-major [out = d][in = d].  The pooling splits the d features into h
 * contiguous head blocks of d_h = d / h features.
 */
typedef struct {
  int d;            /* model width (= M_phi width) */
  int h;            /* pooling heads; the paper uses 4 */
  float ln_eps;     /* LayerNorm epsilon (1e-5) */
  const void *Q;    /* [h][d_h] learned pooling queries q_i */
  const void *W_kv; /* [d][d] token projection Linear_kv */
  const void *b_kv; /* [d] */
  const void *g_kv; /* [d] LN_kv gain */
  const void *beta_kv; /* [d] LN_kv bias */
  const void *W_o;  /* [d][d] output projection Linear_o */
  const void *b_o;  /* [d] */
  const void *g_o;  /* [d] LN_o gain */
  const void *beta_o;  /* [d] LN_o bias */
} sm_merge_params;

/*
 * Paged KV cache of one attention layer, over caller-owned buffers.
 *
 *  k_pool  [num_blocks][num_kv_heads][block_size][head_dim]  token-major pages
 *  v_pool  [num_blocks][num_kv_heads][head_dim][block_size]  dim-major pages
 *          (V is stored transposed inside each page so that the decode
 *          kernel can feed it to the matrix cores without a transpose)
 *  block_table [max_seqs][max_blocks_per_seq]  physical block of each logical
 *          block, -1 when unmapped
 *  lengths     [max_seqs]   cached entries per sequence
 *  free_stack  [num_blocks] LIFO stack of free physical blocks; the next pop
 *          returns free_stack[*free_top - 1]
 *  free_top    [1]
 *  err         [1]          sticky device error word (see above)
 *
 * Entry j of sequence s lives in block block_table[s][j / block_size] at
 * slot j % block_size.  head_dim must be 64 or 128; block_size must be a
 * power of two in [16, 512]; num_kv_heads * head_dim <= 2048.  Pools must
 * be 16-byte aligned.
 */
typedef struct {
  sm_dtype dtype;
  int num_kv_heads;
  int head_dim;
  int block_size;
  int num_blocks;
  int max_seqs;
  int max_blocks_per_seq;
  void *k_pool;
  void *v_pool;
  int32_t *block_table;
  int32_t *lengths;
  int32_t *free_stack;
  int32_t *free_top;
  int32_t *err;
} sm_paged_cache;

/* Human-readable name of a status code (host, static storage). */
const char *sm_status_string(sm_status s);

/* Bytes of workspace sm_merge_spans needs for these sizes. */
size_t sm_merge_workspace_bytes(int total_rows, int num_spans, int d,
                                sm_dtype dt);

/*
 * sm_merge_spans -- z_s = M_phi(E_s) for every span s in one launch sequence
 * (Sec. 3.2 Eq. 1; the appendix form with GELU and LayerNorm in
 * "Attention-based Pooling Architecture"):
 *
 *   P   = LN_kv(GELU(Linear_kv(E_s)))                 E_s: the span's n rows
 *   a_i = softmax_j(P[j, head i] . q_i / sqrt(d_h)),  o_i = sum_j a_i[j] P[j, head i]
 *   z_s = LN_o(GELU(Linear_o([o_1; ...; o_h])))
 *
 * GELU is the exact erf form (evaluated through erfc to about 1e-6
 * relative); LayerNorm uses the biased variance.  bf16 calls round the
 * intermediate rows to bf16 and accumulate in fp32; large bf16 calls run
 * the first projection with the rows in token-id order, so the rounding of
 * one span's result can depend on the other spans of the call.
 *
 *  emb           [emb_rows][d] static embedding table (dtype dt)
 *  row_idx       [total_rows] row of emb for each span token, spans stored
 *                back to back (CSR)
 *  span_offsets  [num_spans + 1] span s owns row_idx[span_offsets[s] ..
 *                span_offsets[s+1]); span_offsets[0] = 0,
 *                span_offsets[num_spans] = total_rows, every span has n >= 1
 *  total_rows    (host) sum of span lengths
 *  p             (host) parameters; d % h == 0, d % 256 == 0, d / h % 64 == 0
 *  out           [num_spans][d] surrogates (dtype dt)
 *  ws, ws_bytes  workspace of at least sm_merge_workspace_bytes(...) bytes
 *  err           [1] device error word: EINVAL when a row index is outside
 *                [0, emb_rows) (that row is read as row 0) or the span
 *                offsets are not a valid CSR (the pooled vector of such a
 *                span is zero, so its surrogate is LN_o(GELU(b_o)); the
 *                other spans are pooled as usual)
 */
sm_status sm_merge_spans(const void *emb, int64_t emb_rows,
                         const int32_t *row_idx, int total_rows,
                         const int32_t *span_offsets, int num_spans,
                         const sm_merge_params *p, sm_dtype dt, void *out,
                         void *ws, size_t ws_bytes, int32_t *err,
                         hipStream_t stream);

/*
 * sm_merge_token_table -- the first stage of M_phi for every row of the
 * embedding table, once (appendix "Attention-based Pooling Architecture":
 * Linear_kv and GELU act on each static token embedding on its own, so
 * their output depends on the token alone -- the same context
 * independence "Computational Scope" notes for whole surrogates):
 *
 *   table[v] = GELU(Linear_kv(emb[v]))     v = 0 .. emb_rows - 1
 *
 *  emb       [emb_rows][d] static embedding table (dtype dt), emb_rows < 2^31
 *  p         (host) the merge parameters (only W_kv, b_kv are read; all
 *            must be set, as for sm_merge_spans)
 *  table     [emb_rows][d] output (dtype dt), caller-owned
 *  err       [1] device error word (no device errors are raised)
 * No workspace.  One GEMM on the matrix cores; it is the cost of
 * sm_merge_spans's first projection for emb_rows rows.
 */
sm_status sm_merge_token_table(const void *emb, int64_t emb_rows,
                               const sm_merge_params *p, sm_dtype dt,
                               void *table, int32_t *err, hipStream_t stream);

/*
 * sm_merge_spans_tabled -- the same surrogates as sm_merge_spans, with the
 * first stage read from a table made by sm_merge_token_table (LN_kv, the
 * pooling, Linear_o, GELU and LN_o run per call):
 *
 *  table, table_rows  [table_rows][d] rows GELU(Linear_kv(emb[v]))
 *  row_idx, total_rows, span_offsets, num_spans, p, dt, out, err:
 *            as sm_merge_spans (row_idx holds token ids, i.e. table rows)
 *  ws, ws_bytes  workspace of at least
 *                sm_merge_workspace_bytes(0, num_spans, d, dt) bytes
 * Device errors: as sm_merge_spans, with table_rows in place of emb_rows.
 */
sm_status sm_merge_spans_tabled(const void *table, int64_t table_rows,
                                const int32_t *row_idx, int total_rows,
                                const int32_t *span_offsets, int num_spans,
                                const sm_merge_params *p, sm_dtype dt,
                                void *out, void *ws, size_t ws_bytes,
                                int32_t *err, hipStream_t stream);

/*
 * sm_pack_spans -- prompt compression bookkeeping (appendix "Prompt-time
 * Integration"; "Inference with UMIM", paragraph "Prompt Merging").
 * A merged span keeps only its LAST position (its surrogate is anchored
 * there: "Mask Construction and Sequence Alignment"); compressed positions
 * are contiguous ("Positional Encoding under Token-Span Merging":
 * pi(t) = t - r(t)).  For sequence b with tokens [seq_offsets[b],
 * seq_offsets[b+1]):
 *
 *   keep[t]   = 0 if t lies in a span and is not its last token, else 1
 *   pi[t]     = sum_{t' < t, same sequence} keep[t']   (span tokens all get
 *               their surrogate's position)
 *   L~_b      = (#tokens of b) - sum_{spans of b} (n - 1)
 *   packed_offsets[b] = sum_{b' < b} L~_b'
 *   packed_src[packed_offsets[b] + pi[t]] = t (global token index) for a
 *               token outside every span, and -1 - s for span s
 *   packed[...] (optional) = emb[token_ids[t]] or surrogates[s], same rule
 *
 *  seq_offsets      [B + 1] token ranges of the B sequences
 *  total_tokens     (host) seq_offsets[B]
 *  span_start       [num_spans] global token index where span s starts
 *  span_len         [num_spans] n >= 1
 *  seq_span_offsets [B + 1] spans of sequence b are [seq_span_offsets[b],
 *                   seq_span_offsets[b+1]), sorted by start, non-overlapping
 *  pi               [total_tokens] out
 *  packed_offsets   [B + 1] out
 *  packed_src       [total_tokens] out (capacity; sum L~ entries written)
 *  token_ids, emb, surrogates, packed: only used when packed != NULL;
 *                   packed is [total_tokens][d] capacity, dtype dt
 *  err              [1] EINVAL when the span list is not sorted,
 *                   non-overlapping and inside its sequence, or a token id
 *                   is outside [0, emb_rows)
 */
sm_status sm_pack_spans(int B, const int32_t *seq_offsets, int total_tokens,
                        int num_spans, const int32_t *span_start,
                        const int32_t *span_len,
                        const int32_t *seq_span_offsets, int32_t *pi,
                        int32_t *packed_offsets, int32_t *packed_src,
                        const int32_t *token_ids, const void *emb,
                        int64_t emb_rows, const void *surrogates, int d,
                        sm_dtype dt, void *packed, int32_t *err,
                        hipStream_t stream);

/*
 * sm_kv_rollback -- the decoding-time cache crop (appendix "Decoding-time
 * Integration" and "Decoding-Time Merging and KV-Cache Update": crop the n-1
 * cached entries of a matched span, L_C' = L_C - (n-1) + 1 once the
 * surrogate is appended).  For request i: lengths[seq_ids[i]] -= k[i].
 * Logical blocks no longer needed are unmapped (-1) and pushed on the free
 * stack; requests are processed in reverse list order, and within a request
 * from the highest logical block down.  KV bytes are not touched.
 *
 *  c        (host) cache descriptor
 *  seq_ids  [n] distinct sequence ids in [0, max_seqs)
 *  k        [n] 0 <= k[i] <= lengths[seq_ids[i]]
 *  n        (host) 0 <= n <= min(max_seqs, SM_MAX_REQUESTS)
 * Device errors: EINVAL (id out of range, duplicate id, k < 0),
 * ERANGE (k > length).
 */
sm_status sm_kv_rollback(const sm_paged_cache *c, const int32_t *seq_ids,
                         const int32_t *k, int n, hipStream_t stream);

/*
 * sm_kv_append -- append K/V rows at the tail of each listed sequence; the
 * surrogate's single-step state after a rollback (Decoding-Time Merging: the
 * surrogate forward "produces one new key and value state"), one ordinary
 * token per decode step, or a whole compressed prompt.  Requests are served
 * in list order; for each row the slot is pos = lengths[s], a block is
 * popped from the free stack when pos % block_size == 0, then the row is
 * copied and lengths[s] += 1.
 *
 *  seq_ids      [n] distinct sequence ids
 *  row_offsets  [n + 1] request i appends rows [row_offsets[i],
 *               row_offsets[i+1]) of K and V; row_offsets[0] = 0,
 *               row_offsets[n] = total_rows
 *  total_rows   (host)
 *  K, V         [total_rows][num_kv_heads][head_dim] (cache dtype)
 * Device errors: EINVAL (bad id, duplicate, bad offsets), ERANGE
 * (length would exceed max_blocks_per_seq * block_size), ENOMEM (not enough
 * free blocks for the whole call).
 */
sm_status sm_kv_append(const sm_paged_cache *c, const int32_t *seq_ids,
                       const int32_t *row_offsets, int n, int total_rows,
                       const void *K, const void *V, hipStream_t stream);

/* Bytes of workspace sm_decode_attention needs for these sizes. */
size_t sm_decode_workspace_bytes(int n, int num_q_heads, int head_dim,
                                 int max_len);

/*
 * sm_decode_attention -- one decode query per sequence attending over all
 * lengths[s] cached entries (the unchanged backbone attention the paper's
 * throughput study measures, "Efficiency Analysis"):
 *
 *   out[i, h] = sum_j softmax_j(scale * q[i, h] . K[s, j, g]) V[s, j, g]
 *   s = seq_ids[i],  g = h / (num_q_heads / num_kv_heads)   (grouped query)
 *
 * A sequence of length 0 gives zeros.  Implemented as one kernel: split-K
 * partials over chunks of the cache, combined exactly by the last workgroup
 * of each (sequence, kv head) to finish.
 *
 *  seq_ids      [n] ids in [0, max_seqs) (repeats allowed)
 *  q            [n][num_q_heads][head_dim] (cache dtype)
 *  num_q_heads  (host) multiple of num_kv_heads, group size <= 16
 *  max_len      (host) upper bound on lengths[seq_ids[i]]; sizes the grid
 *  out          [n][num_q_heads][head_dim] (cache dtype)
 *  ws, ws_bytes at least sm_decode_workspace_bytes(n, num_q_heads,
 *               head_dim, max_len).  Its first 256 KiB hold arrival
 *               counters: zero-fill them once before the first call; every
 *               call leaves them zero again, so one workspace serves calls
 *               of any shape.  Calls that may run concurrently must not
 *               share a workspace.  n * num_kv_heads <= 65536.
 * Device errors (into c->err; the affected rows are zero): EINVAL (bad id,
 * block id out of range), ERANGE (length > max_len).
 */
sm_status sm_decode_attention(const sm_paged_cache *c, const int32_t *seq_ids,
                              int n, const void *q, int num_q_heads,
                              float scale, int max_len, void *out, void *ws,
                              size_t ws_bytes, hipStream_t stream);

/*
 * sm_decode_step -- one decode step of a batch in a single launch: the new
 * token's K/V row of every sequence is appended and each sequence's new
 * query attends over its cache including that row (the per-step cache
 * growth and attention of "Efficiency Analysis").  Same results, cache
 * state and error bits as
 *   sm_kv_append(c, seq_ids, {0, 1, ..., n}, n, n, K, V)
 *   sm_decode_attention(c, seq_ids, n, q, num_q_heads, scale, max_len, ...)
 * issued back to back, up to the rounding order of the attention sums.  If
 * the append fails (or the error word was already set) the cache is left
 * as it was and the attention runs over it unchanged.
 *
 *  seq_ids      [n] distinct ids, n <= 256
 *  K, V         [n][num_kv_heads][head_dim] (cache dtype): the new rows
 *  q, out, num_q_heads, scale: as sm_decode_attention
 *  max_len      (host) upper bound on the lengths after the append
 *  ws, ws_bytes as sm_decode_attention (the same workspace may serve both
 *               calls, one at a time); n * num_kv_heads <= 65534
 * Device errors: those of sm_kv_append, then those of sm_decode_attention.
 */
sm_status sm_decode_step(const sm_paged_cache *c, const int32_t *seq_ids,
                         int n, const void *K, const void *V, const void *q,
                         int num_q_heads, float scale, int max_len, void *out,
                         void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * sm_decode_merge_step -- the decode step at which spans complete, in one
 * launch ("Decoding-Time Merging and KV-Cache Update"; "Decoding-time
 * Integration"): each request first drops its last crop[i] cached entries
 * (the raw tokens of the span that just completed, n - 1 of them), then its
 * row (the surrogate's K/V state, or the plain token's when crop[i] = 0) is
 * appended, and its query attends over the result: the cache goes from L to
 * L - crop[i] + 1 entries.  The crops and the append are one update, made
 * whole or not at all: its state and error bits are those of
 *   sm_kv_rollback(c, seq_ids, crop, n)
 *   sm_kv_append(c, seq_ids, {0, 1, ..., n}, n, n, K, V)
 * issued back to back when both succeed (the freed pages go onto the free
 * stack and the append pops from it exactly as the two calls do); when
 * either would fail, the cache is left as it was, the error bits of the
 * first failing check are set, and the attention runs over the unchanged
 * cache (as sm_decode_step's does when its append fails).  A rule match
 * decides the crops: sm_match_decode with cache = NULL writes them to k_out
 * without cropping, ready to pass here.
 *
 *  c            bf16 caches only (SM_EINVAL otherwise)
 *  seq_ids      [n] distinct ids, n <= 256
 *  crop         [n] (device) entries to drop per request, 0 <= crop[i] <=
 *               lengths[seq_ids[i]]
 *  K, V, q, num_q_heads, scale, out, ws, ws_bytes: as sm_decode_step
 *  max_len      (host) upper bound on the lengths before the crops
 * Device errors: EINVAL (bad or repeated id, negative crop, corrupt free
 * stack or block table), ERANGE (crop longer than the cache, no room on the
 * free stack for the freed blocks, length above capacity after the append),
 * ENOMEM (no free block for the append), then those of
 * sm_decode_attention.
 */
sm_status sm_decode_merge_step(const sm_paged_cache *c, const int32_t *seq_ids,
                               const int32_t *crop, int n, const void *K,
                               const void *V, const void *q, int num_q_heads,
                               float scale, int max_len, void *out, void *ws,
                               size_t ws_bytes, hipStream_t stream);

/*
 * sm_set_commit_wait_limit -- for tests of a fused step's give-up path (not
 * for production use).  A fused step's append is committed by one extra
 * workgroup once every attention workgroup has read the metadata; it polls
 * for that at most `polls` times (default 2^20, restored by polls <= 0),
 * which always suffices because every attention workgroup arrives without
 * waiting on anything.  If the bound is reached anyway, the call commits
 * nothing, sets EINVAL in c->err, and leaves the workspace's arrival counter
 * nonzero: zero the first 256 KiB of that workspace again before reusing it.
 * Process-wide; takes effect for calls issued after it returns.
 */
void sm_set_commit_wait_limit(int polls);

/*
 * sm_decode_step_noalloc -- for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): sm_decode_step with no workspace argument.  Its arrival
 * counters and split partials live in a fixed array inside the library,
 * one per device, held until the process ends; the call itself allocates
 * nothing.  Same results, cache state and error bits as sm_decode_step
 * (bit for bit: the same kernels with the same chunking).
 *
 *  arguments    as sm_decode_step, without ws / ws_bytes; the array of the
 *               current device is used, so `stream` must belong to it.
 *  size limit   n * num_q_heads * chunks * (head_dim + 2) * 4 bytes of
 *               partials must fit sm_decode_step_noalloc_max_bytes()
 *               (8 MiB); chunks is what the call's chunking uses (at most
 *               ceil(max_len / 256); 2 for 16 sequences of up to 4096
 *               entries, 8 KV heads).  Larger calls return SM_EINVAL and
 *               launch nothing.
 *  first call   on a device looks up the array's address and clears its
 *               counters with a fill kernel on `stream` (SM_EHIP if either
 *               fails); every call leaves them zero again.
 *  concurrency  every call on a device shares that device's array: calls
 *               that may overlap on one device (other streams, other host
 *               threads) race and must be serialised by the caller.
 */
size_t sm_decode_step_noalloc_max_bytes(void);
sm_status sm_decode_step_noalloc(const sm_paged_cache *c,
                                 const int32_t *seq_ids, int n, const void *K,
                                 const void *V, const void *q, int num_q_heads,
                                 float scale, int max_len, void *out,
                                 hipStream_t stream);

/*
 * sm_prefill_attention -- the attention of the prefill pass over the
 * compressed prompt ("Efficiency Analysis": prompt merging shortens the
 * sequence before the backbone runs, so every layer attends over the
 * compressed positions).  Request i's m_i = q_offsets[i+1] - q_offsets[i]
 * query rows are the last m_i cached positions of sequence s = seq_ids[i]
 * (append the prompt's K/V with sm_kv_append first; m_i < length gives a
 * chunked prefill over earlier context).  Row r sits at position
 * p = L - m_i + r, L = lengths[s], and attends causally to entries 0..p:
 *
 *   out[q_offsets[i] + r, h] = sum_{j <= p} softmax_j(scale q . K[s, j, g]) V[s, j, g]
 *   g = h / (num_q_heads / num_kv_heads)
 *
 *  seq_ids      [n] ids in [0, max_seqs) (repeats allowed), n <= 65535
 *  q_offsets    [n+1] row ranges into q and out, 0 <= q_offsets[i] <=
 *               q_offsets[i+1] <= total_rows
 *  total_rows   (host) rows of q and out
 *  q            [total_rows][num_q_heads][head_dim], bf16
 *  num_q_heads  (host) multiple of num_kv_heads, group size <= 16
 *  scale        (host) any finite value; 0 gives the mean of V[s, 0..p]
 *  max_rows     (host) upper bound on every m_i; sizes the grid
 *  out          [total_rows][num_q_heads][head_dim], bf16
 * bf16 caches only, head_dim 64 or 128, block_size a power of two >= 16,
 * max_blocks_per_seq <= 4096, one page of all kv heads (num_kv_heads x
 * block_size x head_dim x 2 bytes) < 4 GiB.  No workspace.
 * Device errors (into c->err; the request's rows are zero): EINVAL (bad id,
 * bad row range, m_i > L or > max_rows, block id out of range).
 */
sm_status sm_prefill_attention(const sm_paged_cache *c, const int32_t *seq_ids,
                               int n, const int32_t *q_offsets, int total_rows,
                               const void *q, int num_q_heads, float scale,
                               int max_rows, void *out, hipStream_t stream);

/*
 * Merge rules (appendix "Non-overlapping Assignment in a Sequence": R is the
 * union of the filtered 2-, 3- and 4-gram rules; about 2.17M for the Llama-3
 * tokenizer).  A rule is four int32: its n >= 2 token ids (>= 0), then -1
 * for the unused tail.  The table is an open-addressing hash set over
 * caller-owned device arrays; a built table is read-only.
 */
typedef struct {
  int capacity;      /* slots: a power of two >= 16, and >= 4/3 x the rules */
  int32_t *keys;     /* [capacity][4]; keys[s][0] == -1 marks an empty slot */
  int32_t *ids;      /* [capacity] index, in the build's rule list, of the
                        rule held in slot s (the first one when listed twice) */
  int32_t *err;      /* [1] sticky error bits */
} sm_rule_table;

/* Workspace of sm_rules_build: capacity x 8 bytes. */
size_t sm_rules_build_workspace_bytes(int capacity);

/*
 * sm_rules_build -- fill the table with rules[0..count) ([count][4], device).
 *  count  (host) 0 <= count <= 3/4 x capacity (else SM_EINVAL)
 *  ws     device workspace of sm_rules_build_workspace_bytes(capacity) bytes
 * Device errors: EINVAL for a malformed rule (fewer than 2 leading ids >= 0,
 * or a tail entry other than -1): that rule is left out and the table must
 * be rebuilt.  Slot placement may differ run to run; which keys are present
 * and their ids do not.
 */
sm_status sm_rules_build(const int32_t *rules, int count, const sm_rule_table *t,
                         void *ws, size_t ws_bytes, hipStream_t stream);

/* sm_rules_lookup -- ids[i] = id of grams[i] ([m][4], same form as a rule)
 * in R, or -1 (also for a malformed gram). */
sm_status sm_rules_lookup(const sm_rule_table *t, const int32_t *grams, int m,
                          int32_t *ids, hipStream_t stream);

/* Workspace of sm_match_prompt: about 17 bytes per token. */
size_t sm_match_prompt_workspace_bytes(int B, int total_tokens);

/*
 * sm_match_prompt -- prompt-time span assignment ("Rule Matching"): each
 * sequence is scanned left to right; at position i the 4-, 3- and then
 * 2-gram starting there is looked up, the first (longest) rule found becomes
 * a span and the scan jumps past it, else it steps one token.  A window
 * never crosses a sequence boundary, and a window holding a negative id
 * matches nothing.
 *  token_ids        [total_tokens] int32
 *  seq_offsets      [B+1] with 0 <= seq_offsets[b] <= seq_offsets[b+1] <=
 *                   total_tokens; B <= 65535
 *  span_start       [total_tokens / 2] out: global token index of each span
 *  span_len         [total_tokens / 2] out: 2..4
 *  span_rule        [total_tokens / 2] out: rule id
 *  seq_span_offsets [B+1] out: sequence b's spans are
 *                   [seq_span_offsets[b], seq_span_offsets[b+1]), in order
 * The outputs feed sm_pack_spans (span_start, span_len, seq_span_offsets)
 * and sm_merge_spans (the span's token ids as rows of the embedding table).
 * Device errors (into t->err): EINVAL for a sequence whose offsets are out
 * of order or range; it gets no spans.
 */
sm_status sm_match_prompt(const sm_rule_table *t, const int32_t *token_ids,
                          const int32_t *seq_offsets, int B, int total_tokens,
                          int32_t *span_start, int32_t *span_len,
                          int32_t *span_rule, int32_t *seq_span_offsets,
                          void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * sm_match_decode -- the decode-time check after one generated token per
 * listed sequence ("Decoding-time Integration"): the raw-token suffix ending
 * at the new token is looked up for n = 4, 3, 2 in turn (only tokens
 * generated since the sequence's last merge count; a surrogate is never
 * merged again).  On a match the n tokens become one surrogate: k_out = n-1
 * cached entries are to be cropped (the new token has no entry yet) and
 * rule_out = the rule id.  Otherwise k_out = 0, rule_out = -1.
 *  state      [max_seqs][4] int32 per-sequence match state, device-resident:
 *             {raw tokens since the last merge (capped at 3), the last three
 *             of them}; zero it when a sequence starts generating
 *  seq_ids    [n] distinct ids in [0, max_seqs); n <= 1024
 *  new_tokens [n] the generated token of each listed sequence
 *  k_out, rule_out [n] out
 *  cache      (nullable) if given, sm_kv_rollback(cache, seq_ids, k_out, n)
 *             runs right after on the same stream: the crop the merges
 *             imply.  Its device errors go to cache->err; the match state
 *             is updated either way.
 * Device errors (into t->err): EINVAL for a bad or repeated id; then no
 * state changes and every k_out is 0.
 */
sm_status sm_match_decode(const sm_rule_table *t, int32_t *state, int max_seqs,
                          const int32_t *seq_ids, const int32_t *new_tokens,
                          int n, int32_t *k_out, int32_t *rule_out,
                          const sm_paged_cache *cache, hipStream_t stream);

/*
 * Surrogate lookup ("Computational Scope": a span's surrogate depends on its
 * tokens only, so frequently used surrogates can be precomputed and looked
 * up).  A lookup table is any [lut_rows][d] array of surrogates indexed by
 * rule id, for instance sm_merge_spans run once over the rule list.
 *
 * sm_gather_surrogates -- out[i] = lut[rule_ids[i]] if rule_ids[i] >= 0,
 * else emb[token_ids[i]] (a decode step's input: the surrogate of a
 * just-merged suffix or the plain token; or a prompt's span surrogates for
 * sm_pack_spans).  Bit-exact row copies.
 *  emb        [emb_rows][d] embedding table (may be null with token_ids null)
 *  lut        [lut_rows][d] surrogates by rule id
 *  token_ids  [n] nullable: without it every rule id must be >= 0
 *  rule_ids   [n]
 *  d          (host) (d x element bytes) a multiple of 16
 *  out        [n][d] (dtype dt)
 * Device errors: EINVAL for an index out of range; that row is zero.
 */
sm_status sm_gather_surrogates(const void *emb, int64_t emb_rows,
                               const void *lut, int64_t lut_rows,
                               const int32_t *token_ids, const int32_t *rule_ids,
                               int n, int d, sm_dtype dt, void *out,
                               int32_t *err, hipStream_t stream);

/* Workspace of sm_span_dedupe: 4 bytes per rule and per span, plus 512. */
size_t sm_span_dedupe_workspace_bytes(int S, int num_rules);

/*
 * sm_span_dedupe -- spans of one merge batch that carry the same rule share
 * one surrogate.  For spans s = 0..S-1 (e.g. from sm_match_prompt):
 *  uniq_span[u]   the u-th span, in order, whose rule did not occur before
 *                 it (u < *num_uniq)
 *  span_slot[s]   u of the first span with s's rule
 *  uniq_row_idx, uniq_span_offsets [*num_uniq + 1]: the unique spans' token
 *                 ids as CSR rows, the input of sm_merge_spans; then
 *                 sm_gather_surrogates(lut = its output, rule_ids = span_slot)
 *                 gives every span's surrogate.
 *  num_uniq       [1] out (device); the caller reads it to size the merge
 *  span_rule      [S] rule ids in [0, num_rules)
 *  span_start, span_len [S] global token index and length (>= 1) of each span
 *  token_ids      [total_tokens]
 *  uniq_row_idx   capacity: sum of span_len
 * Device errors: EINVAL for a rule id or span range out of bounds; then
 * *num_uniq = 0 and the other outputs are unspecified.
 */
sm_status sm_span_dedupe(const int32_t *span_rule, const int32_t *span_start,
                         const int32_t *span_len, int S, int num_rules,
                         const int32_t *token_ids, int total_tokens,
                         int32_t *uniq_span, int32_t *span_slot,
                         int32_t *uniq_row_idx, int32_t *uniq_span_offsets,
                         int32_t *num_uniq, void *ws, size_t ws_bytes,
                         int32_t *err, hipStream_t stream);

/*
 * The K/V state of one input row per request at its compressed position
 * (appendix "Decoding-time Integration": the frozen backbone processes the
 * surrogate z_s as one input embedding and produces one K/V state for the
 * span).  For the first attention layer, with the RMSNorm gain folded into
 * the projections:
 *
 *   K[i, g] = RoPE_p(W_k RMSNorm(x[i]))[g],  V[i, g] = (W_v RMSNorm(x[i]))[g]
 *   RMSNorm(x) = x / sqrt(mean(x^2) + rms_eps)
 *   p = lengths[seq_ids[i]] when the call starts (the slot the row takes)
 *   RoPE_p: rotate-half; pair (j, j + D/2) of each head turned by the angle
 *           p * rope_theta^(-2j/D)
 */
typedef struct {
  int d;              /* input width: a multiple of 256, at most 16384 */
  const void *W_k;    /* [num_kv_heads * head_dim][d] bf16, row-major (y = W x) */
  const void *W_v;    /* [num_kv_heads * head_dim][d] bf16 */
  float rope_theta;   /* RoPE base, > 0 (Llama 3: 500000) */
  float rms_eps;      /* >= 0 */
} sm_kv_proj_params;

/* Workspace of sm_kv_project / sm_kv_append_projected (about
 * 8 x n x num_kv_heads x head_dim x d / 256 bytes). */
size_t sm_kv_project_workspace_bytes(int n, int d, int num_kv_heads,
                                     int head_dim);

/*
 * sm_kv_project -- K, V [n][num_kv_heads][head_dim] bf16 of the rows
 * x [n][d] bf16 (the step inputs: sm_gather_surrogates' output), for the
 * sequences seq_ids [n] of the bf16 cache c (only their lengths are read;
 * an id outside [0, max_seqs) takes position 0).  n <= min(max_seqs,
 * SM_MAX_REQUESTS); num_kv_heads x head_dim a multiple of 128; x, W_k and
 * W_v 16-byte aligned.  K and V can go to sm_decode_step as its new rows.
 */
sm_status sm_kv_project(const sm_paged_cache *c, const int32_t *seq_ids, int n,
                        const void *x, const sm_kv_proj_params *p, void *K,
                        void *V, void *ws, size_t ws_bytes, hipStream_t stream);

/* sm_kv_append_projected -- sm_kv_project, then sm_kv_append of one row per
 * listed sequence (all of sm_kv_append's checks and errors apply). */
sm_status sm_kv_append_projected(const sm_paged_cache *c, const int32_t *seq_ids,
                                 int n, const void *x, const sm_kv_proj_params *p,
                                 void *ws, size_t ws_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SPANMERGE_H */
