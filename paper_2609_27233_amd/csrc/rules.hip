// Merge-rule matching on the GPU (gfx950).
//
// The rule set R (appendix "Non-overlapping Assignment in a Sequence": the
// 2- to 4-grams kept after the frequency filter, about 2.17M for the
// Llama-3 tokenizer) lives in an open-addressing hash table in HBM.  Each
// slot holds one rule as four int32 token ids (tail -1) and its index in
// the rule list; linear probing, load at most 3/4.
//
//  * Build: one thread per rule claims a slot with a 64-bit compare-and-swap
//    of (fingerprint, rule index + 1).  A thread that meets its own key
//    (same fingerprint, equal tokens read from the immutable rule list)
//    keeps the smaller index with a 64-bit atomic min, so a rule listed
//    twice resolves to its first index.  A second pass copies the keys into
//    the slots.  No thread ever waits on another.
//  * Prompt matching ("Rule Matching": left to right, 4-, 3-, then 2-grams,
//    take the longest match and jump past it, else step one token):
//      1. every position looks up its longest rule (independent lookups);
//      2. per sequence, the greedy chain is a composition of maps: a chunk
//         of positions maps the chain's entry offset (0..3 past the chunk
//         start) to its exit offset, four entries of two bits.  A workgroup
//         scan of these maps gives every chunk its true entry, and each
//         chunk then emits its spans at scanned offsets;
//      3. the sequences' span counts are scanned into CSR offsets and the
//         spans are compacted.
//    The result is exactly the sequential scan's.
//  * Decode matching ("Decoding-time Integration"): per sequence a 16-byte
//    state (number of raw tokens since the last merge, capped at 3, and
//    those tokens) is enough for suffixes of at most 4.  The new token
//    completes the longest rule suffix (4, 3, 2 in turn) or joins the raw
//    tail.  On a match, n - 1 cached entries are to be cropped; the call can
//    run the cache rollback right after.
#include "common.hpp"

typedef int32_t i32x4_t __attribute__((ext_vector_type(4)));

namespace sm {

// MurmurHash3's 64-bit finalizer (Appleby, MurmurHash3, public domain).
__device__ __forceinline__ uint64_t fmix64(uint64_t k) {
  k ^= k >> 33;
  k *= 0xff51afd7ed558ccdull;
  k ^= k >> 33;
  k *= 0xc4ceb9fe1a85ec53ull;
  k ^= k >> 33;
  return k;
}

__device__ __forceinline__ uint64_t rule_hash(i32x4_t k) {
  const uint64_t lo = (uint64_t)(uint32_t)k.x | ((uint64_t)(uint32_t)k.y << 32);
  const uint64_t hi = (uint64_t)(uint32_t)k.z | ((uint64_t)(uint32_t)k.w << 32);
  return fmix64(lo ^ fmix64(hi + 0x9e3779b97f4a7c15ull));
}

__device__ __forceinline__ bool key_eq(i32x4_t a, i32x4_t b) {
  return a.x == b.x && a.y == b.y && a.z == b.z && a.w == b.w;
}

// n of a well-formed rule (n >= 2 leading ids >= 0, then -1), else 0
__device__ __forceinline__ int key_len(i32x4_t k) {
  const int n = k.x < 0 ? 0 : k.y < 0 ? 1 : k.z < 0 ? 2 : k.w < 0 ? 3 : 4;
  const bool tail = (n > 0 || k.x == -1) && (n > 1 || k.y == -1) && (n > 2 || k.z == -1) && (n > 3 || k.w == -1);
  return tail && n >= 2 ? n : 0;
}

// the rule id of key k, or -1; the probe ends at the first empty slot
__device__ __forceinline__ int rule_find(const i32x4_t *keys, const int32_t *ids, uint32_t mask, i32x4_t k) {
  const uint64_t h = rule_hash(k);
  for (uint32_t p = 0; p <= mask; ++p) {
    const uint32_t s = (uint32_t)(h + p) & mask;
    const i32x4_t e = keys[s];
    if (e.x == -1) return -1;
    if (key_eq(e, k)) return ids[s];
  }
  return -1;
}

// The longest of up to three candidate keys (cand[0] the longest) that is a
// rule: the three probe chains advance together, so their memory latencies
// overlap instead of adding up.  want[c] = false skips a candidate.  Returns
// the index of the winning candidate (or -1) and its rule id in *id.
__device__ __forceinline__ int rule_find_longest(const i32x4_t *keys, const int32_t *ids, uint32_t mask,
                                                 const i32x4_t (&cand)[3], const bool (&want)[3], int *id) {
  uint32_t slot[3];
  int state[3];  // -2 probing, -1 absent, else the slot that holds it
#pragma unroll
  for (int c = 0; c < 3; ++c) {
    slot[c] = (uint32_t)rule_hash(cand[c]) & mask;
    state[c] = want[c] ? -2 : -1;
  }
  for (uint32_t p = 0; p <= mask; ++p) {
    i32x4_t e[3];
#pragma unroll
    for (int c = 0; c < 3; ++c)
      if (state[c] == -2) e[c] = keys[slot[c]];
    bool busy = false;
#pragma unroll
    for (int c = 0; c < 3; ++c) {
      if (state[c] != -2) continue;
      if (e[c].x == -1) state[c] = -1;
      else if (key_eq(e[c], cand[c])) state[c] = (int)slot[c];
      else {
        slot[c] = (slot[c] + 1) & mask;
        busy = true;
      }
    }
    if (!busy) break;
  }
#pragma unroll
  for (int c = 0; c < 3; ++c)
    if (state[c] >= 0) {
      *id = ids[state[c]];
      return c;
    }
  *id = -1;
  return -1;
}

// ---- build ----------------------------------------------------------------

__global__ void rules_clear_kernel(uint64_t *claim, int cap) {
  for (int s = blockIdx.x * blockDim.x + threadIdx.x; s < cap; s += gridDim.x * blockDim.x) claim[s] = 0;
}

__global__ void rules_claim_kernel(const i32x4_t *rules, int count, uint64_t *claim, uint32_t mask,
                                   int32_t *err) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= count) return;
  const i32x4_t k = rules[r];
  if (!key_len(k)) {
    set_err(err, SM_ERR_EINVAL);
    return;
  }
  const uint64_t h = rule_hash(k);
  const uint64_t fp = (h >> 32) | 1ull;  // non-zero: an empty slot reads 0
  const uint64_t word = (fp << 32) | (uint32_t)(r + 1);
  for (uint32_t p = 0; p <= mask; ++p) {
    const uint32_t s = (uint32_t)(h + p) & mask;
    const uint64_t old = atomicCAS((unsigned long long *)&claim[s], 0ull, (unsigned long long)word);
    if (old == 0) return;  // claimed
    if ((old >> 32) == fp && key_eq(rules[(uint32_t)old - 1], k)) {
      atomicMin((unsigned long long *)&claim[s], (unsigned long long)word);  // same key: smallest index
      return;
    }
  }
  set_err(err, SM_ERR_ERANGE);  // no free slot (the host keeps the load at most 3/4)
}

__global__ void rules_fill_kernel(const i32x4_t *rules, const uint64_t *claim, int cap, i32x4_t *keys,
                                  int32_t *ids) {
  for (int s = blockIdx.x * blockDim.x + threadIdx.x; s < cap; s += gridDim.x * blockDim.x) {
    const uint64_t w = claim[s];
    if (w == 0) {
      keys[s] = i32x4_t{-1, -1, -1, -1};
      ids[s] = -1;
    } else {
      const int id = (int)(uint32_t)w - 1;
      keys[s] = rules[id];
      ids[s] = id;
    }
  }
}

__global__ void rules_lookup_kernel(const i32x4_t *keys, const int32_t *ids, uint32_t mask, const i32x4_t *grams,
                                    int m, int32_t *out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= m) return;
  const i32x4_t k = grams[i];
  out[i] = key_len(k) ? rule_find(keys, ids, mask, k) : -1;
}

// ---- prompt matching --------------------------------------------------------

// 1. longest rule starting at every position (0 = none) and its id
__global__ void match_len_kernel(const i32x4_t *keys, const int32_t *ids, uint32_t mask, const int32_t *tokens,
                                 const int32_t *seq_offsets, int B, int total, int8_t *mlen, int32_t *rid) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= total) return;
  // the sequence holding t: the last b with seq_offsets[b] <= t
  int lo = 0, hi = B - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (seq_offsets[mid] <= t) lo = mid;
    else hi = mid - 1;
  }
  const int end = min(seq_offsets[lo + 1], total);
  int x[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) x[j] = t + j < end ? tokens[t + j] : -1;
  i32x4_t cand[3];
  bool want[3];
#pragma unroll
  for (int c = 0; c < 3; ++c) {  // candidate c: the (4 - c)-gram at t
    const int n = 4 - c;
    bool ok = t + n <= end;
#pragma unroll
    for (int j = 0; j < 4; ++j) ok = ok && (j >= n || x[j] >= 0);
    want[c] = ok;
    cand[c] = i32x4_t{x[0], x[1], n > 2 ? x[2] : -1, n > 3 ? x[3] : -1};
  }
  int id;
  const int c = rule_find_longest(keys, ids, mask, cand, want, &id);
  const int len = c >= 0 ? 4 - c : 0;
  mlen[t] = (int8_t)len;
  rid[t] = id;
}

constexpr int kSelThreads = 256;
constexpr int kSelChunk = 16;                        // positions per thread
constexpr int kSelSeg = kSelThreads * kSelChunk;     // positions per workgroup pass
constexpr uint32_t kMapIdentity = 0xE4u;             // e -> e, two bits per entry

__device__ __forceinline__ uint32_t map_at(uint32_t f, uint32_t e) { return (f >> (2 * e)) & 3u; }
// g after f
__device__ __forceinline__ uint32_t map_then(uint32_t f, uint32_t g) {
  uint32_t h = 0;
#pragma unroll
  for (uint32_t e = 0; e < 4; ++e) h |= map_at(g, map_at(f, e)) << (2 * e);
  return h;
}

// 2. the greedy chain of one sequence per workgroup; spans go to the
// sequence's own region of the temporary arrays (at its first token)
__global__ __launch_bounds__(kSelThreads) void match_select_kernel(const int8_t *mlen, const int32_t *rid,
                                                                   const int32_t *seq_offsets, int total,
                                                                   int32_t *tmp_start, int32_t *tmp_len,
                                                                   int32_t *tmp_rule, int32_t *count,
                                                                   int32_t *err) {
  __shared__ uint32_t maps[kSelThreads];
  __shared__ int red[16];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int lo = seq_offsets[b], hi = seq_offsets[b + 1];
  if (!(lo >= 0 && lo <= hi && hi <= total)) {
    if (tid == 0) {
      set_err(err, SM_ERR_EINVAL);
      count[b] = 0;
    }
    return;
  }
  const int T = hi - lo;
  int carry = 0, written = 0;
  for (int seg = 0; seg < T; seg += kSelSeg) {
    const int c0 = seg + tid * kSelChunk;  // my chunk [c0, c0 + 16) of the sequence
    // the chunk's match lengths, four bits each: step(p) = length or 1
    uint64_t Lp = 0;
#pragma unroll
    for (int j = 0; j < kSelChunk; ++j)
      Lp |= (uint64_t)(c0 + j < T ? (uint8_t)mlen[lo + c0 + j] : 0u) << (4 * j);
    auto len_at = [&](int p) { return (int)((Lp >> (4 * p)) & 15u); };
    uint32_t f = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      int p = e;
      while (p < kSelChunk) p += max(len_at(p), 1);
      f |= (uint32_t)(p - kSelChunk) << (2 * e);
    }
    // inclusive scan of the maps: thread j gets F_j after ... after F_0
    maps[tid] = f;
    for (int d = 1; d < kSelThreads; d <<= 1) {
      __syncthreads();
      const uint32_t g = tid >= d ? maps[tid - d] : kMapIdentity;
      __syncthreads();
      maps[tid] = map_then(g, maps[tid]);
    }
    __syncthreads();
    const uint32_t before = tid > 0 ? maps[tid - 1] : kMapIdentity;
    const int entry = (int)map_at(before, (uint32_t)carry);
    const int seg_exit = (int)map_at(maps[kSelThreads - 1], (uint32_t)carry);
    // my spans from my true entry
    int k = 0;
    for (int p = entry; p < kSelChunk; p += max(len_at(p), 1)) k += len_at(p) ? 1 : 0;
    int tot;
    const int off = block_inclusive_scan(k, red, &tot) - k;
    int o = lo + written + off;
    for (int p = entry; p < kSelChunk; p += max(len_at(p), 1)) {
      if (len_at(p)) {
        tmp_start[o] = lo + c0 + p;
        tmp_len[o] = len_at(p);
        tmp_rule[o] = rid[lo + c0 + p];
        ++o;
      }
    }
    written += tot;
    carry = seg_exit;
    __syncthreads();  // maps and red are reused by the next pass
  }
  if (tid == 0) count[b] = written;
}

// 3a. CSR offsets of the spans: exclusive scan of the counts (one workgroup)
__global__ __launch_bounds__(kSelThreads) void match_offsets_kernel(const int32_t *count, int B,
                                                                    int32_t *seq_span_offsets) {
  __shared__ int red[16];
  int base = 0;
  for (int b0 = 0; b0 < B; b0 += kSelThreads) {
    const int b = b0 + threadIdx.x;
    const int c = b < B ? count[b] : 0;
    int tot;
    const int inc = block_inclusive_scan(c, red, &tot);
    if (b < B) seq_span_offsets[b] = base + inc - c;
    base += tot;
    __syncthreads();
  }
  if (threadIdx.x == 0) seq_span_offsets[B] = base;
}

// 3b. compaction: sequence b's spans from its region to its CSR range
__global__ __launch_bounds__(kSelThreads) void match_compact_kernel(const int32_t *seq_offsets, const int32_t *count,
                                                                    const int32_t *seq_span_offsets,
                                                                    const int32_t *tmp_start, const int32_t *tmp_len,
                                                                    const int32_t *tmp_rule, int32_t *span_start,
                                                                    int32_t *span_len, int32_t *span_rule) {
  const int b = blockIdx.x;
  const int n = count[b], src = seq_offsets[b], dst = seq_span_offsets[b];
  for (int j = threadIdx.x; j < n; j += kSelThreads) {
    span_start[dst + j] = tmp_start[src + j];
    span_len[dst + j] = tmp_len[src + j];
    span_rule[dst + j] = tmp_rule[src + j];
  }
}

// ---- decode matching --------------------------------------------------------

constexpr int kDecThreads = 1024;  // one request per thread, one workgroup

__global__ __launch_bounds__(kDecThreads) void match_decode_kernel(const i32x4_t *keys, const int32_t *ids,
                                                                   uint32_t mask, i32x4_t *state, int max_seqs,
                                                                   const int32_t *seq_ids,
                                                                   const int32_t *new_tokens, int n,
                                                                   int32_t *k_out, int32_t *rule_out,
                                                                   int32_t *err) {
  __shared__ int sid[kDecThreads];
  __shared__ int bad;
  const int i = threadIdx.x;
  const int s = i < n ? seq_ids[i] : -1;
  sid[i] = s;
  if (i == 0) bad = 0;
  __syncthreads();
  if (i < n) {
    bool ok = s >= 0 && s < max_seqs;
    for (int j = 0; j < i && ok; ++j) ok = sid[j] != s;
    if (!ok) bad = 1;
  }
  __syncthreads();
  if (i >= n) return;
  if (bad) {  // nothing changes: no state update, no crop
    if (i == 0) set_err(err, SM_ERR_EINVAL);
    k_out[i] = 0;
    rule_out[i] = -1;
    return;
  }
  const i32x4_t st = state[s];
  const int r = min(max(st.x, 0), 3);  // raw tokens since the last merge, at most 3 kept
  const int w[4] = {st.y, st.z, st.w, new_tokens[i]};
  i32x4_t cand[3];
  bool want[3];
#pragma unroll
  for (int c = 0; c < 3; ++c) {  // candidate c: the suffix of m = 4 - c tokens
    const int m = 4 - c;
    bool ok = m <= r + 1;
#pragma unroll
    for (int j = 0; j < 4; ++j) ok = ok && (j < 4 - m || w[j] >= 0);
    want[c] = ok;
    cand[c] = i32x4_t{w[4 - m], w[5 - m], m > 2 ? w[6 - m] : -1, m > 3 ? w[3] : -1};
  }
  int id;
  const int c = rule_find_longest(keys, ids, mask, cand, want, &id);
  const int k = c >= 0 ? 3 - c : 0;  // n - 1 entries to crop
  state[s] = id >= 0 ? i32x4_t{0, -1, -1, -1} : i32x4_t{min(r + 1, 3), w[1], w[2], w[3]};
  k_out[i] = k;
  rule_out[i] = id;
}

static bool table_ok(const sm_rule_table *t) {
  return t && t->keys && t->ids && t->err && t->capacity >= 16 && (t->capacity & (t->capacity - 1)) == 0;
}

}  // namespace sm

using namespace sm;

SM_API size_t sm_rules_build_workspace_bytes(int capacity) {
  return capacity > 0 ? (size_t)capacity * sizeof(uint64_t) : 0;
}

SM_API sm_status sm_rules_build(const int32_t *rules, int count, const sm_rule_table *t, void *ws, size_t ws_bytes,
                                hipStream_t stream) {
  if (!table_ok(t) || count < 0 || (int64_t)count * 4 > (int64_t)t->capacity * 3) return SM_EINVAL;
  if (!ws || ws_bytes < sm_rules_build_workspace_bytes(t->capacity) || (count > 0 && !rules)) return SM_EINVAL;
  uint64_t *claim = (uint64_t *)ws;
  const int cap = t->capacity;
  const int grid = min((cap + 255) / 256, 4096);
  hipLaunchKernelGGL(rules_clear_kernel, dim3(grid), dim3(256), 0, stream, claim, cap);
  if (count > 0)
    hipLaunchKernelGGL(rules_claim_kernel, dim3((count + 255) / 256), dim3(256), 0, stream, (const i32x4_t *)rules,
                       count, claim, (uint32_t)(cap - 1), t->err);
  hipLaunchKernelGGL(rules_fill_kernel, dim3(grid), dim3(256), 0, stream, (const i32x4_t *)rules, claim, cap,
                     (i32x4_t *)t->keys, t->ids);
  return hipGetLastError() == hipSuccess ? SM_OK : SM_EHIP;
}

SM_API sm_status sm_rules_lookup(const sm_rule_table *t, const int32_t *grams, int m, int32_t *ids,
                                 hipStream_t stream) {
  if (!table_ok(t) || m < 0) return SM_EINVAL;
  if (m == 0) return SM_OK;
  if (!grams || !ids) return SM_EINVAL;
  hipLaunchKernelGGL(rules_lookup_kernel, dim3((m + 255) / 256), dim3(256), 0, stream, (const i32x4_t *)t->keys,
                     t->ids, (uint32_t)(t->capacity - 1), (const i32x4_t *)grams, m, ids);
  return hipGetLastError() == hipSuccess ? SM_OK : SM_EHIP;
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

SM_API size_t sm_match_prompt_workspace_bytes(int B, int total_tokens) {
  if (B < 0 || total_tokens < 0) return 0;
  const size_t T = (size_t)total_tokens;
  return align256(T) + 4 * align256(4 * T) + align256(4 * (size_t)B + 4);
}

SM_API sm_status sm_match_prompt(const sm_rule_table *t, const int32_t *token_ids, const int32_t *seq_offsets,
                                 int B, int total_tokens, int32_t *span_start, int32_t *span_len,
                                 int32_t *span_rule, int32_t *seq_span_offsets, void *ws, size_t ws_bytes,
                                 hipStream_t stream) {
  if (!table_ok(t) || B < 0 || total_tokens < 0 || B > 65535) return SM_EINVAL;
  if (!seq_offsets || !seq_span_offsets || (total_tokens > 0 && (!token_ids || !span_start || !span_len ||
                                                                  !span_rule)))
    return SM_EINVAL;
  if (!ws || ws_bytes < sm_match_prompt_workspace_bytes(B, total_tokens)) return SM_EINVAL;
  const size_t T = (size_t)total_tokens;
  char *p = (char *)ws;
  int8_t *mlen = (int8_t *)p;
  p += align256(T);
  int32_t *rid = (int32_t *)p;
  p += align256(4 * T);
  int32_t *tmp_start = (int32_t *)p;
  p += align256(4 * T);
  int32_t *tmp_len = (int32_t *)p;
  p += align256(4 * T);
  int32_t *tmp_rule = (int32_t *)p;
  p += align256(4 * T);
  int32_t *count = (int32_t *)p;
  const uint32_t mask = (uint32_t)(t->capacity - 1);
  if (B > 0 && total_tokens > 0)
    hipLaunchKernelGGL(match_len_kernel, dim3((total_tokens + 255) / 256), dim3(256), 0, stream,
                       (const i32x4_t *)t->keys, t->ids, mask, token_ids, seq_offsets, B, total_tokens, mlen, rid);
  if (B > 0)
    hipLaunchKernelGGL(match_select_kernel, dim3(B), dim3(kSelThreads), 0, stream, mlen, rid, seq_offsets,
                       total_tokens, tmp_start, tmp_len, tmp_rule, count, t->err);
  hipLaunchKernelGGL(match_offsets_kernel, dim3(1), dim3(kSelThreads), 0, stream, count, B, seq_span_offsets);
  if (B > 0)
    hipLaunchKernelGGL(match_compact_kernel, dim3(B), dim3(kSelThreads), 0, stream, seq_offsets, count,
                       seq_span_offsets, tmp_start, tmp_len, tmp_rule, span_start, span_len, span_rule);
  return hipGetLastError() == hipSuccess ? SM_OK : SM_EHIP;
}

SM_API sm_status sm_match_decode(const sm_rule_table *t, int32_t *state, int max_seqs, const int32_t *seq_ids,
                                 const int32_t *new_tokens, int n, int32_t *k_out, int32_t *rule_out,
                                 const sm_paged_cache *cache, hipStream_t stream) {
  if (!table_ok(t) || n < 0 || n > kDecThreads || max_seqs <= 0) return SM_EINVAL;
  if (cache) {  // the rollback's own synchronous checks, before anything is enqueued
    if (sm_kv_rollback(cache, seq_ids, k_out, 0, stream) != SM_OK || n > cache->max_seqs || n > SM_MAX_REQUESTS)
      return SM_EINVAL;
  }
  if (n == 0) return SM_OK;
  if (!state || !seq_ids || !new_tokens || !k_out || !rule_out) return SM_EINVAL;
  hipLaunchKernelGGL(match_decode_kernel, dim3(1), dim3(kDecThreads), 0, stream, (const i32x4_t *)t->keys, t->ids,
                     (uint32_t)(t->capacity - 1), (i32x4_t *)state, max_seqs, seq_ids, new_tokens, n, k_out,
                     rule_out, t->err);
  if (hipGetLastError() != hipSuccess) return SM_EHIP;
  return cache ? sm_kv_rollback(cache, seq_ids, k_out, n, stream) : SM_OK;
}
