// Paged KV-cache bookkeeping for span merging (gfx950):
//   kv_rollback  crop k entries per sequence (decoding-time merge, the paper's
//                "crop the n-1 cached entries" step); metadata only
//   kv_append    append K/V rows (the surrogate's single state, a decode
//                token, or a whole compressed prompt)
//   pack_spans   keep mask -> compressed positions -> packed rows (prompt
//                merging, "Prompt-time Integration")
//
// Metadata kernels run as ONE workgroup of 1024 threads: every request is
// validated first (all-or-nothing), then block ids move between the block
// table and the LIFO free stack at positions fixed by prefix sums, so the
// result is deterministic and identical to the sequential definition
// (rollback pushes in reverse request order, highest logical block first;
// append pops in request order, lowest logical block first).
#include "common.hpp"

namespace sm {

struct CacheArgs {
  void *k_pool;
  void *v_pool;
  int32_t *block_table;
  int32_t *lengths;
  int32_t *free_stack;
  int32_t *free_top;
  int32_t *err;
  int Hkv, DH, dh_log2, bs_log2, num_blocks, max_seqs, max_blocks;
};

constexpr int kMetaThreads = 1024;

__device__ __forceinline__ int blocks_for(int len, int bs_log2) {
  return (len + (1 << bs_log2) - 1) >> bs_log2;
}

// Distinct, in-range sequence ids; thread t checks request t against all
// earlier requests.
__device__ __forceinline__ bool id_ok(const int32_t *seq_ids, int t, int s, int max_seqs) {
  if (s < 0 || s >= max_seqs) return false;
  for (int j = 0; j < t; ++j)
    if (seq_ids[j] == s) return false;
  return true;
}

__global__ __launch_bounds__(kMetaThreads) void rollback_kernel(CacheArgs c, const int32_t *seq_ids,
                                                                 const int32_t *ks, int n) {
  __shared__ int red[16];
  __shared__ int fl_inval, fl_range, s_err, s_top;
  const int t = threadIdx.x;
  if (t == 0) {
    fl_inval = 0;
    fl_range = 0;
    s_err = *c.err;
    s_top = *c.free_top;
  }
  __syncthreads();
  if (s_err != 0) return;  // sticky: the cache is frozen until the caller clears err

  const bool active = t < n;
  int s = 0, k = 0;
  if (active) {
    s = seq_ids[t];
    k = ks[t];
    if (k < 0 || !id_ok(seq_ids, t, s, c.max_seqs)) fl_inval = 1;
  }
  __syncthreads();
  if (fl_inval) {
    if (t == 0) set_err(c.err, SM_ERR_EINVAL);
    return;
  }
  const int cap = c.max_blocks << c.bs_log2;
  int L = 0, freed = 0;
  if (active) {
    L = c.lengths[s];
    if (L < 0 || L > cap || k > L) fl_range = 1;
    else freed = blocks_for(L, c.bs_log2) - blocks_for(L - k, c.bs_log2);
  }
  __syncthreads();
  if (fl_range) {
    if (t == 0) set_err(c.err, SM_ERR_ERANGE);
    return;
  }
  int total;
  const int incl = block_inclusive_scan(freed, red, &total);
  const int top = s_top;
  if (top < 0 || (int64_t)top + total > c.num_blocks) {  // stack cannot take the blocks
    if (t == 0) set_err(c.err, SM_ERR_ERANGE);
    return;
  }
  if (active) {
    // requests are served in reverse order: request t's first push lands
    // above the blocks of every later request
    int pos = top + (total - incl);
    int32_t *row = c.block_table + (int64_t)s * c.max_blocks;
    const int nb_old = blocks_for(L, c.bs_log2), nb_new = blocks_for(L - k, c.bs_log2);
    for (int j = nb_old - 1; j >= nb_new; --j) {
      c.free_stack[pos++] = row[j];
      row[j] = -1;
    }
    c.lengths[s] = L - k;
  }
  if (t == 0) *c.free_top = top + total;
}

// Validation and block allocation of kv_append, run by one workgroup of
// kMetaThreads threads (thread t owns request t).  Returns true, uniformly
// across the workgroup, when the call was applied; on return *L_old holds
// request t's length before the call.
struct AppendShared {
  int red[16];
  int fl_inval, fl_range, fl_stack, s_err, s_top;
};

__device__ bool append_meta_body(const CacheArgs &c, const int32_t *seq_ids, const int32_t *row_offsets, int n,
                                 int total_rows, AppendShared &sh, int &s_out, int &L_old) {
  const int t = threadIdx.x;
  if (t == 0) {
    sh.fl_inval = 0;
    sh.fl_range = 0;
    sh.fl_stack = 0;
    sh.s_err = *c.err;
    sh.s_top = *c.free_top;
    if (row_offsets[0] != 0 || row_offsets[n] != total_rows) sh.fl_inval = 1;
  }
  __syncthreads();
  if (sh.s_err != 0) return false;  // sticky: the cache is frozen

  const bool active = t < n;
  int s = 0, m = 0;
  if (active) {
    s = seq_ids[t];
    m = row_offsets[t + 1] - row_offsets[t];
    if (m < 0 || !id_ok(seq_ids, t, s, c.max_seqs)) sh.fl_inval = 1;
  }
  __syncthreads();
  if (sh.fl_inval) {
    if (t == 0) set_err(c.err, SM_ERR_EINVAL);
    return false;
  }
  const int cap = c.max_blocks << c.bs_log2;
  int L = 0, need = 0;
  if (active) {
    L = c.lengths[s];
    if (L < 0 || (int64_t)L + m > cap) sh.fl_range = 1;
    else need = blocks_for(L + m, c.bs_log2) - blocks_for(L, c.bs_log2);
  }
  __syncthreads();
  if (sh.fl_range) {
    if (t == 0) set_err(c.err, SM_ERR_ERANGE);
    return false;
  }
  int total;
  const int incl = block_inclusive_scan(need, sh.red, &total);
  const int top = sh.s_top;
  if (top < 0 || top > c.num_blocks || total > top) {
    if (t == 0) set_err(c.err, SM_ERR_ENOMEM);
    return false;
  }
  // every id about to be popped must name a real block
  for (int j = t; j < total; j += blockDim.x) {
    const int blk = c.free_stack[top - 1 - j];
    if (blk < 0 || blk >= c.num_blocks) sh.fl_stack = 1;
  }
  __syncthreads();
  if (sh.fl_stack) {
    if (t == 0) set_err(c.err, SM_ERR_EINVAL);
    return false;
  }
  if (active) {
    int32_t *row = c.block_table + (int64_t)s * c.max_blocks;
    const int first = blocks_for(L, c.bs_log2);
    const int pop0 = incl - need;  // pops already taken by earlier requests
    for (int q = 0; q < need; ++q) row[first + q] = c.free_stack[top - 1 - (pop0 + q)];
    c.lengths[s] = L + m;
  }
  if (t == 0) *c.free_top = top - total;
  s_out = s;
  L_old = L;
  return true;
}

__global__ __launch_bounds__(kMetaThreads) void append_meta_kernel(CacheArgs c, const int32_t *seq_ids,
                                                                    const int32_t *row_offsets, int n,
                                                                    int total_rows) {
  __shared__ AppendShared sh;
  int s, L;
  append_meta_body(c, seq_ids, row_offsets, n, total_rows, sh, s, L);
}

// Copy rows [r_begin, r_end) of K and V into their slots; row_blk/row_slot
// (LDS) give the destination of row r - r_begin (block -1: skip).  One unit
// = one 16-byte group of one row (VEC elements of one head); `upr` divides
// by the units per row.  Threads `lane0`, lane0 + stride, ... share the
// units; each unit's K and V loads are issued before its stores.
template <typename T>
__device__ __forceinline__ void copy_rows(const CacheArgs &c, const T *__restrict__ K, const T *__restrict__ V,
                                          int r_begin, int r_end, const FastDiv &upr, const int *row_blk,
                                          const int *row_slot, int lane0, int stride) {
  constexpr int VEC = 16 / sizeof(T);
  const int bs = 1 << c.bs_log2;
  const int gpl2 = c.dh_log2 - (sizeof(T) == 2 ? 3 : 2);  // log2(groups per head)
  const int row_elems = c.Hkv << c.dh_log2;
  const int units = (r_end - r_begin) * (int)upr.d;
  T *kp = (T *)c.k_pool;
  T *vp = (T *)c.v_pool;
  for (int u = lane0; u < units; u += stride) {
    const int rr = (int)fdiv((uint32_t)u, upr);
    const int gi = u - rr * (int)upr.d;           // group within the row
    const int g = gi >> gpl2, d0 = (gi & ((1 << gpl2) - 1)) * VEC;
    const int64_t src = (int64_t)(r_begin + rr) * row_elems + (int64_t)gi * VEC;
    const u32x4_t kv = *(const u32x4_t *)(K + src);
    const u32x4_t vv = *(const u32x4_t *)(V + src);
    const int blk = row_blk[rr];
    if (blk < 0) continue;
    const int slot = row_slot[rr];
    *(u32x4_t *)(kp + (((int64_t)blk * c.Hkv + g) * bs + slot) * c.DH + d0) = kv;
    T *vdst = vp + (((int64_t)blk * c.Hkv + g) * c.DH + d0) * bs + slot;
    const T *ve = (const T *)&vv;
#pragma unroll
    for (int e = 0; e < VEC; ++e) vdst[e * bs] = ve[e];
  }
}

// Small appends (a decode step: one row per sequence) in ONE workgroup,
// metadata and copy together.  The sequence of dependent global accesses is
// kept short: (1) ids / offsets / error word, (2) lengths, (3) the tail
// block of each sequence and the popped free-stack entries, (4) the row
// copies.  Same validation order and block order as the two-kernel path.
constexpr int kSmallBytes = 64 * 1024;  // of K (and of V) per call
constexpr int kSmallRows = 1024;

template <typename T>
__global__ __launch_bounds__(kMetaThreads) void append_small_kernel(CacheArgs c, const int32_t *seq_ids,
                                                                     const int32_t *row_offsets, int n,
                                                                     int total_rows, const T *__restrict__ K,
                                                                     const T *__restrict__ V, FastDiv upr) {
  __shared__ int red[16];
  __shared__ int ids[kMetaThreads];
  __shared__ int fl_inval, fl_range, fl_stack, s_err, s_top;
  __shared__ int row_blk[kSmallRows], row_slot[kSmallRows];
  const int t = threadIdx.x;
  const bool active = t < n;
  // (1)
  int s = -1, r0 = 0, r1 = 0;
  if (active) {
    s = seq_ids[t];
    r0 = row_offsets[t];
    r1 = row_offsets[t + 1];
    ids[t] = s;
  }
  if (t == 0) {
    fl_range = 0;
    fl_stack = 0;
    s_err = *c.err;
    s_top = *c.free_top;
    fl_inval = (row_offsets[0] != 0 || row_offsets[n] != total_rows);
  }
  __syncthreads();
  if (s_err != 0) return;  // sticky: the cache is frozen
  if (active) {
    bool ok = r1 >= r0 && s >= 0 && s < c.max_seqs;
    for (int j = 0; j < t && ok; ++j) ok = ids[j] != s;
    if (!ok) fl_inval = 1;
  }
  __syncthreads();
  if (fl_inval) {
    if (t == 0) set_err(c.err, SM_ERR_EINVAL);
    return;
  }
  // (2)
  const int m = r1 - r0;
  const int cap = c.max_blocks << c.bs_log2;
  int L = 0, need = 0;
  if (active) {
    L = c.lengths[s];
    if (L < 0 || (int64_t)L + m > cap) fl_range = 1;
    else need = blocks_for(L + m, c.bs_log2) - blocks_for(L, c.bs_log2);
  }
  __syncthreads();
  if (fl_range) {
    if (t == 0) set_err(c.err, SM_ERR_ERANGE);
    return;
  }
  int total;
  const int incl = block_inclusive_scan(need, red, &total);
  const int top = s_top;
  if (top < 0 || top > c.num_blocks || total > top) {
    if (t == 0) set_err(c.err, SM_ERR_ENOMEM);
    return;
  }
  // (3) every popped id must name a real block; the partially filled tail
  // block (if a new row lands in it) is read once
  for (int j = t; j < total; j += kMetaThreads) {
    const int blk = c.free_stack[top - 1 - j];
    if (blk < 0 || blk >= c.num_blocks) fl_stack = 1;
  }
  int32_t *brow = c.block_table + (int64_t)(active ? s : 0) * c.max_blocks;
  const int first = blocks_for(L, c.bs_log2);  // first logical block to allocate
  const int lp_tail = L >> c.bs_log2;           // page of the first new row
  const int tail_blk = (active && m > 0 && lp_tail < first) ? brow[lp_tail] : -1;
  __syncthreads();
  if (fl_stack) {
    if (t == 0) set_err(c.err, SM_ERR_EINVAL);
    return;
  }
  const int bs = 1 << c.bs_log2;
  if (active) {
    const int pop0 = incl - need;  // pops already taken by earlier requests
    for (int q = 0; q < need; ++q) brow[first + q] = c.free_stack[top - 1 - (pop0 + q)];
    c.lengths[s] = L + m;
    for (int r = r0; r < r1; ++r) {
      const int pos = L + (r - r0);
      const int lp = pos >> c.bs_log2;
      const int b = (lp < first) ? tail_blk : c.free_stack[top - 1 - (pop0 + lp - first)];
      const bool ok = b >= 0 && b < c.num_blocks;
      if (!ok) set_err(c.err, SM_ERR_EINVAL);  // corrupt block table
      row_blk[r] = ok ? b : -1;
      row_slot[r] = pos & (bs - 1);
    }
  }
  if (t == 0) *c.free_top = top - total;
  __syncthreads();
  // (4) the copy, in units of one 16-byte group of one row: the K group
  // goes to its token-major page with one 16-byte store, the V group's
  // elements go to the dim-major page one slot at a time
  copy_rows<T>(c, K, V, 0, total_rows, upr, row_blk, row_slot, t, kMetaThreads);
}

// Copy phase of kv_append: 16 consecutive input rows per workgroup.  K rows
// go to token-major pages with 16-byte stores; V rows are staged in LDS and
// written transposed into the dim-major V pages, consecutive threads taking
// consecutive slots.
constexpr int kCopyRows = 16;
constexpr int kCopyThreads = 256;
constexpr int kMaxRowElems = 2048;  // num_kv_heads * head_dim

template <typename T>
__global__ __launch_bounds__(kCopyThreads) void append_copy_kernel(CacheArgs c, const int32_t *seq_ids,
                                                                   const int32_t *row_offsets, int n,
                                                                   int total_rows, const T *__restrict__ K,
                                                                   const T *__restrict__ V) {
  extern __shared__ unsigned char smem_raw[];
  T *vs = reinterpret_cast<T *>(smem_raw);  // [kCopyRows][row_elems + pad]
  __shared__ int row_blk[kCopyRows], row_slot[kCopyRows];
  __shared__ int s_err;
  const int t = threadIdx.x;
  if (t == 0) s_err = *c.err;
  __syncthreads();
  if (s_err != 0) return;  // the metadata pass failed (or an earlier call did)

  const int r0 = blockIdx.x * kCopyRows;
  const int bs = 1 << c.bs_log2;
  if (t < kCopyRows) {
    const int r = r0 + t;
    int blk = -1, slot = 0;
    if (r < total_rows) {
      int lo = 0, hi = n - 1;  // request i with row_offsets[i] <= r < row_offsets[i+1]
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (row_offsets[mid] <= r) lo = mid;
        else hi = mid - 1;
      }
      const int s = seq_ids[lo];
      const int m = row_offsets[lo + 1] - row_offsets[lo];
      const int pos = c.lengths[s] - m + (r - row_offsets[lo]);  // lengths already advanced
      const int b = c.block_table[(int64_t)s * c.max_blocks + (pos >> c.bs_log2)];
      if (b < 0 || b >= c.num_blocks) set_err(c.err, SM_ERR_EINVAL);
      else {
        blk = b;
        slot = pos & (bs - 1);
      }
    }
    row_blk[t] = blk;
    row_slot[t] = slot;
  }
  const int row_elems = c.Hkv * c.DH;
  const int pitch = row_elems + 4;
  constexpr int VEC = 16 / sizeof(T);
  const int vpr = row_elems / VEC;  // 16-byte vectors per row
  const int nrows = min(kCopyRows, total_rows - r0);
  // stage V rows (coalesced)
  for (int e = t; e < nrows * vpr; e += kCopyThreads) {
    const int rr = e / vpr, cc = (e - rr * vpr) * VEC;
    const T *src = V + (int64_t)(r0 + rr) * row_elems + cc;
#pragma unroll
    for (int u = 0; u < VEC; ++u) vs[rr * pitch + cc + u] = src[u];
  }
  __syncthreads();
  // K rows: 16-byte vector copies into token-major pages, all loads of a
  // thread issued before its stores
  T *kp = (T *)c.k_pool;
  constexpr int KP = kCopyRows * (kMaxRowElems / VEC) / kCopyThreads;
  u32x4_t kr[KP];
#pragma unroll
  for (int u = 0; u < KP; ++u) {
    const int e = t + u * kCopyThreads;
    if (e < nrows * vpr) {
      const int rr = e / vpr, cc = (e - rr * vpr) * VEC;
      kr[u] = *(const u32x4_t *)(K + (int64_t)(r0 + rr) * row_elems + cc);
    }
  }
#pragma unroll
  for (int u = 0; u < KP; ++u) {
    const int e = t + u * kCopyThreads;
    if (e < nrows * vpr) {
      const int rr = e / vpr, cc = (e - rr * vpr) * VEC;
      const int blk = row_blk[rr];
      if (blk < 0) continue;
      const int g = cc / c.DH, d = cc - g * c.DH;
      *(u32x4_t *)(kp + (((int64_t)blk * c.Hkv + g) * bs + row_slot[rr]) * c.DH + d) = kr[u];
    }
  }
  // V rows: transposed element stores, slot (row) fastest
  T *vp = (T *)c.v_pool;
  for (int e = t; e < nrows * row_elems; e += kCopyThreads) {
    const int gd = e / nrows, rr = e - gd * nrows;
    const int blk = row_blk[rr];
    if (blk < 0) continue;
    const int g = gd / c.DH, d = gd - g * c.DH;
    vp[(((int64_t)blk * c.Hkv + g) * c.DH + d) * bs + row_slot[rr]] = vs[rr * pitch + gd];
  }
}

// ---------------------------------------------------------------------------
// pack_spans

constexpr int kPackThreads = 1024;
constexpr int kPackChunk = 4096;  // tokens per LDS pass
constexpr int kRemoved = INT32_MIN;

struct PackArgs {
  int B, total_tokens, num_spans;
  const int32_t *seq_offsets, *span_start, *span_len, *seq_span_offsets;
  int32_t *pi, *packed_offsets, *packed_src;
  const int32_t *token_ids;
  const void *emb;
  int64_t emb_rows;
  const void *surrogates;
  int d;
  void *packed;
  int32_t *err;
};

// Every workgroup validates the whole span list (cheap) so that no
// workgroup writes with offsets computed from invalid input.
__device__ bool pack_inputs_valid(const PackArgs &a, int *flag) {
  const int t = threadIdx.x;
  if (t == 0) {
    *flag = 0;
    if (a.seq_offsets[0] != 0 || a.seq_offsets[a.B] != a.total_tokens ||
        a.seq_span_offsets[0] != 0 || a.seq_span_offsets[a.B] != a.num_spans)
      *flag = 1;
  }
  __syncthreads();
  for (int b = t; b < a.B; b += blockDim.x)
    if (a.seq_offsets[b + 1] < a.seq_offsets[b] || a.seq_span_offsets[b + 1] < a.seq_span_offsets[b])
      *flag = 1;
  __syncthreads();
  if (*flag) return false;
  for (int s = t; s < a.num_spans; s += blockDim.x) {
    int lo = 0, hi = a.B - 1;  // sequence b with sso[b] <= s < sso[b+1]
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (a.seq_span_offsets[mid] <= s) lo = mid;
      else hi = mid - 1;
    }
    const int st = a.span_start[s], ln = a.span_len[s];
    bool ok = ln >= 1 && st >= a.seq_offsets[lo] && (int64_t)st + ln <= a.seq_offsets[lo + 1];
    if (ok && s > a.seq_span_offsets[lo]) ok = st >= a.span_start[s - 1] + a.span_len[s - 1];
    if (!ok) *flag = 1;
  }
  __syncthreads();
  return *flag == 0;
}

__global__ __launch_bounds__(kPackThreads) void pack_index_kernel(PackArgs a) {
  __shared__ int src[kPackChunk];
  __shared__ int red[16];
  __shared__ int flag, s_err;
  __shared__ float fred[16];
  const int b = blockIdx.x, t = threadIdx.x;
  if (t == 0) s_err = *a.err;
  __syncthreads();
  if (s_err != 0) return;
  if (!pack_inputs_valid(a, &flag)) {
    if (b == 0 && t == 0) set_err(a.err, SM_ERR_EINVAL);
    return;
  }
  const int sp0 = a.seq_span_offsets[b], sp1 = a.seq_span_offsets[b + 1];
  // positions removed before this sequence (and in total, for the last one)
  int removed_before = 0, removed_all = 0;
  for (int s = t; s < a.num_spans; s += kPackThreads) {
    const int r = a.span_len[s] - 1;
    removed_all += r;
    if (s < sp0) removed_before += r;
  }
  int dummy;
  // block sums via the scan helper (totals only)
  block_inclusive_scan(removed_before, red, &removed_before);
  __syncthreads();
  block_inclusive_scan(removed_all, red, &removed_all);
  (void)dummy;
  (void)fred;
  const int base = a.seq_offsets[b] - removed_before;  // packed_offsets[b]
  if (t == 0) {
    a.packed_offsets[b] = base;
    if (b == a.B - 1) a.packed_offsets[a.B] = a.total_tokens - removed_all;
  }
  const int q0 = a.seq_offsets[b], q1 = a.seq_offsets[b + 1];
  int carry = 0;
  for (int c0 = q0; c0 < q1; c0 += kPackChunk) {
    const int cn = min(kPackChunk, q1 - c0);
    __syncthreads();
    for (int e = t; e < cn; e += kPackThreads) src[e] = c0 + e;
    __syncthreads();
    for (int s = sp0 + t; s < sp1; s += kPackThreads) {
      const int st = a.span_start[s], last = st + a.span_len[s] - 1;
      if (last < c0 || st >= c0 + cn) continue;
      for (int u = max(st, c0); u < min(last, c0 + cn); ++u) src[u - c0] = kRemoved;
      if (last < c0 + cn) src[last - c0] = -1 - s;
    }
    __syncthreads();
    // each thread owns 4 consecutive tokens of the chunk
    const int e0 = 4 * t;
    int keep[4], cnt = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      keep[u] = (e0 + u < cn) && src[e0 + u] != kRemoved;
      cnt += keep[u];
    }
    int tot;
    const int incl = block_inclusive_scan(cnt, red, &tot);
    int pos = carry + incl - cnt;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (e0 + u >= cn) break;
      a.pi[c0 + e0 + u] = pos;
      if (keep[u]) a.packed_src[base + pos++] = src[e0 + u];
    }
    carry += tot;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void pack_rows_kernel(PackArgs a) {
  __shared__ int s_err;
  if (threadIdx.x == 0) s_err = *a.err;
  __syncthreads();
  if (s_err != 0) return;
  const int nrows = a.packed_offsets[a.B];
  constexpr int VEC = 16 / sizeof(T);
  const int vpr = a.d / VEC;
  for (int r = blockIdx.x; r < nrows; r += gridDim.x) {
    const int src = a.packed_src[r];
    const T *row;
    if (src >= 0) {
      const int tok = a.token_ids[src];
      if (tok < 0 || tok >= a.emb_rows) {
        if (threadIdx.x == 0) set_err(a.err, SM_ERR_EINVAL);
        continue;
      }
      row = (const T *)a.emb + (int64_t)tok * a.d;
    } else {
      row = (const T *)a.surrogates + (int64_t)(-1 - src) * a.d;
    }
    T *dst = (T *)a.packed + (int64_t)r * a.d;
    for (int v = threadIdx.x; v < vpr; v += blockDim.x)
      *(u32x4_t *)(dst + v * VEC) = *(const u32x4_t *)(row + v * VEC);
  }
}

}  // namespace sm

using namespace sm;

static int ilog2_pow2(int v) {
  if (v <= 0 || (v & (v - 1))) return -1;
  int l = 0;
  while ((1 << l) < v) ++l;
  return l;
}

static bool cache_ok(const sm_paged_cache *c, CacheArgs &a) {
  if (!c) return false;
  if (c->dtype != SM_F32 && c->dtype != SM_BF16) return false;
  if (c->head_dim != 64 && c->head_dim != 128) return false;
  const int l = ilog2_pow2(c->block_size);
  if (l < 4 || l > 9) return false;
  if (c->num_kv_heads <= 0 || c->num_blocks <= 0 || c->max_seqs <= 0 || c->max_blocks_per_seq <= 0)
    return false;
  if ((int64_t)c->max_blocks_per_seq * c->block_size > INT32_MAX / 2) return false;
  if (!c->k_pool || !c->v_pool || !c->block_table || !c->lengths || !c->free_stack || !c->free_top ||
      !c->err)
    return false;
  a.k_pool = c->k_pool;
  a.v_pool = c->v_pool;
  a.block_table = c->block_table;
  a.lengths = c->lengths;
  a.free_stack = c->free_stack;
  a.free_top = c->free_top;
  a.err = c->err;
  a.Hkv = c->num_kv_heads;
  a.DH = c->head_dim;
  a.dh_log2 = c->head_dim == 128 ? 7 : 6;
  a.bs_log2 = l;
  a.num_blocks = c->num_blocks;
  a.max_seqs = c->max_seqs;
  a.max_blocks = c->max_blocks_per_seq;
  return true;
}

SM_API sm_status sm_kv_rollback(const sm_paged_cache *c, const int32_t *seq_ids, const int32_t *k, int n,
                                hipStream_t stream) {
  CacheArgs a;
  if (!cache_ok(c, a) || n < 0 || n > SM_MAX_REQUESTS || n > c->max_seqs) return SM_EINVAL;
  if (n == 0) return SM_OK;
  if (!seq_ids || !k) return SM_EINVAL;
  hipLaunchKernelGGL(rollback_kernel, dim3(1), dim3(kMetaThreads), 0, stream, a, seq_ids, k, n);
  return hipGetLastError() == hipSuccess ? SM_OK : SM_EHIP;
}

SM_API sm_status sm_kv_append(const sm_paged_cache *c, const int32_t *seq_ids, const int32_t *row_offsets,
                              int n, int total_rows, const void *K, const void *V, hipStream_t stream) {
  CacheArgs a;
  if (!cache_ok(c, a) || n < 0 || n > SM_MAX_REQUESTS || n > c->max_seqs || total_rows < 0)
    return SM_EINVAL;
  if (n == 0) return total_rows == 0 ? SM_OK : SM_EINVAL;
  if (!seq_ids || !row_offsets || (total_rows > 0 && (!K || !V))) return SM_EINVAL;
  const size_t es = c->dtype == SM_BF16 ? 2 : 4;
  const size_t lds = (size_t)kCopyRows * (c->num_kv_heads * c->head_dim + 4) * es;
  if (lds > 64 * 1024 || c->num_kv_heads * c->head_dim > kMaxRowElems) return SM_EINVAL;
  const size_t tensor_bytes = (size_t)total_rows * c->num_kv_heads * c->head_dim * es;
  const FastDiv upr = make_fastdiv((uint32_t)(c->num_kv_heads * c->head_dim * es / 16));
  if (total_rows > 0 && total_rows <= kSmallRows && tensor_bytes <= (size_t)kSmallBytes) {
    if (c->dtype == SM_BF16)
      hipLaunchKernelGGL(append_small_kernel<uint16_t>, dim3(1), dim3(kMetaThreads), 0, stream, a, seq_ids,
                         row_offsets, n, total_rows, (const uint16_t *)K, (const uint16_t *)V, upr);
    else
      hipLaunchKernelGGL(append_small_kernel<float>, dim3(1), dim3(kMetaThreads), 0, stream, a, seq_ids,
                         row_offsets, n, total_rows, (const float *)K, (const float *)V, upr);
    return hipGetLastError() == hipSuccess ? SM_OK : SM_EHIP;
  }
  hipLaunchKernelGGL(append_meta_kernel, dim3(1), dim3(kMetaThreads), 0, stream, a, seq_ids, row_offsets, n,
                     total_rows);
  if (hipGetLastError() != hipSuccess) return SM_EHIP;
  if (total_rows == 0) return SM_OK;
  const dim3 grid((total_rows + kCopyRows - 1) / kCopyRows);
  if (c->dtype == SM_BF16)
    hipLaunchKernelGGL(append_copy_kernel<uint16_t>, grid, dim3(kCopyThreads), lds, stream, a, seq_ids,
                       row_offsets, n, total_rows, (const uint16_t *)K, (const uint16_t *)V);
  else
    hipLaunchKernelGGL(append_copy_kernel<float>, grid, dim3(kCopyThreads), lds, stream, a, seq_ids,
                       row_offsets, n, total_rows, (const float *)K, (const float *)V);
  return hipGetLastError() == hipSuccess ? SM_OK : SM_EHIP;
}

SM_API sm_status sm_pack_spans(int B, const int32_t *seq_offsets, int total_tokens, int num_spans,
                               const int32_t *span_start, const int32_t *span_len,
                               const int32_t *seq_span_offsets, int32_t *pi, int32_t *packed_offsets,
                               int32_t *packed_src, const int32_t *token_ids, const void *emb,
                               int64_t emb_rows, const void *surrogates, int d, sm_dtype dt, void *packed,
                               int32_t *err, hipStream_t stream) {
  if (B < 0 || total_tokens < 0 || num_spans < 0 || B > 65535) return SM_EINVAL;
  if (B == 0) return SM_OK;
  if (!seq_offsets || !seq_span_offsets || !packed_offsets || !err) return SM_EINVAL;
  if (total_tokens > 0 && (!pi || !packed_src)) return SM_EINVAL;
  if (num_spans > 0 && (!span_start || !span_len)) return SM_EINVAL;
  if (packed) {
    if (dt != SM_F32 && dt != SM_BF16) return SM_EINVAL;
    if (!token_ids || !emb || (num_spans > 0 && !surrogates) || d <= 0 || d % 8 || emb_rows <= 0)
      return SM_EINVAL;
  }
  PackArgs a;
  a.B = B;
  a.total_tokens = total_tokens;
  a.num_spans = num_spans;
  a.seq_offsets = seq_offsets;
  a.span_start = span_start;
  a.span_len = span_len;
  a.seq_span_offsets = seq_span_offsets;
  a.pi = pi;
  a.packed_offsets = packed_offsets;
  a.packed_src = packed_src;
  a.token_ids = token_ids;
  a.emb = emb;
  a.emb_rows = emb_rows;
  a.surrogates = surrogates;
  a.d = d;
  a.packed = packed;
  a.err = err;
  hipLaunchKernelGGL(pack_index_kernel, dim3(B), dim3(kPackThreads), 0, stream, a);
  if (hipGetLastError() != hipSuccess) return SM_EHIP;
  if (packed && total_tokens > 0) {
    const dim3 grid(total_tokens < 8192 ? total_tokens : 8192);
    if (dt == SM_BF16)
      hipLaunchKernelGGL(pack_rows_kernel<uint16_t>, grid, dim3(256), 0, stream, a);
    else
      hipLaunchKernelGGL(pack_rows_kernel<float>, grid, dim3(256), 0, stream, a);
    if (hipGetLastError() != hipSuccess) return SM_EHIP;
  }
  return SM_OK;
}
