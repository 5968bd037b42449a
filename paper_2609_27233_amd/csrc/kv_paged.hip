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
// request t's sequence id is in range and no earlier request of the call
// names it (ids: the call's ids, staged in LDS; no early exit, so the
// reads issue back to back)
__device__ __forceinline__ bool id_ok(const int *ids, int t, int s, int max_seqs) {
  bool dup = false;
  for (int j = 0; j < t; ++j) dup |= ids[j] == s;
  return s >= 0 && s < max_seqs && !dup;
}

__global__ __launch_bounds__(kMetaThreads) void rollback_kernel(CacheArgs c, const int32_t *seq_ids,
                                                                 const int32_t *ks, int n) {
  __shared__ int red[16];
  __shared__ int fl_inval, fl_range, s_err, s_top;
  __shared__ int ids[kMetaThreads];
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
    ids[t] = s;
  }
  __syncthreads();
  if (active && (k < 0 || !id_ok(ids, t, s, c.max_seqs))) fl_inval = 1;
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
  int incl[kMetaThreads];   // inclusive prefix of the blocks each request pops
  int first[kMetaThreads];  // its first new logical block
  int sid[kMetaThreads];    // its sequence
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
    sh.sid[t] = s;
  }
  __syncthreads();
  if (active && (m < 0 || !id_ok(sh.sid, t, s, c.max_seqs))) sh.fl_inval = 1;
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
  // (the first kPopCache ids of each thread stay in registers for the pops)
  constexpr int kPopCache = 4;
  int popv[kPopCache];
#pragma unroll
  for (int k = 0; k < kPopCache; ++k) {
    const int j = t + k * (int)blockDim.x;
    popv[k] = j < total ? c.free_stack[top - 1 - j] : 0;
  }
#pragma unroll
  for (int k = 0; k < kPopCache; ++k)
    if (t + k * (int)blockDim.x < total && (popv[k] < 0 || popv[k] >= c.num_blocks)) sh.fl_stack = 1;
  for (int j = t + kPopCache * (int)blockDim.x; j < total; j += blockDim.x) {
    const int blk = c.free_stack[top - 1 - j];
    if (blk < 0 || blk >= c.num_blocks) sh.fl_stack = 1;
  }
  __syncthreads();
  if (sh.fl_stack) {
    if (t == 0) set_err(c.err, SM_ERR_EINVAL);
    return false;
  }
  if (active) {
    sh.incl[t] = incl;
    sh.first[t] = blocks_for(L, c.bs_log2);
    sh.sid[t] = s;
    c.lengths[s] = L + m;
  }
  __syncthreads();
  // pop p goes to the request whose range [incl - need, incl) holds it:
  // free_stack[top - 1 - p] -> block_table[s][first + p - (incl - need)];
  // all threads share the pops (a prompt batch takes thousands of blocks)
  auto pop = [&](int p, int blk) {
    int lo = 0, hi = n - 1;  // first request with incl > p
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (sh.incl[mid] > p) hi = mid;
      else lo = mid + 1;
    }
    const int before = lo ? sh.incl[lo - 1] : 0;
    c.block_table[(int64_t)sh.sid[lo] * c.max_blocks + sh.first[lo] + (p - before)] = blk;
  };
#pragma unroll
  for (int k = 0; k < kPopCache; ++k) {
    const int p = t + k * (int)blockDim.x;
    if (p < total) pop(p, popv[k]);
  }
  for (int p = t + kPopCache * (int)blockDim.x; p < total; p += blockDim.x) pop(p, c.free_stack[top - 1 - p]);
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

// Copy phase of kv_append, run after append_meta_kernel has validated the
// call, taken the blocks and advanced the lengths.  The unit of work is a
// 16-slot segment (16-aligned positions) of a destination page that the
// call writes: request i writes positions [L_old, L_new) of its sequence,
// which touch segments L_old / 16 .. (L_new - 1) / 16.  The grid is
// persistent (at most the resident workgroups): each workgroup forms the
// prefix sum of the segment counts over the requests once, then takes
// kSegPerWg consecutive segments at a time, one per group of kSegThreads
// threads, stepping by the grid (measured 7% faster for a 39k-row prompt
// batch than one launch-wide wave of two-segment workgroups, which paid
// the prefix sum's chain of dependent reads for every 256 KB they moved).
// Slots outside [L_old, L_new) are never written.
//  * K pages are token-major ([head][slot][dim]): every 16-byte group of a
//    row is a 16-byte load and a 16-byte store.
//  * V pages are dim-major ([head][dim][slot]): a thread loads VEC rows x
//    VEC dims (VEC 16-byte loads: VEC consecutive positions, VEC dims of
//    one head), transposes them in registers and stores VEC 16-byte
//    groups (VEC consecutive slots of one dim); partly covered groups fall
//    back to one store per element.
// Every load of a thread is issued before its stores.  The error word is
// read beside the first index loads; nothing is written if it is set.
constexpr int kSegSlots = 16;
constexpr int kSegThreads = 256;
constexpr int kSegPerWg = 1;
constexpr int kSegWgThreads = kSegThreads * kSegPerWg;
constexpr int kMaxRowElems = 2048;  // num_kv_heads * head_dim

// out[i] = element i of in[0..VEC-1] (a VEC x VEC transpose of 16-byte rows)
__device__ __forceinline__ void transpose_rows(const u32x4_t (&in)[8], u32x4_t (&out)[8]) {  // bf16
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t x = in[2 * w][i >> 1], y = in[2 * w + 1][i >> 1];
      out[i][w] = (i & 1) ? ((x >> 16) | (y & 0xffff0000u)) : ((x & 0xffffu) | (y << 16));
    }
}
__device__ __forceinline__ void transpose_rows(const u32x4_t (&in)[4], u32x4_t (&out)[4]) {  // fp32
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) out[i][j] = in[j][i];
}

struct SegDesc {
  int row0, lold, lnew, seg, blk;  // blk -1: nothing to write
};

template <typename T>
__global__ __launch_bounds__(kSegWgThreads) void append_segments_kernel(CacheArgs c, const int32_t *seq_ids,
                                                                        const int32_t *row_offsets, int n,
                                                                        const T *__restrict__ K,
                                                                        const T *__restrict__ V) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int RPT = (SM_MAX_REQUESTS + kSegWgThreads - 1) / kSegWgThreads;  // requests per thread
  __shared__ int red[16];
  __shared__ SegDesc sd[kSegPerWg];
  const int t = threadIdx.x;
  // segments per request, requests RPT t .. RPT t + RPT - 1, and the error word
  const int err0 = *c.err;
  int cnt[RPT], sq[RPT], ro[RPT], mm[RPT], ln[RPT], mine = 0;
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    const int j = RPT * t + k;
    sq[k] = j < n ? seq_ids[j] : 0;
    ro[k] = j < n ? row_offsets[j] : 0;
    mm[k] = j < n ? row_offsets[j + 1] - ro[k] : 0;
  }
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    const int j = RPT * t + k;
    // advanced by the metadata pass (ids are checked: this read precedes
    // the error word's, which tells whether that pass failed)
    ln[k] = (j < n && sq[k] >= 0 && sq[k] < c.max_seqs) ? c.lengths[sq[k]] : 0;
    cnt[k] = (j < n && mm[k] > 0) ? ((ln[k] - 1) >> 4) - ((ln[k] - mm[k]) >> 4) + 1 : 0;
    mine += cnt[k];
  }
  if (t < kSegPerWg) sd[t].blk = -1;
  int total;
  const int incl = block_inclusive_scan(mine, red, &total);  // (its barriers order the sd writes)
  if (__syncthreads_or(err0 != 0)) return;  // uniform
  for (int b0 = blockIdx.x * kSegPerWg; b0 < total; b0 += gridDim.x * kSegPerWg) {
    if (b0 != (int)blockIdx.x * kSegPerWg) {
      __syncthreads();  // every thread holds the previous segments' descriptors
      if (t < kSegPerWg) sd[t].blk = -1;
      __syncthreads();
    }
    {
      int before = incl - mine;
#pragma unroll
      for (int k = 0; k < RPT; ++k) {
#pragma unroll
        for (int q = 0; q < kSegPerWg; ++q) {
          const int b = b0 + q;
          if (b < total && b >= before && b < before + cnt[k]) {
            const int seg = ((ln[k] - mm[k]) >> 4) + (b - before);
            SegDesc d;
            d.row0 = ro[k];
            d.lold = ln[k] - mm[k];
            d.lnew = ln[k];
            d.seg = seg;
            d.blk = c.block_table[(int64_t)sq[k] * c.max_blocks + ((seg << 4) >> c.bs_log2)];
            if (d.blk < 0 || d.blk >= c.num_blocks) {
              set_err(c.err, SM_ERR_EINVAL);  // corrupt block table: the segment is not written
              d.blk = -1;
            }
            sd[q] = d;
          }
        }
        before += cnt[k];
      }
    }
    __syncthreads();
    const int q = t / kSegThreads, tt = t - q * kSegThreads;
    const SegDesc d = sd[q];
    if (d.blk < 0) continue;  // (no barrier in the copy: the next one is the next iteration's)
    const int bs = 1 << c.bs_log2;
    const int p0 = d.seg << 4;                       // first position of the segment
    const int lo = max(p0, d.lold) - p0, hi = min(p0 + kSegSlots, d.lnew) - p0;  // valid slots [lo, hi)
    const int slot0 = p0 & (bs - 1);
    const int64_t row_elems = (int64_t)c.Hkv << c.dh_log2;
    const int64_t rbase = (int64_t)(d.row0 + p0 - d.lold) * row_elems;  // input offset of slot 0's row
    T *kp = (T *)c.k_pool + (int64_t)d.blk * row_elems * bs;
    T *vp = (T *)c.v_pool + (int64_t)d.blk * row_elems * bs;
    const int vpr = (int)(row_elems / VEC);        // 16-byte groups per row
    const int gshift = c.dh_log2;                  // element index -> head

    // V: sub-unit = (head, VEC dims, VEC slots)
    const int dgs = (1 << c.dh_log2) / VEC;        // dim groups per head
    const int sub_units = c.Hkv * dgs * (kSegSlots / VEC);
    // K: unit = one 16-byte group of one slot's row
    const int k_units = kSegSlots * vpr;
    for (int base_v = 0, base_k = 0; base_v < sub_units || base_k < k_units;
         base_v += kSegThreads, base_k += 8 * kSegThreads) {
      // loads
      u32x4_t va[VEC];
      const int su = base_v + tt;
      int sg = 0, g = 0, dg = 0;
      if (su < sub_units) {
        sg = su % (kSegSlots / VEC);
        const int hd = su / (kSegSlots / VEC);
        g = hd / dgs;
        dg = hd - g * dgs;
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
          const int sl = sg * VEC + j;
          va[j] = (sl >= lo && sl < hi)
                      ? *(const u32x4_t *)(V + rbase + (int64_t)sl * row_elems + ((int64_t)g << gshift) + dg * VEC)
                      : u32x4_t{0u, 0u, 0u, 0u};
        }
      }
      u32x4_t ka[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = base_k + u * kSegThreads + tt;
        const int sl = e / vpr;
        ka[u] = (e < k_units && sl >= lo && sl < hi)
                    ? *(const u32x4_t *)(K + rbase + (int64_t)sl * row_elems + (int64_t)(e - sl * vpr) * VEC)
                    : u32x4_t{0u, 0u, 0u, 0u};
      }
      // stores
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = base_k + u * kSegThreads + tt;
        const int sl = e / vpr;
        if (e < k_units && sl >= lo && sl < hi) {
          const int el = (e - sl * vpr) * VEC;      // element within the row
          const int gg = el >> gshift, dd = el & ((1 << gshift) - 1);
          // streaming stores: whole 256-byte runs of a token-major page
          // (measured 1.2x faster for the call than plain stores; the V
          // pages' 32-byte pieces are faster as plain stores that L2 merges)
          __builtin_nontemporal_store(ka[u], (u32x4_t *)(kp + (((int64_t)gg * bs + slot0 + sl) << gshift) + dd));
        }
      }
      if (su < sub_units) {
        u32x4_t vt[VEC];
        transpose_rows(va, vt);
        const int s_first = sg * VEC;
        T *vd = vp + (((int64_t)g << gshift) + dg * VEC) * bs + slot0 + s_first;
        if (s_first >= lo && s_first + VEC <= hi) {
#pragma unroll
          for (int i = 0; i < VEC; ++i) *(u32x4_t *)(vd + (int64_t)i * bs) = vt[i];
        } else {
#pragma unroll
          for (int i = 0; i < VEC; ++i) {
            const T *e = (const T *)&vt[i];
#pragma unroll
            for (int j = 0; j < VEC; ++j)
              if (s_first + j >= lo && s_first + j < hi) vd[(int64_t)i * bs + j] = e[j];
          }
        }
      }
    }
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
// workgroup writes with offsets computed from invalid input.  The span ->
// sequence search and the sequence bounds it checks read LDS copies of
// seq_span_offsets and seq_offsets when they fit (kPackSsoLds entries),
// else global memory; each thread loads its spans kPackBatch at a time
// (22.4 -> 17.3 us for the index pass of a 16 x 4096-token batch, with the
// removed-position counts folded into the same pass).
constexpr int kPackSsoLds = 4096;

__device__ bool pack_inputs_valid(const PackArgs &a, int *flag, int *sso, int *so, int sp0, int &removed_before,
                                  int &removed_all) {
  const int t = threadIdx.x;
  if (t == 0) {
    *flag = 0;
    if (a.seq_offsets[0] != 0 || a.seq_offsets[a.B] != a.total_tokens ||
        a.seq_span_offsets[0] != 0 || a.seq_span_offsets[a.B] != a.num_spans)
      *flag = 1;
  }
  const bool in_lds = a.B + 1 <= kPackSsoLds;
  if (in_lds)
    for (int b = t; b <= a.B; b += blockDim.x) {
      sso[b] = a.seq_span_offsets[b];
      so[b] = a.seq_offsets[b];
    }
  __syncthreads();
  for (int b = t; b < a.B; b += blockDim.x)
    if (a.seq_offsets[b + 1] < a.seq_offsets[b] || a.seq_span_offsets[b + 1] < a.seq_span_offsets[b])
      *flag = 1;
  __syncthreads();
  if (*flag) return false;
  const int *sso_src = in_lds ? sso : a.seq_span_offsets;
  const int *so_src = in_lds ? so : a.seq_offsets;
  // kPackBatch spans per thread at a time: their loads share one round trip.
  // The same pass counts the positions the spans remove (len - 1 each), in
  // total and before this workgroup's sequence (first span sp0).
  constexpr int kPackBatch = 4;
  for (int s0 = t; s0 < a.num_spans; s0 += kPackBatch * (int)blockDim.x) {
    int st[kPackBatch], ln[kPackBatch], pe[kPackBatch];
#pragma unroll
    for (int k = 0; k < kPackBatch; ++k) {
      const int s = s0 + k * (int)blockDim.x;
      const bool in = s < a.num_spans;
      st[k] = in ? a.span_start[s] : 0;
      ln[k] = in ? a.span_len[s] : 1;
      pe[k] = (in && s > 0) ? a.span_start[s - 1] + a.span_len[s - 1] : 0;  // end of the previous span
    }
#pragma unroll
    for (int k = 0; k < kPackBatch; ++k) {
      const int s = s0 + k * (int)blockDim.x;
      if (s >= a.num_spans) break;
      int lo = 0, hi = a.B - 1;  // sequence b with sso[b] <= s < sso[b+1]
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (sso_src[mid] <= s) lo = mid;
        else hi = mid - 1;
      }
      bool ok = ln[k] >= 1 && st[k] >= so_src[lo] && (int64_t)st[k] + ln[k] <= so_src[lo + 1];
      if (ok && s > sso_src[lo]) ok = st[k] >= pe[k];
      if (!ok) *flag = 1;
      removed_all += ln[k] - 1;
      if (s < sp0) removed_before += ln[k] - 1;
    }
  }
  __syncthreads();
  return *flag == 0;
}

__global__ __launch_bounds__(kPackThreads) void pack_index_kernel(PackArgs a) {
  __shared__ int src[kPackChunk];
  __shared__ int sso[kPackSsoLds], so[kPackSsoLds];
  __shared__ int red[16];
  __shared__ int flag, s_err;
  __shared__ float fred[16];
  const int b = blockIdx.x, t = threadIdx.x;
  if (t == 0) s_err = *a.err;
  __syncthreads();
  if (s_err != 0) return;
  int removed_before = 0, removed_all = 0;  // (this thread's spans)
  if (!pack_inputs_valid(a, &flag, sso, so, a.seq_span_offsets[b], removed_before, removed_all)) {
    if (b == 0 && t == 0) set_err(a.err, SM_ERR_EINVAL);
    return;
  }
  const int sp0 = a.seq_span_offsets[b], sp1 = a.seq_span_offsets[b + 1];
  // positions removed before this sequence (and in total, for the last
  // one), summed over the threads
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

// Copy phase of pack_spans: packed[r] = emb[token_ids[src]] (src >= 0) or
// surrogates[-1 - src], src = packed_src[r].  One wave per packed row, the
// waves striding over the rows; no barriers.  The next row's source index
// is loaded before the current row's data and its token id right after, so
// the two dependent index loads ride along the data round trip.
constexpr int kPackRowThreads = 256;
constexpr int kPackLaneGroups = 16;  // 16-byte groups per lane and pass (1024 per wave)

template <typename T>
__device__ __forceinline__ const T *pack_source(const PackArgs &a, int src, int tok) {
  if (src < 0) return (const T *)a.surrogates + (int64_t)(-1 - src) * a.d;
  if (tok < 0 || tok >= a.emb_rows) return nullptr;
  return (const T *)a.emb + (int64_t)tok * a.d;
}

template <typename T>
__global__ __launch_bounds__(kPackRowThreads) void pack_rows_kernel(PackArgs a) {
  const int lane = threadIdx.x & 63;
  const int nwaves = gridDim.x * (kPackRowThreads / 64);
  int r = blockIdx.x * (kPackRowThreads / 64) + (threadIdx.x >> 6);
  const int err0 = *a.err;
  const int nrows = a.packed_offsets[a.B];
  if (err0 != 0 || r >= nrows) return;
  constexpr int VEC = 16 / sizeof(T);
  const int vpr = a.d / VEC;
  int src = a.packed_src[r];
  const T *row = pack_source<T>(a, src, src >= 0 ? a.token_ids[src] : 0);
  for (; r < nrows; r += nwaves) {
    const int rn = r + nwaves;
    const int src_n = rn < nrows ? a.packed_src[rn] : -1;
    if (!row && lane == 0) set_err(a.err, SM_ERR_EINVAL);  // token id out of range: row skipped
    T *dst = (T *)a.packed + (int64_t)r * a.d;
    int tok_n = 0;
    for (int v0 = 0; v0 < vpr; v0 += 64 * kPackLaneGroups) {
      u32x4_t v[kPackLaneGroups];
#pragma unroll
      for (int u = 0; u < kPackLaneGroups; ++u) {
        const int idx = v0 + 64 * u + lane;
        if (row && idx < vpr) v[u] = *(const u32x4_t *)(row + (int64_t)idx * VEC);
      }
      if (v0 == 0 && rn < nrows && src_n >= 0) tok_n = a.token_ids[src_n];
#pragma unroll
      for (int u = 0; u < kPackLaneGroups; ++u) {
        const int idx = v0 + 64 * u + lane;
        // streaming stores: the packed rows are read back by the backbone's
        // prefill, not by this pass (measured 1.3x faster than plain stores)
        if (row && idx < vpr) __builtin_nontemporal_store(v[u], (u32x4_t *)(dst + (int64_t)idx * VEC));
      }
    }
    row = rn < nrows ? pack_source<T>(a, src_n, tok_n) : nullptr;
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

// Resident copy workgroups over the whole device (looked up once per
// element type): the persistent grid of append_segments_kernel.
template <typename T>
static int seg_resident() {
  static const int nb = [] {
    int dev = 0, cus = 0, occ = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
      cus = 256;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, append_segments_kernel<T>, kSegWgThreads, 0) !=
            hipSuccess ||
        occ <= 0)
      occ = 1;
    return cus * occ;
  }();
  return nb;
}

SM_API sm_status sm_kv_append(const sm_paged_cache *c, const int32_t *seq_ids, const int32_t *row_offsets,
                              int n, int total_rows, const void *K, const void *V, hipStream_t stream) {
  CacheArgs a;
  if (!cache_ok(c, a) || n < 0 || n > SM_MAX_REQUESTS || n > c->max_seqs || total_rows < 0)
    return SM_EINVAL;
  if (n == 0) return total_rows == 0 ? SM_OK : SM_EINVAL;
  if (!seq_ids || !row_offsets || (total_rows > 0 && (!K || !V))) return SM_EINVAL;
  const size_t es = c->dtype == SM_BF16 ? 2 : 4;
  if (c->num_kv_heads * c->head_dim > kMaxRowElems) return SM_EINVAL;
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
  // segments touched: at most ceil(m / 16) + 1 per request
  const int64_t segs = (int64_t)(total_rows + kSegSlots - 1) / kSegSlots + 2 * (int64_t)n;
  const int64_t wgs = (segs + kSegPerWg - 1) / kSegPerWg;
  const int resident = c->dtype == SM_BF16 ? seg_resident<uint16_t>() : seg_resident<float>();
  const dim3 grid((unsigned)(wgs < resident ? wgs : resident));
  if (c->dtype == SM_BF16)
    hipLaunchKernelGGL(append_segments_kernel<uint16_t>, grid, dim3(kSegWgThreads), 0, stream, a, seq_ids,
                       row_offsets, n, (const uint16_t *)K, (const uint16_t *)V);
  else
    hipLaunchKernelGGL(append_segments_kernel<float>, grid, dim3(kSegWgThreads), 0, stream, a, seq_ids,
                       row_offsets, n, (const float *)K, (const float *)V);
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
    // one wave per packed row, striding: up to 4 waves per compute unit's
    // worth of workgroups (the packed rows are at most total_tokens)
    const int64_t wgs = ((int64_t)total_tokens + 3) / 4;
    const dim3 grid((unsigned)(wgs < 2048 ? wgs : 2048));
    if (dt == SM_BF16)
      hipLaunchKernelGGL(pack_rows_kernel<uint16_t>, grid, dim3(kPackRowThreads), 0, stream, a);
    else
      hipLaunchKernelGGL(pack_rows_kernel<float>, grid, dim3(kPackRowThreads), 0, stream, a);
    if (hipGetLastError() != hipSuccess) return SM_EHIP;
  }
  return SM_OK;
}
