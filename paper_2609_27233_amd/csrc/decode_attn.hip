// Split-K grouped-query decode attention over the paged KV cache (gfx950).
//
// Each decode step of the frozen backbone attends from one new query per
// sequence to every cached entry; span merging shortens that cache, which is
// where the method's decode-time saving comes from (paper, "Efficiency
// Analysis").  The operation itself is ordinary attention:
//   out[i,h] = sum_j softmax_j(scale * q[i,h] . K[s,j,g]) V[s,j,g],  g = h / G.
//
// Phase 1 (split): one workgroup per (chunk, kv head, sequence).  Four
// waves stream 32-token tiles of the chunk straight from HBM into registers
// in the matrix-core operand layout (no LDS staging: every K/V byte is used
// by exactly one MFMA), compute S^T = K Q^T and O^T += V^T P^T with
// v_mfma_f32_16x16x32_bf16 (the G query heads of the group padded to 16
// columns), and keep an online softmax per head.  The waves merge through
// LDS and write one unnormalised partial (O, m, l) per chunk.  The last
// workgroup of a (sequence, kv head) to finish -- found with an arrival
// counter in the workspace -- rescales and sums the partials exactly and
// writes the output, so one kernel launch does the whole operation.
//
// The fused decode step (sm_decode_step) runs the same kernel with the
// step's one-row-per-sequence append folded in: the new row is read from
// the input and folded into the softmax of the chunk that holds its
// position, that chunk's workgroup stores it into its page, and the
// append's metadata (lengths, new block-table entries, free-stack top) is
// committed by one extra workgroup once every attention workgroup is past
// its metadata reads (details at the step helpers below).
//
// V pages are stored dim-major ([head_dim][block_size]), so the 8 tokens a
// lane feeds to the PV product are 16 contiguous bytes.  The QK rows of the
// two 16-row score tiles are permuted so that the score tile's output layout
// is already the PV operand layout: lane (r, q) of a wave owns the scores of
// tokens 8q .. 8q+7 of the tile for head r.
#include <atomic>
#include <mutex>

#include "common.hpp"

namespace sm {

constexpr int kDecThreads = 256;
constexpr int kDecWaves = kDecThreads / 64;
constexpr int kMaxChunkTokens = 8192;
constexpr int kMaxChunkPages = kMaxChunkTokens / 16 + 2;
constexpr int kF32ChunkTokens = 256;
constexpr float kLog2e = 1.4426950408889634f;

struct DecodeArgs {
  const void *k_pool;
  const void *v_pool;
  const int32_t *block_table;
  const int32_t *lengths;
  const int32_t *seq_ids;
  const void *q;
  void *out;
  float *ws_o;   // [n][Hq][max_chunks][DH]
  float *ws_ml;  // [n][Hq][max_chunks][2]
  int32_t *counters;  // [n][Hkv] arrival counters, zero between calls
  int32_t *err;
  int Hkv, Hq, G, bs_log2, num_blocks, max_seqs, max_blocks;
  int chunk_nominal, max_chunks, max_len;
  float scale_log2e;
  // fused decode step only (sm_decode_step)
  const void *k_new;         // [n][Hkv][DH] rows appended, request order
  const void *v_new;
  int32_t *free_stack;
  int32_t *free_top;
  int32_t *block_table_w;    // the same arrays as block_table / lengths,
  int32_t *lengths_w;        // written only by the committing workgroup
  int32_t *step_err;         // workspace word: error bits parked until commit
  int32_t *step_arrivals;    // workspace word: workgroups past their reads
  int n, cap, total_wgs;
  int spin_limit;            // polls of the commit workgroup's bounded wait  // bf16 kernels, one chunk per (sequence, kv head): with order_n > 0 the
  // grid's workgroups take the (sequence, head) pairs longest first, dealt
  // over order_cus compute units holding order_occ workgroups each
  int order_n, order_cus, order_occ;
  // decode-time merge step only (sm_decode_merge_step): entries cropped
  // from each request's cache before its row is appended, request order
  const int32_t *crop;
};

// Chunking of a sequence of L cached entries: nc non-empty chunks of
// `chunk` tokens (a multiple of 32, at most C), all of nearly equal size.
// Every workgroup of the sequence computes the same split from the same L.
__device__ __forceinline__ void chunking(int L, int C, int &nc, int &chunk) {
  const int n0 = (L + C - 1) / C;
  chunk = n0 ? ((L + n0 - 1) / n0 + 31) / 32 * 32 : 0;
  nc = chunk ? (L + chunk - 1) / chunk : 0;
}

// Sequence-level checks shared by split and combine.  Returns 0 when the
// sequence can be processed, else the error bit (0 length is fine).
__device__ __forceinline__ int seq_status(const DecodeArgs &a, int s, int &L, bool known = false,
                                          int L_known = 0) {
  L = 0;
  if (s < 0 || s >= a.max_seqs) return SM_ERR_EINVAL;
  L = known ? L_known : a.lengths[s];
  if (L < 0 || L > (a.max_blocks << a.bs_log2)) return SM_ERR_EINVAL;
  if (L > a.max_len) return SM_ERR_ERANGE;
  return 0;
}

// Ragged batches with more (sequence, kv head) pairs than compute units
// (one chunk each): every workgroup sorts the requests by cached length
// (longest first, ties by request index) and takes the pair of its rank, so
// that long pairs start first.  While the grid's first order_occ *
// order_cus workgroups are all resident, workgroup b shares a compute unit
// with b +- order_cus (the dispatcher deals one per unit in grid order), so
// alternate rounds of order_cus ranks are dealt in reverse: a unit that
// got a long pair in one round gets a short one in the next.  Workgroups
// past that point are dispatched as units free up, longest first.  The
// order only decides which workgroup does which pair: results do not
// depend on it.
__device__ __forceinline__ int dealt_rank(int b, int W, int cus, int occ) {
  const int M = min(W, cus * occ);
  if (b >= M || cus <= 0) return b;
  const int r = b / cus;
  if (!(r & 1)) return b;
  const int mr = min(cus, M - r * cus);
  return r * cus + (mr - 1 - (b - r * cus));
}

// The (request, kv head) of grid position (row i, head column g) under the
// length order; s_out / L_out: the request's sequence id and its cached
// length (-1 for an id out of range).  All threads take part: order_n is at
// most the workgroup size.  Request j's sort key is (length, then the
// smaller index) packed into one 64-bit integer, so that its rank is the
// number of larger keys; P = 256 / n (at most 4) threads count over
// contiguous shares of the keys and add their counts.  LDS: `key` order_n
// 64-bit keys, `sid` order_n ints, `pick` one int.
__device__ __forceinline__ void order_pick(const DecodeArgs &a, int &g, int &i, int &s_out, int &L_out,
                                           int64_t *key, int *sid, int *pick) {
  const int n = a.order_n, tid = threadIdx.x;
  const int rho = dealt_rank(i * a.Hkv + g, n * a.Hkv, a.order_cus, a.order_occ);
  const int k = rho / a.Hkv;
  g = rho - k * a.Hkv;
  if (tid < n) {
    const int sj = a.seq_ids[tid];
    const int kj = (sj >= 0 && sj < a.max_seqs) ? a.lengths[sj] : -1;
    key[tid] = (int64_t)kj * 512 + (511 - tid);
    sid[tid] = sj;
  }
  lds_barrier();
  const int P = n <= 64 ? 4 : n <= 128 ? 2 : 1;
  const int j = tid / P, part = tid - j * P;
  int r = 0;
  if (j < n) {
    const int64_t kj = key[j];
    const int m0 = part * n / P, m1 = (part + 1) * n / P;
#pragma unroll 8
    for (int m = m0; m < m1; ++m) r += key[m] > kj;
  }
  // the P threads of a request are consecutive lanes of one wave
  if (P >= 2) r += __shfl_xor(r, 1, kWave);
  if (P >= 4) r += __shfl_xor(r, 2, kWave);
  if (j < n && part == 0 && r == k) *pick = j;  // ranks are a permutation of 0 .. n - 1: exactly one
  lds_barrier();
  i = *pick;
  s_out = sid[i];
  L_out = (int)((key[i] - (511 - i)) / 512);
}

// Load the block ids of logical pages [lp0, lp0 + npages) into LDS and
// range-check them.  Returns true when every id is a valid block.
__device__ __forceinline__ bool load_pages(const DecodeArgs &a, int s, int lp0,
                                           int npages, int *pages, int *flag) {
  if (threadIdx.x == 0) *flag = 0;
  __syncthreads();
  for (int p = threadIdx.x; p < npages; p += blockDim.x) {
    int blk = a.block_table[(int64_t)s * a.max_blocks + lp0 + p];
    if (blk < 0 || blk >= a.num_blocks) {
      *flag = 1;
      blk = 0;
    }
    pages[p] = blk;
  }
  __syncthreads();
  return *flag == 0;
}

// Partials travel between workgroups as device-scope ("agent") relaxed
// atomic stores and loads: on gfx950 these go through the coherent level of
// the memory hierarchy, so no cache-wide writeback/invalidate fence is
// needed (such fences cost more than the whole attention pass).  Every
// store a workgroup makes has completed before its thread 0 bumps the
// arrival counter (the barrier waits for outstanding memory operations).
__device__ __forceinline__ void put_partial(float *p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float get_partial(const float *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void write_bad_partial(const DecodeArgs &a, int i,
                                                  int g, int c, int32_t *esink) {
  if (threadIdx.x < a.G) {
    const int64_t pidx = ((int64_t)i * a.Hq + g * a.G + threadIdx.x) * a.max_chunks + c;
    put_partial(&a.ws_ml[pidx * 2 + 0], 0.f);
    put_partial(&a.ws_ml[pidx * 2 + 1], -1.f);  // marks the chunk as unusable
  }
  if (threadIdx.x == 0 && esink) set_err(esink, SM_ERR_EINVAL);  // (no sink: reported elsewhere)
}

// Zero the output rows of group g's query heads (done by the chunk-0
// workgroup of a sequence that cannot be processed or is empty) and report a
// sequence-level error.
template <typename OutT>
__device__ void write_zero_rows(const DecodeArgs &a, int i, int g, int DH, int st, int32_t *esink) {
  OutT *o = (OutT *)a.out + ((int64_t)i * a.Hq + g * a.G) * DH;
  for (int e = threadIdx.x; e < a.G * DH; e += blockDim.x) o[e] = Elem<OutT>::to_store(0.f);
  if (st != 0 && threadIdx.x == 0 && esink) set_err(esink, st);  // (no sink: reported elsewhere)
}

// Every workgroup calls this once its partial is stored.  The last of the
// nc workgroups of (sequence i, kv head g) to arrive rescales and sums all
// partials of the group, writes the output rows and re-arms the counter.
// The partials are fetched kCombineBatch chunks at a time for all of a
// thread's output elements in one go (each fetch is a round trip to the
// coherent level of the memory hierarchy); across batches the running sum
// is rescaled to the running maximum, so for nc <= kCombineBatch the result
// is exactly max-then-sum over all chunks.
constexpr int kCombineBatch = 4;

template <typename OutT>
__device__ void finish_group(const DecodeArgs &a, int i, int g, int nc, int DH, int *last) {
  int32_t *ctr = a.counters + (int64_t)i * a.Hkv + g;
  __builtin_amdgcn_s_waitcnt(0);  // this thread's partial stores are done
  __syncthreads();
  if (threadIdx.x == 0)
    *last = __hip_atomic_fetch_add(ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == nc - 1;
  __syncthreads();
  if (!*last) return;
  OutT *out = (OutT *)a.out;
  constexpr int kPer = 2;  // output elements per thread and pass
  const int ne = a.G * DH;
  for (int e0 = 0; e0 < ne; e0 += kPer * kDecThreads) {
    float M[kPer], acc[kPer], ls[kPer];
    bool bad[kPer];
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      M[k] = -INFINITY;
      acc[k] = 0.f;
      ls[k] = 0.f;
      bad[k] = false;
    }
    for (int c0 = 0; c0 < nc; c0 += kCombineBatch) {
      float pm[kPer][kCombineBatch], pl[kPer][kCombineBatch], po[kPer][kCombineBatch];
#pragma unroll
      for (int k = 0; k < kPer; ++k) {
#pragma unroll
        for (int cc = 0; cc < kCombineBatch; ++cc) {
          pm[k][cc] = -INFINITY;
          pl[k][cc] = 0.f;
          po[k][cc] = 0.f;
        }
        const int e = e0 + threadIdx.x + kDecThreads * k;
        if (e < ne) {
          const int hh = e / DH, dd = e - hh * DH;
          const int64_t base = ((int64_t)i * a.Hq + g * a.G + hh) * a.max_chunks + c0;
#pragma unroll
          for (int cc = 0; cc < kCombineBatch; ++cc)
            if (c0 + cc < nc) {
              pm[k][cc] = get_partial(&a.ws_ml[(base + cc) * 2 + 0]);
              pl[k][cc] = get_partial(&a.ws_ml[(base + cc) * 2 + 1]);
              po[k][cc] = get_partial(&a.ws_o[(base + cc) * DH + dd]);
            }
        }
      }
#pragma unroll
      for (int k = 0; k < kPer; ++k) {
        float Mb = M[k];
#pragma unroll
        for (int cc = 0; cc < kCombineBatch; ++cc)
          if (c0 + cc < nc) {
            bad[k] |= pl[k][cc] < 0.f;
            Mb = fmaxf(Mb, pm[k][cc]);
          }
        if (M[k] != -INFINITY && Mb != M[k]) {  // rescale what earlier batches summed
          const float r = exp2f(M[k] - Mb);
          acc[k] *= r;
          ls[k] *= r;
        }
        M[k] = Mb;
#pragma unroll
        for (int cc = 0; cc < kCombineBatch; ++cc)
          if (c0 + cc < nc) {
            const float f = pm[k][cc] == -INFINITY ? 0.f : exp2f(pm[k][cc] - Mb);
            acc[k] += po[k][cc] * f;
            ls[k] += pl[k][cc] * f;
          }
      }
    }
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int e = e0 + threadIdx.x + kDecThreads * k;
      if (e < ne) {
        const int hh = e / DH, dd = e - hh * DH;
        out[((int64_t)i * a.Hq + g * a.G + hh) * DH + dd] =
            Elem<OutT>::to_store(bad[k] || !(ls[k] > 0.f) ? 0.f : acc[k] / ls[k]);
      }
    }
  }
  if (threadIdx.x == 0) *ctr = 0;
}

// ---------------------------------------------------------------------------
// Fused decode step (sm_decode_step): the one-row-per-sequence append of
// sm_kv_append followed by the attention over the appended cache, in the
// attention's own launch.
//
// Every workgroup derives the append's outcome from the cache as it was
// before the call -- the same checks in the same order as sm_kv_append
// (sticky error word, ids, lengths, free blocks, popped ids) and the same
// pops (request order, top of the free stack first) -- so all of them
// agree on it.  The new row is taken from the input: the workgroup whose
// chunk holds the new position folds the token into its softmax and
// writes the row into its page, a slot no other workgroup reads.  What the
// append changes in the metadata (lengths, the new block-table entries,
// the free-stack top, the error word) is written only by the workgroup
// that arrives last at a counter every workgroup bumps once all its
// metadata reads are done; error bits found on the way are parked in a
// workspace word and folded into the error word by that same workgroup.

struct StepShared {
  int ids[kDecThreads];  // request sequence ids
  int len[kDecThreads];  // lengths before the call
  int pop[kDecThreads];  // block popped for request t, or -1
  int red[16];
  int frozen, top, total, bits, errs, last, tail;
};

// Plan of the append, phases 1 and 2 (all threads, n <= kDecThreads):
// request ids, error word and stack top; then id checks, lengths and the
// blocks each request needs.  Leaves sp.bits = the first failing check
// (stack contents not yet looked at) and returns this thread's inclusive
// pop count; need_t = pops of request t (0 or 1).
__device__ int step_plan(const DecodeArgs &a, StepShared &sp, int &need_t) {
  const int t = threadIdx.x, n = a.n;
  if (t == 0) {
    sp.frozen = *a.err != 0;
    sp.top = *a.free_top;
    sp.errs = 0;
    sp.last = 0;
    sp.tail = -1;
  }
  int s = -1;
  if (t < n) {
    s = a.seq_ids[t];
    sp.ids[t] = s;
  }
  __syncthreads();
  int inval = 0, range = 0, need = 0, L = 0;
  if (t < n) {
    const bool id_ok = s >= 0 && s < a.max_seqs;
    bool ok = id_ok;
    for (int j = 0; j < t && ok; ++j) ok = sp.ids[j] != s;
    inval = !ok;
    if (id_ok) L = a.lengths[s];
    if (ok) {
      if (L < 0 || (int64_t)L + 1 > a.cap) range = 1;
      else need = (L & ((1 << a.bs_log2) - 1)) == 0;
    }
    sp.len[t] = L;
  }
  int total;
  const int incl = block_inclusive_scan(need, sp.red, &total);
  // (__syncthreads_or answers "any thread nonzero", one predicate per call)
  const int any_inval = __syncthreads_or(inval);
  const int any_range = __syncthreads_or(range);
  if (t == 0) {
    const int top = sp.top;
    sp.total = total;
    sp.bits = any_inval   ? SM_ERR_EINVAL
              : any_range ? SM_ERR_ERANGE
              : (top < 0 || top > a.num_blocks || total > top) ? SM_ERR_ENOMEM
                                                               : 0;
  }
  __syncthreads();
  need_t = need;
  return incl;
}

// Phase 3 (all threads): the popped block ids are read and checked, the
// page ids of this workgroup's chunk [lp0, lp0 + npages) of sequence s are
// loaded into LDS, and thread 0 fetches the tail block of request i when
// the new row lands in an existing page.  One barrier.  Returns whether
// every page id is valid; sets ok = the append will be committed.
__device__ bool step_pages(const DecodeArgs &a, StepShared &sp, int incl, int need_t, int i, int s,
                           int lp0, int npages, bool want_tail, int *pages, bool &ok) {
  const int t = threadIdx.x;
  const bool go = !sp.frozen && sp.bits == 0;
  int bad_stack = 0, bad_page = 0;
  if (t < a.n) {
    int blk = -1;
    if (go && need_t) {
      blk = a.free_stack[sp.top - 1 - (incl - 1)];
      if (blk < 0 || blk >= a.num_blocks) bad_stack = 1;
    }
    sp.pop[t] = blk;
  }
  for (int p = t; p < npages; p += kDecThreads) {
    int blk = a.block_table[(int64_t)s * a.max_blocks + lp0 + p];
    if (blk < 0 || blk >= a.num_blocks) {
      bad_page = 1;
      blk = 0;
    }
    pages[p] = blk;
  }
  if (t == 0 && want_tail) sp.tail = a.block_table[(int64_t)s * a.max_blocks + (sp.len[i] >> a.bs_log2)];
  const int any_stack = __syncthreads_or(bad_stack);
  const int any_page = __syncthreads_or(bad_page);
  ok = go && !any_stack;
  if (t == 0 && go && any_stack) sp.bits = SM_ERR_EINVAL;  // corrupt free stack
  return !any_page;
}

// Reads of the append's inputs for a register-held plan (request t = lane
// + 64 k, n <= 256), in two steps that ride along a workgroup's own round
// trips: ids, error word, stack top; then lengths and the top of the free
// stack (the blocks the call may pop).
struct PlanRegs {
  int sk[4], Lk[4], win[4];
  int ck[4];  // entries cropped first (decode-time merge step; else unused)
  int frozen, top;
};

template <bool CROP = false>
__device__ __forceinline__ void step_plan_read1(const DecodeArgs &a, PlanRegs &pr) {
  const int lane = threadIdx.x & 63;
  pr.frozen = *a.err != 0;
  pr.top = *a.free_top;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int t = lane + 64 * k;
    pr.sk[k] = t < a.n ? a.seq_ids[t] : -1;
    if constexpr (CROP) pr.ck[k] = t < a.n ? a.crop[t] : 0;
  }
}

__device__ __forceinline__ void step_plan_read2(const DecodeArgs &a, PlanRegs &pr) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int t = lane + 64 * k;
    const int sk = pr.sk[k];
    pr.Lk[k] = (t < a.n && sk >= 0 && sk < a.max_seqs) ? a.lengths[sk] : 0;
    pr.win[k] = (t < a.n && t < pr.top && pr.top <= a.num_blocks) ? a.free_stack[pr.top - 1 - t] : -1;
  }
}

// The same plan in registers only, worked out by one wave on its own (no
// LDS, no barriers): request ids are compared through shuffles, the pops
// are read out of the window by shuffles.  Every wave of every workgroup
// that calls it gets the same outcome.  Lane l holds requests l + 64 k.
struct PlanOut {
  bool ok;      // the append commits
  int bits;     // the append's error bits (0 when the error word was set)
  int total;    // blocks popped
  int need[4];  // per request of this lane: a block is popped for it
  int pop[4];   // ... and which one (or -1)
};

// Whether any id occurs twice among the n requests (lane l of the calling
// wave holds requests l + 64 k).  With the bitmap (one bit per sequence id,
// max_seqs <= 32 * kDupBitmapWords) it takes one LDS atomic per request;
// otherwise every earlier id is compared, a loop of n steps.  Only the
// calling wave uses the bitmap, and its LDS operations complete in order,
// so the clearing stores precede the atomics.
constexpr int kDupBitmapWords = 1024;

__device__ bool wave_any_dup(const DecodeArgs &a, const int (&sk)[4], uint32_t *bm) {
  const int lane = threadIdx.x & 63, n = a.n;
  int dup = 0;
  if (bm && a.max_seqs <= 32 * kDupBitmapWords) {
    const int words = (a.max_seqs + 31) >> 5;
    for (int wd = lane; wd < words; wd += kWave) bm[wd] = 0u;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int t = lane + 64 * k, s = sk[k];
      if (t < n && s >= 0 && s < a.max_seqs) {
        const uint32_t bit = 1u << (s & 31);
        const uint32_t old = __hip_atomic_fetch_or(&bm[s >> 5], bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        dup |= (old & bit) != 0;
      }
    }
  } else {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {  // every earlier request, 64 at a time
      if (64 * kk < n) {
        const int jn = min(64, n - 64 * kk);
        for (int jl = 0; jl < jn; ++jl) {
          const int idj = __builtin_amdgcn_readlane(sk[kk], jl);
          const int j = 64 * kk + jl;
#pragma unroll
          for (int k = 0; k < 4; ++k) dup |= (j < lane + 64 * k) && (lane + 64 * k < n) && idj == sk[k];
        }
      }
    }
  }
  return __ballot(dup) != 0;
}

__device__ void plan_regs(const DecodeArgs &a, const PlanRegs &pr, PlanOut &po, uint32_t *bm) {
  const int lane = threadIdx.x & 63, n = a.n;
  const bool any_dup = wave_any_dup(a, pr.sk, bm);
  int inval = 0, range = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int t = lane + 64 * k, sk = pr.sk[k], Lk = pr.Lk[k];
    po.need[k] = 0;
    if (t < n) {
      if (sk < 0 || sk >= a.max_seqs || any_dup) inval = 1;
      else if (Lk < 0 || (int64_t)Lk + 1 > a.cap) range = 1;
      else po.need[k] = (Lk & ((1 << a.bs_log2) - 1)) == 0;
    }
  }
  const bool any_inval = __ballot(inval) != 0;
  const bool any_range = __ballot(range) != 0;
  int incl[4] = {0, 0, 0, 0}, total = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {  // inclusive prefix of `need` (0 or 1) in request order
    if (64 * k < n) {
      const uint64_t m = __ballot(po.need[k]);
      const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
      incl[k] = total + below + po.need[k];
      total += __popcll(m);
    }
  }
  const int top = pr.top;
  int bits = any_inval ? SM_ERR_EINVAL
             : any_range ? SM_ERR_ERANGE
             : (top < 0 || top > a.num_blocks || total > top) ? SM_ERR_ENOMEM
                                                              : 0;
  const bool go = !pr.frozen && bits == 0;
  int bad = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    po.pop[k] = -1;
    if (64 * k < n) {
      // pop index incl - 1 < total <= min(top, n): entry of the window
      const int pidx = (go && po.need[k]) ? incl[k] - 1 : 0;
      int blk = __shfl(pr.win[0], pidx & 63, kWave);
      if (total > 64) {
        const int w1 = __shfl(pr.win[1], pidx & 63, kWave);
        const int w2 = __shfl(pr.win[2], pidx & 63, kWave), w3 = __shfl(pr.win[3], pidx & 63, kWave);
        const int q = pidx >> 6;
        blk = q == 0 ? blk : q == 1 ? w1 : q == 2 ? w2 : w3;
      }
      po.pop[k] = (go && po.need[k]) ? blk : -1;
      if (go && po.need[k] && (blk < 0 || blk >= a.num_blocks)) bad = 1;
    }
  }
  const bool any_stack = __ballot(bad) != 0;
  if (go && any_stack) bits = SM_ERR_EINVAL;  // corrupt free stack
  po.ok = go && !any_stack;
  po.bits = pr.frozen ? 0 : bits;
  po.total = total;
}

// The same plan when every request fits one slot (n <= 64, lane l holds
// request l): one pass over the earlier requests for duplicates and a
// single window of popped blocks.  Same outcome as plan_regs.
__device__ void plan_regs_one(const DecodeArgs &a, const PlanRegs &pr, PlanOut &po) {
  const int lane = threadIdx.x & 63, n = a.n;
  const int sk = pr.sk[0], Lk = pr.Lk[0];
  int dup = 0;
  for (int j = 0; j < n; ++j) dup |= (j < lane) & (__builtin_amdgcn_readlane(sk, j) == sk);
  int inval = 0, range = 0, need = 0;
  if (lane < n) {
    if (sk < 0 || sk >= a.max_seqs || dup) inval = 1;
    else if (Lk < 0 || (int64_t)Lk + 1 > a.cap) range = 1;
    else need = (Lk & ((1 << a.bs_log2) - 1)) == 0;
  }
  const bool any_inval = __ballot(inval) != 0;
  const bool any_range = __ballot(range) != 0;
  const uint64_t m = __ballot(need);
  const int incl = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0)) + need;
  const int total = __popcll(m);
  const int top = pr.top;
  int bits = any_inval ? SM_ERR_EINVAL
             : any_range ? SM_ERR_ERANGE
             : (top < 0 || top > a.num_blocks || total > top) ? SM_ERR_ENOMEM
                                                              : 0;
  const bool go = !pr.frozen && bits == 0;
  // pop index incl - 1 < total <= n <= 64: an entry of the first window
  const int blk = __shfl(pr.win[0], (go && need) ? incl - 1 : 0, kWave);
  const bool popped = go && need;
  const bool any_stack = __ballot(popped && (blk < 0 || blk >= a.num_blocks)) != 0;
  if (go && any_stack) bits = SM_ERR_EINVAL;  // corrupt free stack
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    po.need[k] = 0;
    po.pop[k] = -1;
  }
  po.need[0] = need;
  po.pop[0] = popped ? blk : -1;
  po.ok = go && !any_stack;
  po.bits = pr.frozen ? 0 : bits;
  po.total = total;
}

__device__ __forceinline__ void plan_any(const DecodeArgs &a, const PlanRegs &pr, PlanOut &po, uint32_t *bm) {
  if (a.n <= 64) plan_regs_one(a, pr, po);
  else plan_regs(a, pr, po, bm);
}

// Value of request i's slot k-array entry (held by lane i % 64) in every lane.
__device__ __forceinline__ int request_value(const int (&v)[4], int i) {
  const int l = i & 63, q = i >> 6;  // uniform
  return q == 0   ? __builtin_amdgcn_readlane(v[0], l)
         : q == 1 ? __builtin_amdgcn_readlane(v[1], l)
         : q == 2 ? __builtin_amdgcn_readlane(v[2], l)
                  : __builtin_amdgcn_readlane(v[3], l);
}

// The commit workgroup of a fused step (wave 0 only): the plan, then a wait
// -- bounded, sleeping -- until every attention workgroup has taken its
// reads of the metadata, then the metadata writes and the error bits.
// Every attention workgroup arrives exactly once, early, and nothing waits
// on this workgroup, so the wait ends; the bound (a.spin_limit polls) only
// guards the invariant.  If it ever gives up, nothing is committed and
// EINVAL is set; workgroups still arriving then leave the arrival counter
// nonzero, so the caller must zero the workspace's counters again before
// its next call.  (A lower bound can be set for tests of this path.)
constexpr int kCommitSpinLimit = 1 << 20;

__device__ void step_commit_wave(const DecodeArgs &a, uint32_t *bm) {
  const int lane = threadIdx.x & 63;
  PlanRegs pr;
  step_plan_read1(a, pr);
  step_plan_read2(a, pr);
  PlanOut po;
  plan_any(a, pr, po, bm);
  int arrived = 0;
  if (lane == 0) {
    for (int it = 0; it < a.spin_limit; ++it) {
      if (__hip_atomic_load(a.step_arrivals, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= a.total_wgs) {
        arrived = 1;
        break;
      }
      __builtin_amdgcn_s_sleep(8);
    }
  }
  arrived = __shfl(arrived, 0, kWave);
  if (arrived && po.ok) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int t = lane + 64 * k;
      if (t < a.n) {
        const int s = pr.sk[k], L = pr.Lk[k];
        if (po.pop[k] >= 0) a.block_table_w[(int64_t)s * a.max_blocks + (L >> a.bs_log2)] = po.pop[k];
        a.lengths_w[s] = L + 1;
      }
    }
  }
  if (lane == 0) {
    if (arrived && po.ok) *a.free_top = pr.top - po.total;
    int bits = __hip_atomic_load(a.step_err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) | po.bits;
    if (!arrived) bits |= SM_ERR_EINVAL;  // not reached while every workgroup arrives
    if (bits) set_err(a.err, bits);
    __hip_atomic_store(a.step_err, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(a.step_arrivals, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// The plan of a decode-time merge step (one wave, registers only, lane l
// holding requests l + 64 k): crop c_t entries of request t, then append
// its one row, as one update that is made whole or not at all.  The checks
// come in the order of the two operations: ids (in range, no repeats) and
// c_t >= 0, else EINVAL; 0 <= L_t <= capacity and c_t <= L_t, then room on
// the free stack for every freed block, then L_t - c_t + 1 <= capacity,
// else ERANGE; enough free blocks after the crop, else ENOMEM; every block
// popped a valid id, else EINVAL.  The crop pushes request t's freed pages
// (pages of entries >= L_t - c_t) onto the free stack, highest page first,
// requests in reverse order; the append then pops, requests in order, one
// block for each request whose cropped length ends a page.  So the c-th
// pop takes, while c <= F (the blocks all crops free), the c-th freed page
// in the order (request 0's pages ascending, then request 1's, ...), and
// after that the old stack's entry top - 1 - (c - F - 1).
struct PlanOutC {
  bool ok;      // the update commits
  int bits;     // its error bits (0 when the error word was set)
  int total;    // blocks popped
  int freed;    // blocks pushed by the crops
  int need[4];  // per request of this lane: a block is popped for it
  int pop[4];   // ... and which one (or -1)
  int F[4];     // blocks its crop frees
  int E[4];     // blocks freed by the requests before it
  int Lc[4];    // its length after the crop
};

__device__ __forceinline__ int blocks_for_len(int L, int bs_log2) { return (L + (1 << bs_log2) - 1) >> bs_log2; }

// Inclusive prefix sum over the wave's lanes.
__device__ __forceinline__ int wave_incl_scan(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int u = __shfl_up(v, d, kWave);
    if (lane >= d) v += u;
  }
  return v;
}

__device__ void plan_crop(const DecodeArgs &a, const PlanRegs &pr, PlanOutC &po, uint32_t *bm) {
  const int lane = threadIdx.x & 63, n = a.n, bsl = a.bs_log2;
  const bool any_dup = wave_any_dup(a, pr.sk, bm);
  int inval = 0, range = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int t = lane + 64 * k, sk = pr.sk[k], Lk = pr.Lk[k], ck = pr.ck[k];
    po.need[k] = 0;
    po.F[k] = 0;
    po.Lc[k] = 0;
    if (t < n) {
      if (sk < 0 || sk >= a.max_seqs || any_dup || ck < 0) inval = 1;
      else if (Lk < 0 || (int64_t)Lk > a.cap || ck > Lk) range = 1;
      else {
        const int Lc = Lk - ck;
        po.Lc[k] = Lc;
        po.F[k] = blocks_for_len(Lk, bsl) - blocks_for_len(Lc, bsl);
        if ((int64_t)Lc + 1 > a.cap) range = 1;
        po.need[k] = (Lc & ((1 << bsl) - 1)) == 0;
      }
    }
  }
  const bool any_inval = __ballot(inval) != 0;
  const bool any_range = __ballot(range) != 0;
  int incl[4] = {0, 0, 0, 0}, total = 0, freed = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {  // prefixes in request order
    if (64 * k < n) {
      const uint64_t m = __ballot(po.need[k]);
      const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
      incl[k] = total + below + po.need[k];
      total += __popcll(m);
      const int f_incl = wave_incl_scan(po.F[k]);
      po.E[k] = freed + f_incl - po.F[k];
      freed += __shfl(f_incl, 63, kWave);
    } else {
      po.E[k] = freed;
    }
  }
  const int top = pr.top;
  int bits = any_inval ? SM_ERR_EINVAL
             : (any_range || top < 0 || (int64_t)top + freed > a.num_blocks) ? SM_ERR_ERANGE
             : (total > top + freed) ? SM_ERR_ENOMEM
                                     : 0;
  const bool go = !pr.frozen && bits == 0;
  // pops of freed pages: the owner of the c-th freed page, looked up over
  // the requests whose crop frees any
  int own_s[4] = {-1, -1, -1, -1}, own_pg[4] = {0, 0, 0, 0};
  if (go && freed > 0) {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      if (64 * kk < n) {
        uint64_t m = __ballot(po.F[kk] > 0);
        while (m) {
          const int jl = __builtin_ctzll(m);
          m &= m - 1;
          const int Ej = __builtin_amdgcn_readlane(po.E[kk], jl), Fj = __builtin_amdgcn_readlane(po.F[kk], jl);
          const int sj = __builtin_amdgcn_readlane(pr.sk[kk], jl), Lcj = __builtin_amdgcn_readlane(po.Lc[kk], jl);
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const int cidx = incl[k];
            if (po.need[k] && cidx > Ej && cidx <= Ej + Fj) {
              own_s[k] = sj;
              own_pg[k] = blocks_for_len(Lcj, bsl) + (cidx - Ej - 1);
            }
          }
        }
      }
    }
  }
  int bad = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    po.pop[k] = -1;
    if (64 * k < n) {
      const bool popped = go && po.need[k];
      // from the old stack: entry incl - freed - 1 < total - freed <= min(top, n) of the window
      const int widx = (popped && incl[k] > freed) ? incl[k] - freed - 1 : 0;
      int blk = __shfl(pr.win[0], widx & 63, kWave);
      if (total > 64) {
        const int w1 = __shfl(pr.win[1], widx & 63, kWave);
        const int w2 = __shfl(pr.win[2], widx & 63, kWave), w3 = __shfl(pr.win[3], widx & 63, kWave);
        const int q = widx >> 6;
        blk = q == 0 ? blk : q == 1 ? w1 : q == 2 ? w2 : w3;
      }
      if (popped && incl[k] <= freed)
        blk = own_s[k] >= 0 ? a.block_table[(int64_t)own_s[k] * a.max_blocks + own_pg[k]] : -1;
      po.pop[k] = popped ? blk : -1;
      if (popped && (blk < 0 || blk >= a.num_blocks)) bad = 1;
    }
  }
  const bool any_stack = __ballot(bad) != 0;
  if (go && any_stack) bits = SM_ERR_EINVAL;  // corrupt free stack or block table
  po.ok = go && !any_stack;
  po.bits = pr.frozen ? 0 : bits;
  po.total = total;
  po.freed = freed;
}

// The commit wave of a decode-time merge step: as step_commit_wave, and
// the crops' writes before the append's: the freed pages' block ids go onto
// the free stack (request t's at top + freed - E_t - F_t onward, highest
// page first) and their table entries become -1; then each popped block
// enters its request's table, lengths become L_t - c_t + 1 and the stack top
// top + freed - popped.
__device__ void step_commit_wave_crop(const DecodeArgs &a, uint32_t *bm) {
  const int lane = threadIdx.x & 63, bsl = a.bs_log2;
  PlanRegs pr;
  step_plan_read1<true>(a, pr);
  step_plan_read2(a, pr);
  PlanOutC po;
  plan_crop(a, pr, po, bm);
  int arrived = 0;
  if (lane == 0) {
    for (int it = 0; it < a.spin_limit; ++it) {
      if (__hip_atomic_load(a.step_arrivals, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= a.total_wgs) {
        arrived = 1;
        break;
      }
      __builtin_amdgcn_s_sleep(8);
    }
  }
  arrived = __shfl(arrived, 0, kWave);
  if (arrived && po.ok) {
    // push slot p of [0, freed) (stack entry top + p) holds the c-th freed
    // page in pop order, c = freed - p; a lane takes four slots at a time:
    // owners found, the table entries read, then the stack written and the
    // entries cleared (all reads before any write)
    for (int p0 = 0; p0 < po.freed; p0 += 4 * kWave) {
      int own_s[4] = {-1, -1, -1, -1}, own_pg[4] = {0, 0, 0, 0};
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        if (64 * kk < a.n) {
          uint64_t m = __ballot(po.F[kk] > 0);
          while (m) {
            const int jl = __builtin_ctzll(m);
            m &= m - 1;
            const int Ej = __builtin_amdgcn_readlane(po.E[kk], jl), Fj = __builtin_amdgcn_readlane(po.F[kk], jl);
            const int sj = __builtin_amdgcn_readlane(pr.sk[kk], jl), Lcj = __builtin_amdgcn_readlane(po.Lc[kk], jl);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int cidx = po.freed - (p0 + lane + kWave * r);
              if (cidx > Ej && cidx <= Ej + Fj) {
                own_s[r] = sj;
                own_pg[r] = blocks_for_len(Lcj, bsl) + (cidx - Ej - 1);
              }
            }
          }
        }
      }
      int blk[4];
#pragma unroll
      for (int r = 0; r < 4; ++r)
        blk[r] = own_s[r] >= 0 ? a.block_table_w[(int64_t)own_s[r] * a.max_blocks + own_pg[r]] : -1;
      __builtin_amdgcn_s_waitcnt(0);  // every read of the table before its entries are cleared
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if (own_s[r] >= 0) {
          a.free_stack[pr.top + p0 + lane + kWave * r] = blk[r];
          a.block_table_w[(int64_t)own_s[r] * a.max_blocks + own_pg[r]] = -1;
        }
      }
      __builtin_amdgcn_s_waitcnt(0);  // cleared before the pops are written (a pop may land on one)
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int t = lane + 64 * k;
      if (t < a.n) {
        const int s = pr.sk[k], Lc = po.Lc[k];
        if (po.pop[k] >= 0) a.block_table_w[(int64_t)s * a.max_blocks + (Lc >> bsl)] = po.pop[k];
        a.lengths_w[s] = Lc + 1;
      }
    }
  }
  if (lane == 0) {
    if (arrived && po.ok) *a.free_top = pr.top + po.freed - po.total;
    int bits = __hip_atomic_load(a.step_err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) | po.bits;
    if (!arrived) bits |= SM_ERR_EINVAL;  // not reached while every workgroup arrives
    if (bits) set_err(a.err, bits);
    __hip_atomic_store(a.step_err, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(a.step_arrivals, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// An attention workgroup of a fused step is done with the metadata: park
// its error bits (waiting for that atomic, so that they are in before the
// count) and count it.  Thread 0 only.
__device__ __forceinline__ void step_arrive_nowait(const DecodeArgs &a, int errs) {
  if (errs) {
    const int prev = __hip_atomic_fetch_or(a.step_err, errs, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __builtin_amdgcn_s_waitcnt(0);
    (void)prev;
  }
  __hip_atomic_fetch_add(a.step_arrivals, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Thread 0 parks this workgroup's error bits and arrives; returns the
// arrival ticket (the workgroup whose ticket is total_wgs - 1 commits).
__device__ __forceinline__ int step_arrive(const DecodeArgs &a, int errs) {
  if (errs) __hip_atomic_fetch_or(a.step_err, errs, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __builtin_amdgcn_s_waitcnt(0);  // the bits are in before the arrival counts
  return __hip_atomic_fetch_add(a.step_arrivals, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Run by the workgroup holding the last ticket, after its own work: every
// other workgroup has finished reading the metadata.
__device__ void step_commit(const DecodeArgs &a, StepShared &sp, bool ok) {
  const int t = threadIdx.x;
  if (ok && t < a.n) {
    const int s = sp.ids[t], L = sp.len[t];
    if (sp.pop[t] >= 0) a.block_table_w[(int64_t)s * a.max_blocks + (L >> a.bs_log2)] = sp.pop[t];
    a.lengths_w[s] = L + 1;
  }
  if (t == 0) {
    if (ok) *a.free_top = sp.top - sp.total;
    int bits = __hip_atomic_load(a.step_err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (!sp.frozen) bits |= sp.bits;
    if (bits) set_err(a.err, bits);
    __hip_atomic_store(a.step_err, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(a.step_arrivals, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// This workgroup's view of its request: attention status and the chunking
// length (the appended length when the append passes phases 1-2; if the
// stack check then fails the new token is simply not folded in).
__device__ __forceinline__ void step_request(const DecodeArgs &a, const StepShared &sp, int i, int &s,
                                             int &L_old, int &L_c, int &st) {
  s = sp.ids[i];
  L_old = sp.len[i];
  st = 0;
  if (s < 0 || s >= a.max_seqs || L_old < 0 || L_old > (a.max_blocks << a.bs_log2)) {
    st = SM_ERR_EINVAL;
    L_c = 0;
    return;
  }
  L_c = L_old + ((!sp.frozen && sp.bits == 0) ? 1 : 0);
  if (L_c > a.max_len) st = SM_ERR_ERANGE;
}

// ---------------------------------------------------------------------------
// bf16 split kernel (matrix cores)

template <int DH>
struct KVTile {
  u32x4_t ka[DH / 32];  // K rows of score tile A (16 tokens x 8 dims / lane)
  u32x4_t kb[DH / 32];  // K rows of score tile B
  u32x4_t v[DH / 16];   // V^T: 16 dims x 8 tokens per lane
};

// ORD: the grid takes the (request, kv head) pairs in length order (see
// order_pick); a separate instantiation, so that the grid-order kernels
// carry none of its code.
// CROP (with STEP): the decode-time merge step; the crops and the append
// are planned before the streaming loop, since they decide what is read.
template <int DH, bool STEP, bool ORD, bool CROP = false>
__global__ __launch_bounds__(kDecThreads, 2) void decode_split_bf16(DecodeArgs a) {
  __shared__ int pages[kMaxChunkPages];
  __shared__ int flag;
  __shared__ float red_m[kDecWaves][16];
  __shared__ float red_l[kDecWaves][16];
  __shared__ float red_o[kDecWaves][16][DH];
  __shared__ float step_sn[16];       // fused step: scaled score of the new token per query head
  __shared__ float step_vn[DH];       // ... and its V row
  __shared__ int step_bad_page[kDecWaves];
  __shared__ int step_plan_sh[3];     // ... the append commits; block popped for this request; its crop
  __shared__ uint32_t dup_bm[STEP ? kDupBitmapWords : 1];  // the plan's duplicate-id check (one wave)

  const int c = blockIdx.x;
  int g = blockIdx.y, i = blockIdx.z;  // (request, kv head): grid position, or by length order
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int bs_log2 = a.bs_log2, bs = 1 << bs_log2;
  int s = 0, L = 0, st = 0, L_pool = 0;  // chunking covers [0, L), the pool holds [0, L_pool)
  const bool ordered = ORD && i < a.order_n;  // (the step's commit row is not)
  int s_ord = 0, L_ord = 0;
  __shared__ int64_t ord_key[ORD ? kDecThreads : 1];
  __shared__ int ord_sid[ORD ? kDecThreads : 1], ord_pick[1];
  int nc = 0, chunk = 0, t0 = 0, t1 = 0, lp0 = 0, npages = 0;
  bool work = false, pages_ok = true;

  // fused step state (all uniform over the workgroup)
  PlanRegs pr;
  bool has_new = false;   // this chunk holds the new position (if the append commits)
  bool may_write = false; // this workgroup stores the new row (if the append commits)
  bool late = false;      // new length = max_len + 1 exactly: ERANGE iff the append commits
  bool own_can = false;
  uint32_t kn2 = 0u, qn2[4] = {0u, 0u, 0u, 0u};  // the new token's score inputs (bf16 pairs)
  uint16_t krow_e = 0, vrow_e = 0;
  int32_t *esink = a.err;

  if constexpr (STEP) {
    if (i == a.n) {  // the commit workgroup; the rest of this grid row has nothing to do
      if (c == 0 && g == 0 && w == 0) {
        if constexpr (CROP) step_commit_wave_crop(a, dup_bm);
        else step_commit_wave(a, dup_bm);
      }
      return;
    }
    esink = nullptr;  // errors travel with the arrival
    // wave 3 (no page ids to fetch at these sizes) issues the reads the
    // append's plan needs, two round trips beside the other waves' chain of
    // this request's id, length and page ids; the plan itself is worked
    // out after the streaming loop, where it is first needed
    if (w == kDecWaves - 1) step_plan_read1<CROP>(a, pr);
    if constexpr (ORD)
      if (ordered) order_pick(a, g, i, s_ord, L_ord, ord_key, ord_sid, ord_pick);
    s = ordered ? s_ord : a.seq_ids[i];
    const int frozen = *a.err != 0;
    const bool own_ok = s >= 0 && s < a.max_seqs;
    if (w == kDecWaves - 1) step_plan_read2(a, pr);
    L_pool = own_ok ? (ordered ? L_ord : a.lengths[s]) : 0;
    if (!own_ok || L_pool < 0 || L_pool > (a.max_blocks << bs_log2)) st = SM_ERR_EINVAL;
    if constexpr (CROP) {
      // whether the crops and the append commit decides what this request
      // attends over: its first L - c entries and the new row, or its
      // unchanged cache; wave 3 works the plan out now and publishes it
      if (w == kDecWaves - 1) {
        PlanOutC po;
        plan_crop(a, pr, po, dup_bm);
        const int pop_i = request_value(po.pop, i), ck_i = request_value(pr.ck, i);
        if (lane == 0) {
          step_plan_sh[0] = po.ok;
          step_plan_sh[1] = pop_i;
          step_plan_sh[2] = ck_i;
        }
      }
      lds_barrier();
      own_can = step_plan_sh[0] != 0;  // (then every request passed its checks)
      if (own_can) L_pool -= step_plan_sh[2];
    } else {
      own_can = !frozen && st == 0 && (int64_t)L_pool + 1 <= a.cap;
    }
    if (st == 0) {  // chunked for the appended length whenever this request can append
      if (own_can && L_pool + 1 <= a.max_len) L = L_pool + 1;
      else {
        L = L_pool;
        if (L_pool > a.max_len) st = SM_ERR_ERANGE;
        else late = own_can;
      }
    }
    work = st == 0 && L > 0;
    if (work) {
      chunking(L, a.chunk_nominal, nc, chunk);
      work = c < nc;
    }
    int bad_page = 0;
    if (work) {
      t0 = c * chunk;
      t1 = min(L, t0 + chunk);
      has_new = L > L_pool && t0 <= L_pool && L_pool < t1;
      const int t1p = min(t1, L_pool);
      lp0 = t0 >> bs_log2;
      npages = t1p > t0 ? ((t1p - 1) >> bs_log2) - lp0 + 1 : 0;
      for (int p = tid; p < npages; p += kDecThreads) {
        int blk = a.block_table[(int64_t)s * a.max_blocks + lp0 + p];
        if (blk < 0 || blk >= a.num_blocks) {
          bad_page = 1;
          blk = 0;
        }
        pages[p] = blk;
      }
    }
    // the new token's score inputs and rows: lane l of wave w takes dims
    // l, l + 64 of query heads w, w + 4, ...
    const uint16_t *kn = (const uint16_t *)a.k_new + ((int64_t)i * a.Hkv + g) * DH;
    const uint16_t *vn = (const uint16_t *)a.v_new + ((int64_t)i * a.Hkv + g) * DH;
    if (has_new && 2 * lane < DH) {  // loaded now, multiplied after the streaming loop
      const uint16_t *qg = (const uint16_t *)a.q + ((int64_t)i * a.Hq + g * a.G) * DH + 2 * lane;
      kn2 = *(const uint32_t *)(kn + 2 * lane);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int hh = w + kDecWaves * u;
        qn2[u] = hh < a.G ? *(const uint32_t *)(qg + hh * DH) : 0u;
      }
    }
    may_write = own_can && (has_new || (c == 0 && (st == SM_ERR_ERANGE || late)));
    if (may_write && tid < DH) {
      krow_e = kn[tid];
      vrow_e = vn[tid];
    }
    {
      const bool wave_bad = __ballot(bad_page) != 0;
      if (lane == 0) step_bad_page[w] = wave_bad;
    }
    // the new row's loads stay in flight: they are consumed after the loop
    lds_barrier();
#pragma unroll
    for (int ww = 0; ww < kDecWaves; ++ww) pages_ok = pages_ok && !step_bad_page[ww];
  } else {
    if constexpr (ORD)
      if (ordered) order_pick(a, g, i, s_ord, L_ord, ord_key, ord_sid, ord_pick);
    s = ordered ? s_ord : a.seq_ids[i];
    st = seq_status(a, s, L, ordered, L_ord);
    L_pool = L;
    work = st == 0 && L > 0;
    if (work) {
      chunking(L, a.chunk_nominal, nc, chunk);
      work = c < nc;
    }
    if (work) {
      t0 = c * chunk;
      t1 = min(L, t0 + chunk);
      lp0 = t0 >> bs_log2;
      const int npg = ((t1 - 1) >> bs_log2) - lp0 + 1;
      pages_ok = load_pages(a, s, lp0, npg, pages, &flag);
    }
  }

  // Fused step, after the streaming loop (or right away for a workgroup
  // that streams nothing): wave 3 works out the plan from the reads it
  // issued in the prologue and publishes it, then every wave decides this
  // workgroup's share of the append.  The new row's stores and the arrival
  // follow (stores and atomics count in the same wait counter as loads, so
  // issued before the tile loads they would hold up the first tile waits).
  bool step_ok = false, late_range = false;
  int step_errs = 0, new_blk = -1;
  auto step_decide = [&]() __attribute__((always_inline)) {
    step_ok = step_plan_sh[0] != 0;
    has_new = has_new && step_ok;
    late_range = late && step_ok;
    const bool writes_row = may_write && step_ok;
    step_errs = st | (late_range ? SM_ERR_ERANGE : 0);
    if (work && !pages_ok) step_errs |= SM_ERR_EINVAL;
    if (writes_row) {  // the new row's block: popped, or the tail page's
      new_blk = step_plan_sh[1];
      if (new_blk < 0) {
        const int tp = L_pool >> bs_log2;
        new_blk = (work && pages_ok && tp >= lp0 && tp < lp0 + npages)
                      ? pages[tp - lp0]
                      : a.block_table[(int64_t)s * a.max_blocks + tp];
      }
      if (new_blk < 0 || new_blk >= a.num_blocks) {
        step_errs |= SM_ERR_EINVAL;  // corrupt block table: the row is not written
        new_blk = -1;
      }
    }
  };
  auto step_plan_decide = [&]() __attribute__((always_inline)) {
    if constexpr (CROP) {  // planned and published in the prologue
      step_decide();
    } else {
      if (w == kDecWaves - 1) {
        PlanOut po;
        plan_any(a, pr, po, dup_bm);
        const int pop_i = request_value(po.pop, i);
        if (lane == 0) {
          step_plan_sh[0] = po.ok;
          step_plan_sh[1] = pop_i;
        }
      }
      lds_barrier();
      step_decide();
    }
  };
  auto step_finish = [&]() __attribute__((always_inline)) {
    if (new_blk >= 0 && tid < DH) {  // the appended row of head g into its page
      const int64_t page_elems = (int64_t)bs * DH;
      const int slot = L_pool & (bs - 1);
      uint16_t *kd = (uint16_t *)a.k_pool + ((int64_t)new_blk * a.Hkv + g) * page_elems + (int64_t)slot * DH;
      uint16_t *vd = (uint16_t *)a.v_pool + ((int64_t)new_blk * a.Hkv + g) * page_elems + slot;
      // streaming stores: the scattered 2-byte V row is not left dirty in L2
      // for the end-of-kernel writeback
      __builtin_nontemporal_store(krow_e, kd + tid);
      __builtin_nontemporal_store(vrow_e, vd + (int64_t)tid * bs);
    }
    if (tid == 0) step_arrive_nowait(a, step_errs);
    if (has_new) {
      const float k0 = __uint_as_float(kn2 << 16), k1 = __uint_as_float(kn2 & 0xffff0000u);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int hh = w + kDecWaves * u;
        const float kq = __uint_as_float(qn2[u] << 16) * k0 + __uint_as_float(qn2[u] & 0xffff0000u) * k1;
        const float d = wave_sum(kq);
        if (hh < a.G && lane == 0) step_sn[hh] = d * a.scale_log2e;
      }
      if (tid < DH) step_vn[tid] = bf16_to_f32(vrow_e);
    }
  };

  auto body = [&]() {
    if constexpr (STEP) {
      if (!(st == 0 && L > 0 && work && pages_ok)) {
        step_plan_decide();
        if (late_range) st = SM_ERR_ERANGE;  // zero rows; the bit travels with the arrival
        step_finish();
      }
    }
    if (st != 0 || L == 0) {
      if (c == 0) write_zero_rows<uint16_t>(a, i, g, DH, st, esink);
      return;
    }
    if (!work) return;
    if (!pages_ok) {
      write_bad_partial(a, i, g, c, esink);
      finish_group<uint16_t>(a, i, g, nc, DH, &flag);
      return;
    }
    const int t1p = min(t1, L_pool);  // pool entries of this chunk: [t0, t1p)
    const int r = lane & 15;   // score-tile row / head column / V dim row
    const int q4 = lane >> 4;  // k-slot group of the MFMA operands
    const int G = a.G;

    // Q^T operand: lane (r, q4) holds q[head r][32*kk + 8*q4 .. +7]
    u32x4_t qreg[DH / 32];
    {
      const uint16_t *qb = (const uint16_t *)a.q + ((int64_t)i * a.Hq + g * G + r) * DH + 8 * q4;
#pragma unroll
      for (int kk = 0; kk < DH / 32; ++kk)
        qreg[kk] = (r < G) ? *(const u32x4_t *)(qb + 32 * kk) : u32x4_t{0u, 0u, 0u, 0u};
    }

    const uint16_t *kp = (const uint16_t *)a.k_pool;
    const uint16_t *vp = (const uint16_t *)a.v_pool;
    const int64_t page_elems = (int64_t)bs * DH;  // one (block, head) page
    const int offA = 8 * (r >> 2) + (r & 3);      // token of score-tile A row r
    const int offB = offA + 4;                     // token of score-tile B row r
    const int offV = 8 * q4;                       // first of this lane's 8 tokens
    const int ntiles = t1p > t0 ? (t1p - t0 + 31) >> 5 : 0;

    auto load = [&](KVTile<DH> &T, int tile) {
      const int T0 = t0 + 32 * tile;
      // tokens past the pool range read the chunk's first entry instead
      // (their scores are masked and their V lanes zeroed below)
      const int tA = (T0 + offA < t1p) ? T0 + offA : t0;
      const int tB = (T0 + offB < t1p) ? T0 + offB : t0;
      const int tV = (T0 + offV < t1p) ? T0 + offV : t0;
      const int bA = pages[(tA >> bs_log2) - lp0];
      const int bB = pages[(tB >> bs_log2) - lp0];
      const int bV = pages[(tV >> bs_log2) - lp0];
      const uint16_t *pA = kp + ((int64_t)bA * a.Hkv + g) * page_elems + (tA & (bs - 1)) * DH + 8 * q4;
      const uint16_t *pB = kp + ((int64_t)bB * a.Hkv + g) * page_elems + (tB & (bs - 1)) * DH + 8 * q4;
      const uint16_t *pV = vp + ((int64_t)bV * a.Hkv + g) * page_elems + (int64_t)r * bs + (tV & (bs - 1));
#pragma unroll
      for (int kk = 0; kk < DH / 32; ++kk) {
        T.ka[kk] = __builtin_nontemporal_load((const u32x4_t *)(pA + 32 * kk));
        T.kb[kk] = __builtin_nontemporal_load((const u32x4_t *)(pB + 32 * kk));
      }
#pragma unroll
      for (int dt = 0; dt < DH / 16; ++dt)
        T.v[dt] = __builtin_nontemporal_load((const u32x4_t *)(pV + (int64_t)16 * dt * bs));
    };

    f32x4_t o[DH / 16];
#pragma unroll
    for (int dt = 0; dt < DH / 16; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;
    const float sl2 = a.scale_log2e;

    auto compute = [&](KVTile<DH> &T, int tile) {
      const int T0 = t0 + 32 * tile;
      f32x4_t sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < DH / 32; ++kk) {
        sa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(T.ka[kk]), as_bf16x8(qreg[kk]), sa, 0, 0, 0);
        sb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(T.kb[kk]), as_bf16x8(qreg[kk]), sb, 0, 0, 0);
      }
      // lane (r, q4) now holds head r's scores of tokens T0 + 8*q4 + 0..7
      float sc[8] = {sa[0], sa[1], sa[2], sa[3], sb[0], sb[1], sb[2], sb[3]};
      const int nvalid = min(8, max(0, t1p - (T0 + offV)));
#pragma unroll
      for (int j = 0; j < 8; ++j) sc[j] = (j < nvalid) ? sc[j] * sl2 : -INFINITY;
      float mx = sc[0];
#pragma unroll
      for (int j = 1; j < 8; ++j) mx = fmaxf(mx, sc[j]);
      {
        float a, b;
        swap16(mx, a, b);
        swap32(fmaxf(a, b), a, b);
        mx = fmaxf(a, b);
      }
      const float m_new = fmaxf(m_run, mx);  // finite: every tile has a valid token
      const float alpha = exp2f(m_run - m_new);
      float p[8], ps = 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        p[j] = exp2f(sc[j] - m_new);
        ps += p[j];
      }
      l_run = l_run * alpha + ps;
      m_run = m_new;
#pragma unroll
      for (int dt = 0; dt < DH / 16; ++dt) o[dt] *= alpha;
      if (nvalid < 8) {  // stale slots past the end may hold anything
#pragma unroll
        for (int dt = 0; dt < DH / 16; ++dt) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            uint32_t word = T.v[dt][e];
            if (2 * e >= nvalid) word = 0u;
            else if (2 * e + 1 >= nvalid) word &= 0xffffu;
            T.v[dt][e] = word;
          }
        }
      }
      const u32x4_t pp = {pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]),
                          pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7])};
#pragma unroll
      for (int dt = 0; dt < DH / 16; ++dt)
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(T.v[dt]), as_bf16x8(pp), o[dt], 0, 0, 0);
    };

    // two register buffers, alternating without copies: while one tile is
    // multiplied the next one's 16 loads are in flight
    KVTile<DH> bufA, bufB;
    constexpr int step = kDecWaves;
    if (w < ntiles) load(bufA, w);
    for (int tile = w; tile < ntiles; tile += 2 * step) {
      if (tile + step < ntiles) load(bufB, tile + step);
      compute(bufA, tile);
      if (tile + step >= ntiles) break;
      if (tile + 2 * step < ntiles) load(bufA, tile + 2 * step);
      compute(bufB, tile + step);
    }
    if constexpr (STEP) {
      // a request whose appended length reaches max_len + 1 streamed its
      // old length; once the append is known to commit it gets zero rows
      // and ERANGE, carried as an unusable partial into the combine
      step_plan_decide();
      step_finish();
    }

    // per-head totals of this wave (lanes r, r+16, r+32, r+48 share head r)
    float l_tot;
    {
      float a, b;
      swap16(l_run, a, b);
      swap32(a + b, a, b);
      l_tot = a + b;
    }
    if (q4 == 0) {
      red_m[w][r] = m_run;
      red_l[w][r] = l_tot;
    }
#pragma unroll
    for (int dt = 0; dt < DH / 16; ++dt)
#pragma unroll
      for (int j = 0; j < 4; ++j) red_o[w][r][16 * dt + 4 * q4 + j] = o[dt][j];
    // LDS only: the fused step's row stores and arrival need not land first
    lds_barrier();

    for (int e = tid; e < G * DH; e += kDecThreads) {
      const int hh = e / DH, dd = e - hh * DH;
      float M = red_m[0][hh];
#pragma unroll
      for (int ww = 1; ww < kDecWaves; ++ww) M = fmaxf(M, red_m[ww][hh]);
      // a chunk with no cached entries (only the appended one) leaves every
      // wave at -inf: rescale against 0 so that they all contribute 0
      const float Mb = M == -INFINITY ? 0.f : M;
      float acc = 0.f, ls = 0.f;
#pragma unroll
      for (int ww = 0; ww < kDecWaves; ++ww) {
        const float f = exp2f(red_m[ww][hh] - Mb);  // idle waves: exp2(-inf) = 0
        acc += red_o[ww][hh][dd] * f;
        ls += red_l[ww][hh] * f;
      }
      if constexpr (STEP) {
        if (has_new) {  // fold in the appended token
          const float sN = step_sn[hh];
          const float M2 = fmaxf(M, sN);
          const float f = exp2f(M - M2), fN = exp2f(sN - M2);
          acc = acc * f + step_vn[dd] * fN;
          ls = ls * f + fN;
          M = M2;
        }
      }
      if constexpr (STEP) {
        if (late_range) {
          M = 0.f;
          ls = -1.f;  // marks the chunk as unusable: the group's rows become zero
        }
      }
      if (nc == 1) {  // the only chunk: write the result directly
        ((uint16_t *)a.out)[((int64_t)i * a.Hq + g * G + hh) * DH + dd] = f32_to_bf16(ls > 0.f ? acc / ls : 0.f);
        continue;
      }
      const int64_t pidx = ((int64_t)i * a.Hq + g * G + hh) * a.max_chunks + c;
      put_partial(&a.ws_o[pidx * DH + dd], acc);
      if (dd == 0) {
        put_partial(&a.ws_ml[pidx * 2 + 0], M);
        put_partial(&a.ws_ml[pidx * 2 + 1], ls);
      }
    }
    if (nc > 1) finish_group<uint16_t>(a, i, g, nc, DH, &flag);
  };
  body();
}

// ---------------------------------------------------------------------------
// fp32 split kernel (vector ALU; chunks of at most 256 tokens, one token per
// thread for the scores)

template <int DH, bool STEP>
__global__ __launch_bounds__(kDecThreads) void decode_split_f32(DecodeArgs a) {
  __shared__ int pages[kF32ChunkTokens / 16 + 2];
  __shared__ int flag;
  __shared__ float qs[DH];
  __shared__ float ps[kF32ChunkTokens];
  __shared__ float red[kDecWaves];
  constexpr int NG = kDecThreads / DH;  // token groups for the PV sums
  __shared__ float opart[NG][DH];
  __shared__ StepShared sp;

  const int c = blockIdx.x, g = blockIdx.y, i = blockIdx.z;
  const int tid = threadIdx.x;
  const int bs_log2 = a.bs_log2, bs = 1 << bs_log2;
  int32_t *esink = a.err;
  int s = 0, L = 0, st = 0, L_pool = 0;  // chunking covers [0, L), the pool holds [0, L_pool)
  int nc = 0, chunk = 0, t0 = 0, t1 = 0;
  bool work = false, pages_ok = true, step_ok = false, has_new = false;
  int ticket = 0;

  if constexpr (STEP) {
    esink = &sp.errs;
    int need_t;
    const int incl = step_plan(a, sp, need_t);
    step_request(a, sp, i, s, L_pool, L, st);
    work = st == 0 && L > 0;
    if (work) {
      chunking(L, a.chunk_nominal, nc, chunk);
      work = c < nc;
    }
    int lp0 = 0, npages = 0;
    // the workgroup storing the appended row of head g: the one whose chunk
    // holds the new position, or chunk 0 when the sequence gets no
    // attention because its new length exceeds max_len
    bool writes_row = false;
    if (work) {
      t0 = c * chunk;
      t1 = min(L, t0 + chunk);
      has_new = L > L_pool && t0 <= L_pool && L_pool < t1;
      writes_row = has_new;
      const int t1p = min(t1, L_pool);
      lp0 = t0 >> bs_log2;
      npages = t1p > t0 ? ((t1p - 1) >> bs_log2) - lp0 + 1 : 0;
    } else {
      writes_row = c == 0 && st == SM_ERR_ERANGE && !sp.frozen && sp.bits == 0;
    }
    const bool want_tail = writes_row && (L_pool & (bs - 1)) != 0;
    pages_ok = step_pages(a, sp, incl, need_t, i, s, lp0, npages, want_tail, pages, step_ok);
    has_new = has_new && step_ok;
    writes_row = writes_row && step_ok;
    int errs = st, new_blk = -1;
    if (work && !pages_ok) errs |= SM_ERR_EINVAL;
    if (writes_row) {  // the new row's block: popped, or the tail page's
      new_blk = sp.pop[i] >= 0 ? sp.pop[i] : sp.tail;
      if (new_blk < 0 || new_blk >= a.num_blocks) {
        errs |= SM_ERR_EINVAL;  // corrupt block table: the row is not written
        new_blk = -1;
      }
    }
    if (tid == 0) ticket = step_arrive(a, errs);
    if (writes_row && new_blk >= 0) {  // the appended row of head g into its page
      const int64_t page_elems = (int64_t)bs * DH;
      const int slot = L_pool & (bs - 1);
      const float *kn = (const float *)a.k_new + ((int64_t)i * a.Hkv + g) * DH;
      const float *vn = (const float *)a.v_new + ((int64_t)i * a.Hkv + g) * DH;
      float *kd = (float *)a.k_pool + ((int64_t)new_blk * a.Hkv + g) * page_elems + (int64_t)slot * DH;
      float *vd = (float *)a.v_pool + ((int64_t)new_blk * a.Hkv + g) * page_elems + slot;
      for (int e = tid; e < DH; e += kDecThreads) {
        kd[e] = kn[e];
        vd[(int64_t)e * bs] = vn[e];
      }
    }
  } else {
    s = a.seq_ids[i];
    st = seq_status(a, s, L);
    L_pool = L;
    work = st == 0 && L > 0;
    if (work) {
      chunking(L, a.chunk_nominal, nc, chunk);
      work = c < nc;
    }
    if (work) {
      t0 = c * chunk;
      t1 = min(L, t0 + chunk);
      const int lp0 = t0 >> bs_log2;
      const int npages = ((t1 - 1) >> bs_log2) - lp0 + 1;
      pages_ok = load_pages(a, s, lp0, npages, pages, &flag);
    }
  }

  auto body = [&]() {
    if (st != 0 || L == 0) {
      if (c == 0) write_zero_rows<float>(a, i, g, DH, st, esink);
      return;
    }
    if (!work) return;
    if (!pages_ok) {
      write_bad_partial(a, i, g, c, esink);
      finish_group<float>(a, i, g, nc, DH, &flag);
      return;
    }
    const int t1p = min(t1, L_pool);  // pool entries of this chunk: [t0, t1p)
    const int lp0 = t0 >> bs_log2;
    const float *kp = (const float *)a.k_pool;
    const float *vp = (const float *)a.v_pool;
    const int64_t page_elems = (int64_t)bs * DH;
    const int ntok = max(0, t1p - t0);
    const int tok = t0 + tid;
    const bool valid = tid < ntok;
    const float *krow = kp;
    if (valid) {
      const int b = pages[(tok >> bs_log2) - lp0];
      krow = kp + ((int64_t)b * a.Hkv + g) * page_elems + (int64_t)(tok & (bs - 1)) * DH;
    }
    const int dd = tid % DH, tg = tid / DH;
    const float *kn = nullptr, *vn = nullptr;
    if constexpr (STEP) {
      if (has_new) {
        kn = (const float *)a.k_new + ((int64_t)i * a.Hkv + g) * DH;
        vn = (const float *)a.v_new + ((int64_t)i * a.Hkv + g) * DH;
      }
    }

    for (int hh = 0; hh < a.G; ++hh) {
      const int hq = g * a.G + hh;
      if (tid < DH) qs[tid] = ((const float *)a.q)[((int64_t)i * a.Hq + hq) * DH + tid];
      __syncthreads();
      float sc = -INFINITY;
      if (valid) {
        float dot = 0.f;
        for (int d = 0; d < DH; ++d) dot += qs[d] * krow[d];
        sc = dot * a.scale_log2e;
      }
      float M = block_max(sc, red);
      const float p = valid ? exp2f(sc - M) : 0.f;
      float l = block_sum(p, red);
      ps[tid] = p;
      __syncthreads();
      float acc = 0.f;
      for (int t = tg; t < ntok; t += NG) {
        const int tt = t0 + t;
        const int b = pages[(tt >> bs_log2) - lp0];
        acc += ps[t] * vp[((int64_t)b * a.Hkv + g) * page_elems + (int64_t)dd * bs + (tt & (bs - 1))];
      }
      opart[tg][dd] = acc;
      float sN = 0.f;
      if constexpr (STEP) {
        if (has_new) {  // scaled score of the appended token
          float d = 0.f;
          for (int e = 0; e < DH; ++e) d += qs[e] * kn[e];
          sN = d * a.scale_log2e;
        }
      }
      __syncthreads();
      if (tid < DH) {
        float o = 0.f;
        for (int k = 0; k < NG; ++k) o += opart[k][tid];
        if constexpr (STEP) {
          if (has_new) {  // fold in the appended token
            const float M2 = fmaxf(M, sN);
            const float f = exp2f(M - M2), fN = exp2f(sN - M2);
            o = o * f + vn[tid] * fN;
            l = l * f + fN;
            M = M2;
          }
        }
        const int64_t pidx = ((int64_t)i * a.Hq + hq) * a.max_chunks + c;
        put_partial(&a.ws_o[pidx * DH + tid], o);
        if (tid == 0) {
          put_partial(&a.ws_ml[pidx * 2 + 0], M);
          put_partial(&a.ws_ml[pidx * 2 + 1], l);
        }
      }
      __syncthreads();
    }
    finish_group<float>(a, i, g, nc, DH, &flag);
  };
  body();

  if constexpr (STEP) {
    if (tid == 0) sp.last = ticket == a.total_wgs - 1;
    __syncthreads();
    if (sp.last) step_commit(a, sp, step_ok);
  }
}

}  // namespace sm

using namespace sm;

static int ilog2_exact(int v) {
  if (v <= 0 || (v & (v - 1))) return -1;
  int l = 0;
  while ((1 << l) < v) ++l;
  return l;
}

static int chunk_policy_bf16(int n, int Hkv, int max_len) {
  // One workgroup per compute unit when every sequence is at max_len (long
  // contiguous streams per workgroup measured fastest: at the 4 x 32768
  // long-context batch, 8 chunks of 2.5k entries per pair run 1.34x faster
  // than 10 of 2k; at 32 x 4915 entries one chunk per pair runs 1.09x
  // faster than three), a multiple of 128 entries (32 per wave), at least
  // 256 and at most kMaxChunkTokens (the chunk's page ids sit in LDS).
  const int64_t cus = 256;
  int64_t c = ((int64_t)max_len * n * Hkv + cus - 1) / cus;
  c = (c + 127) / 128 * 128;
  if (c < 256) c = 256;
  if (c > kMaxChunkTokens) c = kMaxChunkTokens;
  return (int)c;
}

// Workspace layout: [arrival counters, kCounterBytes][partial O][partial m, l]
constexpr int64_t kCounterBytes = 256 * 1024;
constexpr int64_t kMaxPairs = kCounterBytes / 4;  // n * num_kv_heads

SM_API size_t sm_decode_workspace_bytes(int n, int num_q_heads, int head_dim, int max_len) {
  if (n <= 0 || num_q_heads <= 0 || head_dim <= 0 || max_len < 0) return 0;
  const int64_t max_chunks = (max_len + 127) / 128 + 1;  // any chunk size >= 128
  return (size_t)(kCounterBytes + (int64_t)n * num_q_heads * max_chunks * (head_dim + 2) * sizeof(float));
}

// Shared host checks and argument setup of sm_decode_attention and
// sm_decode_step.
// With exact_ws the workspace only has to hold what this call's chunking
// uses (the scratch-array entry point); otherwise it must hold
// sm_decode_workspace_bytes for these sizes, as documented.
static sm_status decode_setup(const sm_paged_cache *c, const int32_t *seq_ids, int n, const void *q,
                              int num_q_heads, float scale, int max_len, void *out, void *ws, size_t ws_bytes,
                              int64_t max_pairs, DecodeArgs &a, bool exact_ws = false) {
  if (!c || n < 0 || max_len < 0) return SM_EINVAL;
  if (n == 0) return SM_OK;
  if (!seq_ids || !q || !out || !ws || !c->k_pool || !c->v_pool || !c->block_table ||
      !c->lengths || !c->err)
    return SM_EINVAL;
  if (c->dtype != SM_F32 && c->dtype != SM_BF16) return SM_EINVAL;
  if (c->head_dim != 64 && c->head_dim != 128) return SM_EINVAL;
  const int bs_log2 = ilog2_exact(c->block_size);
  if (bs_log2 < 4 || bs_log2 > 9) return SM_EINVAL;
  if (c->num_kv_heads <= 0 || num_q_heads <= 0 || num_q_heads % c->num_kv_heads) return SM_EINVAL;
  const int G = num_q_heads / c->num_kv_heads;
  if (G > 16) return SM_EINVAL;
  if (c->num_blocks <= 0 || c->max_seqs <= 0 || c->max_blocks_per_seq <= 0) return SM_EINVAL;
  if ((int64_t)max_len > (int64_t)c->max_blocks_per_seq * c->block_size) return SM_EINVAL;
  if (n > 65535 || (int64_t)n * c->num_kv_heads > max_pairs) return SM_EINVAL;
  if (!exact_ws && ws_bytes < sm_decode_workspace_bytes(n, num_q_heads, c->head_dim, max_len)) return SM_EINVAL;

  a = DecodeArgs{};
  a.k_pool = c->k_pool;
  a.v_pool = c->v_pool;
  a.block_table = c->block_table;
  a.lengths = c->lengths;
  a.seq_ids = seq_ids;
  a.q = q;
  a.out = out;
  a.err = c->err;
  a.Hkv = c->num_kv_heads;
  a.Hq = num_q_heads;
  a.G = G;
  a.bs_log2 = bs_log2;
  a.num_blocks = c->num_blocks;
  a.max_seqs = c->max_seqs;
  a.max_blocks = c->max_blocks_per_seq;
  a.max_len = max_len;
  a.chunk_nominal = (c->dtype == SM_BF16) ? chunk_policy_bf16(n, c->num_kv_heads, max_len)
                                          : kF32ChunkTokens;
  a.max_chunks = max_len > 0 ? (max_len + a.chunk_nominal - 1) / a.chunk_nominal : 1;
  a.scale_log2e = scale * kLog2e;
  if (exact_ws &&
      (uint64_t)ws_bytes < (uint64_t)kCounterBytes + (uint64_t)n * num_q_heads * a.max_chunks * (c->head_dim + 2) * 4)
    return SM_EINVAL;
  a.counters = (int32_t *)ws;
  a.ws_o = (float *)((char *)ws + kCounterBytes);
  a.ws_ml = a.ws_o + (int64_t)n * num_q_heads * a.max_chunks * c->head_dim;
  a.n = n;
  return SM_OK;
}

// Compute units of the current device (looked up once per device), or 0.
static int device_cus() {
  static std::atomic<int> cus[64];
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  int v = cus[dev].load(std::memory_order_relaxed);
  if (v <= 0) {
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) return 0;
    cus[dev].store(v, std::memory_order_relaxed);
  }
  return v;
}

// Workgroups of a bf16 decode kernel resident on one compute unit at once.
template <int DH, bool STEP, bool CROP>
static int bf16_occupancy() {
  static const int occ = [] {
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, decode_split_bf16<DH, STEP, true, CROP>, kDecThreads, 0) !=
        hipSuccess)
      nb = 1;
    return nb > 0 ? nb : 1;
  }();
  return occ;
}

template <bool STEP>
static sm_status decode_launch(const sm_paged_cache *c, DecodeArgs a, int n, hipStream_t stream) {
  // one launch: split, and the last workgroup of each (sequence, kv head)
  // combines; with max_len = 0 the single chunk column writes zero rows
  // a fused bf16 step adds one grid row: its first workgroup commits the append
  const int rows = n + ((STEP && c->dtype == SM_BF16) ? 1 : 0);
  const dim3 grid(a.max_chunks, c->num_kv_heads, rows);
  if (c->dtype == SM_BF16 && a.max_chunks == 1 && n <= kDecThreads) {
    // more single-chunk pairs than compute units: deal them longest first
    const int cus = device_cus();
    if (cus > 0 && (int64_t)n * c->num_kv_heads > cus) {
      a.order_n = n;
      a.order_cus = cus;
      const bool d128 = c->head_dim == 128;
      if (STEP && a.crop)
        a.order_occ = d128 ? bf16_occupancy<128, STEP, STEP>() : bf16_occupancy<64, STEP, STEP>();
      else
        a.order_occ = d128 ? bf16_occupancy<128, STEP, false>() : bf16_occupancy<64, STEP, false>();
    }
  }
  if (c->dtype == SM_BF16 && STEP && a.crop) {
    const bool ord = a.order_n > 0;
    if (c->head_dim == 128) {
      if (ord)
        hipLaunchKernelGGL((decode_split_bf16<128, true, true, true>), grid, dim3(kDecThreads), 0, stream, a);
      else
        hipLaunchKernelGGL((decode_split_bf16<128, true, false, true>), grid, dim3(kDecThreads), 0, stream, a);
    } else {
      if (ord)
        hipLaunchKernelGGL((decode_split_bf16<64, true, true, true>), grid, dim3(kDecThreads), 0, stream, a);
      else
        hipLaunchKernelGGL((decode_split_bf16<64, true, false, true>), grid, dim3(kDecThreads), 0, stream, a);
    }
  } else if (c->dtype == SM_BF16) {
    const bool ord = a.order_n > 0;
    if (c->head_dim == 128) {
      if (ord)
        hipLaunchKernelGGL((decode_split_bf16<128, STEP, true>), grid, dim3(kDecThreads), 0, stream, a);
      else
        hipLaunchKernelGGL((decode_split_bf16<128, STEP, false>), grid, dim3(kDecThreads), 0, stream, a);
    } else {
      if (ord)
        hipLaunchKernelGGL((decode_split_bf16<64, STEP, true>), grid, dim3(kDecThreads), 0, stream, a);
      else
        hipLaunchKernelGGL((decode_split_bf16<64, STEP, false>), grid, dim3(kDecThreads), 0, stream, a);
    }
  } else {
    if (c->head_dim == 128)
      hipLaunchKernelGGL((decode_split_f32<128, STEP>), grid, dim3(kDecThreads), 0, stream, a);
    else
      hipLaunchKernelGGL((decode_split_f32<64, STEP>), grid, dim3(kDecThreads), 0, stream, a);
  }
  return hipGetLastError() == hipSuccess ? SM_OK : SM_EHIP;
}

SM_API sm_status sm_decode_attention(const sm_paged_cache *c, const int32_t *seq_ids, int n,
                                     const void *q, int num_q_heads, float scale, int max_len,
                                     void *out, void *ws, size_t ws_bytes, hipStream_t stream) {
  DecodeArgs a;
  const sm_status st = decode_setup(c, seq_ids, n, q, num_q_heads, scale, max_len, out, ws, ws_bytes,
                                    kMaxPairs, a);
  if (st != SM_OK || n == 0) return st;
  return decode_launch<false>(c, a, n, stream);
}

// Polls of the fused step's commit wait (kCommitSpinLimit unless a test
// lowers it to exercise the give-up path).
static std::atomic<int> g_commit_spin_limit{kCommitSpinLimit};

SM_API void sm_set_commit_wait_limit(int polls) {
  g_commit_spin_limit.store(polls > 0 ? polls : kCommitSpinLimit);
}

static sm_status decode_step_impl(const sm_paged_cache *c, const int32_t *seq_ids, int n, const void *K,
                                  const void *V, const void *q, int num_q_heads, float scale, int max_len,
                                  void *out, void *ws, size_t ws_bytes, bool exact_ws, hipStream_t stream,
                                  const int32_t *crop = nullptr) {
  if (n > kDecThreads) return SM_EINVAL;
  if (n > 0 && (!K || !V || !c || !c->free_stack || !c->free_top)) return SM_EINVAL;
  DecodeArgs a;
  // the last two counter words are the step's error word and arrival counter
  const sm_status st = decode_setup(c, seq_ids, n, q, num_q_heads, scale, max_len, out, ws, ws_bytes,
                                    kMaxPairs - 2, a, exact_ws);
  if (st != SM_OK || n == 0) return st;
  a.k_new = K;
  a.crop = crop;
  a.v_new = V;
  a.free_stack = c->free_stack;
  a.free_top = c->free_top;
  a.block_table_w = c->block_table;
  a.lengths_w = c->lengths;
  a.step_err = a.counters + kMaxPairs - 2;
  a.step_arrivals = a.counters + kMaxPairs - 1;
  const int64_t cap = (int64_t)c->max_blocks_per_seq * c->block_size;
  a.cap = cap > INT32_MAX ? INT32_MAX : (int)cap;
  a.total_wgs = a.max_chunks * c->num_kv_heads * n;
  a.spin_limit = g_commit_spin_limit.load();
  return decode_launch<true>(c, a, n, stream);
}

SM_API sm_status sm_decode_step(const sm_paged_cache *c, const int32_t *seq_ids, int n, const void *K,
                                const void *V, const void *q, int num_q_heads, float scale, int max_len,
                                void *out, void *ws, size_t ws_bytes, hipStream_t stream) {
  return decode_step_impl(c, seq_ids, n, K, V, q, num_q_heads, scale, max_len, out, ws, ws_bytes, false, stream);
}

SM_API sm_status sm_decode_merge_step(const sm_paged_cache *c, const int32_t *seq_ids, const int32_t *crop, int n,
                                      const void *K, const void *V, const void *q, int num_q_heads, float scale,
                                      int max_len, void *out, void *ws, size_t ws_bytes, hipStream_t stream) {
  if (!c || c->dtype != SM_BF16) return SM_EINVAL;
  if (n > 0 && !crop) return SM_EINVAL;
  return decode_step_impl(c, seq_ids, n, K, V, q, num_q_heads, scale, max_len, out, ws, ws_bytes, false, stream,
                          crop);
}

// ---------------------------------------------------------------------------
// sm_decode_step_noalloc: the fused step with its workspace (arrival
// counters + split partials) in a fixed device array instead of a caller
// buffer, for callers that cannot allocate.  Each device the library runs
// on holds its own copy of the array until the process ends; its address is
// looked up once per device and kept.  The counters must be zero before the
// first call: they are cleared once, by a fill kernel on the first call's
// stream, and every call leaves them zero again.  Calls that overlap on one
// device share the array and race.

constexpr int64_t kScratchPartialBytes = 8ll << 20;
constexpr int64_t kScratchBytes = kCounterBytes + kScratchPartialBytes;
constexpr int kScratchMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

static __global__ void scratch_clear_kernel(uint32_t *p, int64_t words) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < words; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

static std::mutex g_scratch_mu;
static void *g_scratch_ptr[kScratchMaxDevices];

// Device address of this device's scratch array (cleared on first use), or
// nullptr when it cannot be had.
static void *scratch_for_current_device(hipStream_t stream) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kScratchMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    // counters only: the partials are written before they are read
    hipLaunchKernelGGL(scratch_clear_kernel, dim3(64), dim3(256), 0, stream, (uint32_t *)ptr,
                       (int64_t)(kCounterBytes / 4));
    if (hipGetLastError() != hipSuccess) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

SM_API size_t sm_decode_step_noalloc_max_bytes(void) { return (size_t)kScratchPartialBytes; }

SM_API sm_status sm_decode_step_noalloc(const sm_paged_cache *c, const int32_t *seq_ids, int n, const void *K,
                                        const void *V, const void *q, int num_q_heads, float scale, int max_len,
                                        void *out, hipStream_t stream) {
  void *ws = scratch_for_current_device(stream);
  if (!ws) return SM_EHIP;
  return decode_step_impl(c, seq_ids, n, K, V, q, num_q_heads, scale, max_len, out, ws, (size_t)kScratchBytes,
                          true, stream);
}
