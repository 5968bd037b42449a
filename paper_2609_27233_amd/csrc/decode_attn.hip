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
// V pages are stored dim-major ([head_dim][block_size]), so the 8 tokens a
// lane feeds to the PV product are 16 contiguous bytes.  The QK rows of the
// two 16-row score tiles are permuted so that the score tile's output layout
// is already the PV operand layout: lane (r, q) of a wave owns the scores of
// tokens 8q .. 8q+7 of the tile for head r.
#include "common.hpp"

namespace sm {

constexpr int kDecThreads = 256;
constexpr int kDecWaves = kDecThreads / 64;
constexpr int kMaxChunkTokens = 4096;
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
__device__ __forceinline__ int seq_status(const DecodeArgs &a, int s, int &L) {
  L = 0;
  if (s < 0 || s >= a.max_seqs) return SM_ERR_EINVAL;
  L = a.lengths[s];
  if (L < 0 || L > (a.max_blocks << a.bs_log2)) return SM_ERR_EINVAL;
  if (L > a.max_len) return SM_ERR_ERANGE;
  return 0;
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
                                                  int g, int c) {
  if (threadIdx.x < a.G) {
    const int64_t pidx = ((int64_t)i * a.Hq + g * a.G + threadIdx.x) * a.max_chunks + c;
    put_partial(&a.ws_ml[pidx * 2 + 0], 0.f);
    put_partial(&a.ws_ml[pidx * 2 + 1], -1.f);  // marks the chunk as unusable
  }
  if (threadIdx.x == 0) set_err(a.err, SM_ERR_EINVAL);
}

// Zero the output rows of group g's query heads (done by the chunk-0
// workgroup of a sequence that cannot be processed or is empty) and report a
// sequence-level error.
template <typename OutT>
__device__ void write_zero_rows(const DecodeArgs &a, int i, int g, int DH, int st) {
  OutT *o = (OutT *)a.out + ((int64_t)i * a.Hq + g * a.G) * DH;
  for (int e = threadIdx.x; e < a.G * DH; e += blockDim.x) o[e] = Elem<OutT>::to_store(0.f);
  if (st != 0 && threadIdx.x == 0) set_err(a.err, st);
}

// Every workgroup calls this once its partial is stored.  The last of the
// nc workgroups of (sequence i, kv head g) to arrive rescales and sums all
// partials of the group, writes the output rows and re-arms the counter.
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
  for (int e = threadIdx.x; e < a.G * DH; e += blockDim.x) {
    const int hh = e / DH, dd = e - hh * DH;
    const int64_t base = ((int64_t)i * a.Hq + g * a.G + hh) * a.max_chunks;
    float M = -INFINITY;
    bool bad = false;
    for (int c = 0; c < nc; ++c) {
      bad |= get_partial(&a.ws_ml[(base + c) * 2 + 1]) < 0.f;
      M = fmaxf(M, get_partial(&a.ws_ml[(base + c) * 2 + 0]));
    }
    float acc = 0.f, ls = 0.f;
    if (!bad) {
      for (int c = 0; c < nc; ++c) {
        const float f = exp2f(get_partial(&a.ws_ml[(base + c) * 2 + 0]) - M);
        acc += get_partial(&a.ws_o[(base + c) * DH + dd]) * f;
        ls += get_partial(&a.ws_ml[(base + c) * 2 + 1]) * f;
      }
    }
    out[((int64_t)i * a.Hq + g * a.G + hh) * DH + dd] = Elem<OutT>::to_store(bad ? 0.f : acc / ls);
  }
  if (threadIdx.x == 0) *ctr = 0;
}

// ---------------------------------------------------------------------------
// bf16 split kernel (matrix cores)

template <int DH>
struct KVTile {
  u32x4_t ka[DH / 32];  // K rows of score tile A (16 tokens x 8 dims / lane)
  u32x4_t kb[DH / 32];  // K rows of score tile B
  u32x4_t v[DH / 16];   // V^T: 16 dims x 8 tokens per lane
};

template <int DH>
__global__ __launch_bounds__(kDecThreads, 2) void decode_split_bf16(DecodeArgs a) {
  __shared__ int pages[kMaxChunkPages];
  __shared__ int flag;
  __shared__ float red_m[kDecWaves][16];
  __shared__ float red_l[kDecWaves][16];
  __shared__ float red_o[kDecWaves][16][DH];

  const int c = blockIdx.x, g = blockIdx.y, i = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int s = a.seq_ids[i];
  int L;
  const int st = seq_status(a, s, L);
  if (st != 0 || L == 0) {
    if (c == 0) write_zero_rows<uint16_t>(a, i, g, DH, st);
    return;
  }
  int nc, chunk;
  chunking(L, a.chunk_nominal, nc, chunk);
  if (c >= nc) return;
  const int t0 = c * chunk;
  const int t1 = min(L, t0 + chunk);
  const int bs_log2 = a.bs_log2, bs = 1 << bs_log2;
  const int lp0 = t0 >> bs_log2;
  const int npages = ((t1 - 1) >> bs_log2) - lp0 + 1;
  if (!load_pages(a, s, lp0, npages, pages, &flag)) {
    write_bad_partial(a, i, g, c);
    finish_group<uint16_t>(a, i, g, nc, DH, &flag);
    return;
  }

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
  const int ntiles = (t1 - t0 + 31) >> 5;

  auto load = [&](KVTile<DH> &T, int tile) {
    const int T0 = t0 + 32 * tile;
    // tokens past the chunk end read the chunk's first entry instead (their
    // scores are masked and their V lanes zeroed below)
    const int tA = (T0 + offA < t1) ? T0 + offA : t0;
    const int tB = (T0 + offB < t1) ? T0 + offB : t0;
    const int tV = (T0 + offV < t1) ? T0 + offV : t0;
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
    const int nvalid = min(8, max(0, t1 - (T0 + offV)));
#pragma unroll
    for (int j = 0; j < 8; ++j) sc[j] = (j < nvalid) ? sc[j] * sl2 : -INFINITY;
    float mx = sc[0];
#pragma unroll
    for (int j = 1; j < 8; ++j) mx = fmaxf(mx, sc[j]);
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
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

  // per-head totals of this wave (lanes r, r+16, r+32, r+48 share head r)
  float l_tot = l_run + __shfl_xor(l_run, 16, 64);
  l_tot += __shfl_xor(l_tot, 32, 64);
  if (q4 == 0) {
    red_m[w][r] = m_run;
    red_l[w][r] = l_tot;
  }
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt)
#pragma unroll
    for (int j = 0; j < 4; ++j) red_o[w][r][16 * dt + 4 * q4 + j] = o[dt][j];
  __syncthreads();

  for (int e = tid; e < G * DH; e += kDecThreads) {
    const int hh = e / DH, dd = e - hh * DH;
    float M = red_m[0][hh];
#pragma unroll
    for (int ww = 1; ww < kDecWaves; ++ww) M = fmaxf(M, red_m[ww][hh]);
    float acc = 0.f, ls = 0.f;
#pragma unroll
    for (int ww = 0; ww < kDecWaves; ++ww) {
      const float f = exp2f(red_m[ww][hh] - M);  // idle waves: exp2(-inf) = 0
      acc += red_o[ww][hh][dd] * f;
      ls += red_l[ww][hh] * f;
    }
    if (nc == 1) {  // the only chunk: write the result directly
      ((uint16_t *)a.out)[((int64_t)i * a.Hq + g * G + hh) * DH + dd] = f32_to_bf16(acc / ls);
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
}

// ---------------------------------------------------------------------------
// fp32 split kernel (vector ALU; chunks of at most 256 tokens, one token per
// thread for the scores)

template <int DH>
__global__ __launch_bounds__(kDecThreads) void decode_split_f32(DecodeArgs a) {
  __shared__ int pages[kF32ChunkTokens / 16 + 2];
  __shared__ int flag;
  __shared__ float qs[DH];
  __shared__ float ps[kF32ChunkTokens];
  __shared__ float red[kDecWaves];
  constexpr int NG = kDecThreads / DH;  // token groups for the PV sums
  __shared__ float opart[NG][DH];

  const int c = blockIdx.x, g = blockIdx.y, i = blockIdx.z;
  const int tid = threadIdx.x;
  const int s = a.seq_ids[i];
  int L;
  const int st = seq_status(a, s, L);
  if (st != 0 || L == 0) {
    if (c == 0) write_zero_rows<float>(a, i, g, DH, st);
    return;
  }
  int nc, chunk;
  chunking(L, a.chunk_nominal, nc, chunk);
  if (c >= nc) return;
  const int t0 = c * chunk;
  const int t1 = min(L, t0 + chunk);
  const int bs_log2 = a.bs_log2, bs = 1 << bs_log2;
  const int lp0 = t0 >> bs_log2;
  const int npages = ((t1 - 1) >> bs_log2) - lp0 + 1;
  if (!load_pages(a, s, lp0, npages, pages, &flag)) {
    write_bad_partial(a, i, g, c);
    finish_group<float>(a, i, g, nc, DH, &flag);
    return;
  }
  const float *kp = (const float *)a.k_pool;
  const float *vp = (const float *)a.v_pool;
  const int64_t page_elems = (int64_t)bs * DH;
  const int ntok = t1 - t0;
  const int tok = t0 + tid;
  const bool valid = tid < ntok;
  const float *krow = kp;
  if (valid) {
    const int b = pages[(tok >> bs_log2) - lp0];
    krow = kp + ((int64_t)b * a.Hkv + g) * page_elems + (int64_t)(tok & (bs - 1)) * DH;
  }
  const int dd = tid % DH, tg = tid / DH;

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
    const float M = block_max(sc, red);
    const float p = valid ? exp2f(sc - M) : 0.f;
    const float l = block_sum(p, red);
    ps[tid] = p;
    __syncthreads();
    float acc = 0.f;
    for (int t = tg; t < ntok; t += NG) {
      const int tt = t0 + t;
      const int b = pages[(tt >> bs_log2) - lp0];
      acc += ps[t] * vp[((int64_t)b * a.Hkv + g) * page_elems + (int64_t)dd * bs + (tt & (bs - 1))];
    }
    opart[tg][dd] = acc;
    __syncthreads();
    if (tid < DH) {
      float o = 0.f;
      for (int k = 0; k < NG; ++k) o += opart[k][tid];
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
  // contiguous streams per workgroup measured fastest), with chunks kept
  // between 256 and 2048 tokens so that batches of mixed lengths still
  // split into enough pieces to balance; a multiple of 128 tokens (32 per
  // wave).
  const int64_t cus = 256;
  int64_t c = ((int64_t)max_len * n * Hkv + cus - 1) / cus;
  c = (c + 127) / 128 * 128;
  if (c < 256) c = 256;
  if (c > 2048) c = 2048;
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

SM_API sm_status sm_decode_attention(const sm_paged_cache *c, const int32_t *seq_ids, int n,
                                     const void *q, int num_q_heads, float scale, int max_len,
                                     void *out, void *ws, size_t ws_bytes, hipStream_t stream) {
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
  if (n > 65535 || (int64_t)n * c->num_kv_heads > kMaxPairs) return SM_EINVAL;
  if (ws_bytes < sm_decode_workspace_bytes(n, num_q_heads, c->head_dim, max_len)) return SM_EINVAL;

  DecodeArgs a;
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
  a.counters = (int32_t *)ws;
  a.ws_o = (float *)((char *)ws + kCounterBytes);
  a.ws_ml = a.ws_o + (int64_t)n * num_q_heads * a.max_chunks * c->head_dim;

  // one launch: split, and the last workgroup of each (sequence, kv head)
  // combines; with max_len = 0 the single chunk column writes zero rows
  const dim3 grid(a.max_chunks, c->num_kv_heads, n);
  if (c->dtype == SM_BF16) {
    if (c->head_dim == 128)
      hipLaunchKernelGGL(decode_split_bf16<128>, grid, dim3(kDecThreads), 0, stream, a);
    else
      hipLaunchKernelGGL(decode_split_bf16<64>, grid, dim3(kDecThreads), 0, stream, a);
  } else {
    if (c->head_dim == 128)
      hipLaunchKernelGGL(decode_split_f32<128>, grid, dim3(kDecThreads), 0, stream, a);
    else
      hipLaunchKernelGGL(decode_split_f32<64>, grid, dim3(kDecThreads), 0, stream, a);
  }
  return hipGetLastError() == hipSuccess ? SM_OK : SM_EHIP;
}
