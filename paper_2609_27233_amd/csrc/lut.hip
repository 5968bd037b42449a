// Surrogate lookup and span dedupe (gfx950).
//
// A span's surrogate depends on its tokens only ("Computational Scope"), so
// surrogates can be computed once per rule and looked up:
//  * sm_gather_surrogates: out[i] = lut[rule_ids[i]] when rule_ids[i] >= 0,
//    else emb[token_ids[i]].  This gives a decode step's input row (the
//    surrogate of a just-merged suffix, or the plain token) and a prompt's
//    span surrogates without running the merge module.  One wave per row,
//    16-byte copies.
//  * sm_span_dedupe: spans of one merge batch that carry the same rule
//    share one surrogate.  The first span of each rule is found with an
//    atomic min per rule (repeats within a workgroup settled in LDS first);
//    per-block counts of first occurrences and their lengths are scanned
//    into the unique spans' order and CSR row offsets; a last pass gives
//    every span the slot of its rule's first span and writes the unique
//    spans' token ids, the merge module's input.
#include "common.hpp"

namespace sm {

constexpr int kGatherWaves = 4;

template <typename T>
__global__ __launch_bounds__(64 * kGatherWaves) void gather_rows_kernel(const T *emb, int64_t emb_rows, const T *lut,
                                                                        int64_t lut_rows, const int32_t *token_ids,
                                                                        const int32_t *rule_ids, int n, int d,
                                                                        T *out, int32_t *err) {
  const int i = blockIdx.x * kGatherWaves + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i >= n) return;
  const int r = rule_ids[i];
  const T *src = nullptr;
  if (r >= 0) {
    if (r < lut_rows) src = lut + (int64_t)r * d;
  } else if (token_ids) {
    const int tok = token_ids[i];
    if (tok >= 0 && tok < emb_rows) src = emb + (int64_t)tok * d;
  }
  if (!src && lane == 0) set_err(err, SM_ERR_EINVAL);
  constexpr int VEC = 16 / sizeof(T);
  T *dst = out + (int64_t)i * d;
  for (int v = lane; v < d / VEC; v += 64)
    *(u32x4_t *)(dst + v * VEC) = src ? *(const u32x4_t *)(src + v * VEC) : u32x4_t{0u, 0u, 0u, 0u};
}

__global__ void fill_i32_kernel(int32_t *p, int n, int v) {
  for (int r = blockIdx.x * blockDim.x + threadIdx.x; r < n; r += gridDim.x * blockDim.x) p[r] = v;
}

// The first span of every rule; a bad rule id or span range flags the call.
// A frequent rule would pile many atomics onto one address, so each
// workgroup first settles its own repeats in an LDS hash (one entry per
// distinct rule, holding its smallest span index) and only those entries go
// to the global atomic minimum.
constexpr int kDedupThreads = 256;
constexpr int kDedupSlots = 2 * kDedupThreads;

__global__ __launch_bounds__(kDedupThreads) void dedupe_owner_kernel(const int32_t *span_rule,
                                                                     const int32_t *span_start,
                                                                     const int32_t *span_len, int S, int num_rules,
                                                                     int total_tokens, int32_t *owner, int32_t *flag) {
  __shared__ int hkey[kDedupSlots], hmin[kDedupSlots];
  for (int j = threadIdx.x; j < kDedupSlots; j += kDedupThreads) {
    hkey[j] = -1;
    hmin[j] = 0x7fffffff;
  }
  __syncthreads();
  const int s = blockIdx.x * kDedupThreads + threadIdx.x;
  if (s < S) {
    const int r = span_rule[s], a = span_start[s], n = span_len[s];
    if (r < 0 || r >= num_rules || n < 1 || a < 0 || a > total_tokens - n) {
      atomicOr(flag, 1);
    } else {
      // at most kDedupThreads distinct keys in kDedupSlots slots: a free or
      // matching slot is always found
      uint32_t h = ((uint32_t)r * 2654435761u) >> 23;  // 9 bits
      for (int p = 0; p < kDedupSlots; ++p) {
        const int k = atomicCAS(&hkey[h], -1, r);
        if (k == -1 || k == r) {
          atomicMin(&hmin[h], s);
          break;
        }
        h = (h + 1) & (kDedupSlots - 1);
      }
    }
  }
  __syncthreads();
  for (int j = threadIdx.x; j < kDedupSlots; j += kDedupThreads) {
    const int r = hkey[j];
    if (r >= 0 && __atomic_load_n(&owner[r], __ATOMIC_RELAXED) > hmin[j]) atomicMin(&owner[r], hmin[j]);
  }
}

// per block of spans: how many are first occurrences, and their rows
__global__ __launch_bounds__(kDedupThreads) void dedupe_count_kernel(const int32_t *span_rule,
                                                                     const int32_t *span_len, int S,
                                                                     const int32_t *owner, const int32_t *flag,
                                                                     int32_t *blk_u, int32_t *blk_r) {
  __shared__ int red[16];
  if (*flag) return;
  const int s = blockIdx.x * kDedupThreads + threadIdx.x;
  const bool first = s < S && owner[span_rule[s]] == s;
  const int len = first ? span_len[s] : 0;
  int ut, rt;
  block_inclusive_scan(first ? 1 : 0, red, &ut);
  block_inclusive_scan(len, red, &rt);
  if (threadIdx.x == 0) {
    blk_u[blockIdx.x] = ut;
    blk_r[blockIdx.x] = rt;
  }
}

// exclusive scan of the block totals (one workgroup)
__global__ __launch_bounds__(kDedupThreads) void dedupe_blocks_kernel(int nblk, const int32_t *flag, int32_t *blk_u,
                                                                      int32_t *blk_r, int32_t *uniq_span_offsets,
                                                                      int32_t *num_uniq, int32_t *err) {
  __shared__ int red[16];
  if (*flag) {  // nothing to merge
    if (threadIdx.x == 0) {
      set_err(err, SM_ERR_EINVAL);
      *num_uniq = 0;
      uniq_span_offsets[0] = 0;
    }
    return;
  }
  int ub = 0, rb = 0;
  for (int b0 = 0; b0 < nblk; b0 += kDedupThreads) {
    const int b = b0 + threadIdx.x;
    const int u = b < nblk ? blk_u[b] : 0, r = b < nblk ? blk_r[b] : 0;
    int ut, rt;
    const int ui = block_inclusive_scan(u, red, &ut) - u;
    const int ri = block_inclusive_scan(r, red, &rt) - r;
    __syncthreads();  // every thread has read its totals before they are replaced
    if (b < nblk) {
      blk_u[b] = ub + ui;
      blk_r[b] = rb + ri;
    }
    ub += ut;
    rb += rt;
  }
  if (threadIdx.x == 0) {
    uniq_span_offsets[ub] = rb;
    *num_uniq = ub;
  }
}

// unique spans in order and their CSR row offsets, from the block offsets
__global__ __launch_bounds__(kDedupThreads) void dedupe_place_kernel(const int32_t *span_rule,
                                                                     const int32_t *span_len, int S,
                                                                     const int32_t *owner, const int32_t *flag,
                                                                     const int32_t *blk_u, const int32_t *blk_r,
                                                                     int32_t *ufirst, int32_t *uniq_span,
                                                                     int32_t *uniq_span_offsets) {
  __shared__ int red[16];
  if (*flag) return;
  const int s = blockIdx.x * kDedupThreads + threadIdx.x;
  const bool first = s < S && owner[span_rule[s]] == s;
  const int len = first ? span_len[s] : 0;
  int ut, rt;
  const int ui = block_inclusive_scan(first ? 1 : 0, red, &ut) - (first ? 1 : 0);
  const int ri = block_inclusive_scan(len, red, &rt) - len;
  if (first) {
    const int u = blk_u[blockIdx.x] + ui;
    ufirst[s] = u;
    uniq_span[u] = s;
    uniq_span_offsets[u] = blk_r[blockIdx.x] + ri;
  }
}

// every span's slot; the unique spans' token ids
__global__ void dedupe_slot_kernel(const int32_t *span_rule, const int32_t *span_start, const int32_t *span_len,
                                   int S, const int32_t *owner, const int32_t *flag, const int32_t *ufirst,
                                   const int32_t *uniq_span_offsets, const int32_t *token_ids, int32_t *span_slot,
                                   int32_t *uniq_row_idx) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= S || *flag) return;
  const int f = owner[span_rule[s]];
  const int u = ufirst[f];
  span_slot[s] = u;
  if (f == s) {
    const int a = span_start[s], o = uniq_span_offsets[u];
    for (int j = 0; j < span_len[s]; ++j) uniq_row_idx[o + j] = token_ids[a + j];
  }
}

}  // namespace sm

using namespace sm;

SM_API sm_status sm_gather_surrogates(const void *emb, int64_t emb_rows, const void *lut, int64_t lut_rows,
                                      const int32_t *token_ids, const int32_t *rule_ids, int n, int d, sm_dtype dt,
                                      void *out, int32_t *err, hipStream_t stream) {
  if (n < 0 || d <= 0 || emb_rows < 0 || lut_rows < 0 || (dt != SM_BF16 && dt != SM_F32)) return SM_EINVAL;
  const int es = dt == SM_BF16 ? 2 : 4;
  if ((d * es) % 16 != 0) return SM_EINVAL;
  if (n == 0) return SM_OK;
  if (!rule_ids || !out || !err || (lut_rows > 0 && !lut) || (token_ids && emb_rows > 0 && !emb)) return SM_EINVAL;
  const dim3 grid((n + kGatherWaves - 1) / kGatherWaves);
  if (dt == SM_BF16)
    hipLaunchKernelGGL(gather_rows_kernel<uint16_t>, grid, dim3(64 * kGatherWaves), 0, stream, (const uint16_t *)emb,
                       emb_rows, (const uint16_t *)lut, lut_rows, token_ids, rule_ids, n, d, (uint16_t *)out, err);
  else
    hipLaunchKernelGGL(gather_rows_kernel<float>, grid, dim3(64 * kGatherWaves), 0, stream, (const float *)emb,
                       emb_rows, (const float *)lut, lut_rows, token_ids, rule_ids, n, d, (float *)out, err);
  return hipGetLastError() == hipSuccess ? SM_OK : SM_EHIP;
}

static size_t a256(size_t v) { return (v + 255) & ~(size_t)255; }

SM_API size_t sm_span_dedupe_workspace_bytes(int S, int num_rules) {
  if (S < 0 || num_rules < 0) return 0;
  const size_t nblk = (size_t)(S + kDedupThreads - 1) / kDedupThreads;
  return 256 + a256((size_t)num_rules * 4) + a256((size_t)S * 4) + 2 * a256(nblk * 4);
}

SM_API sm_status sm_span_dedupe(const int32_t *span_rule, const int32_t *span_start, const int32_t *span_len, int S,
                                int num_rules, const int32_t *token_ids, int total_tokens, int32_t *uniq_span,
                                int32_t *span_slot, int32_t *uniq_row_idx, int32_t *uniq_span_offsets,
                                int32_t *num_uniq, void *ws, size_t ws_bytes, int32_t *err, hipStream_t stream) {
  if (S < 0 || num_rules < 0 || total_tokens < 0) return SM_EINVAL;
  if (!uniq_span_offsets || !num_uniq || !err || !ws || ws_bytes < sm_span_dedupe_workspace_bytes(S, num_rules))
    return SM_EINVAL;
  if (S > 0 && (!span_rule || !span_start || !span_len || !token_ids || !uniq_span || !span_slot || !uniq_row_idx))
    return SM_EINVAL;
  const int nblk = (S + kDedupThreads - 1) / kDedupThreads;
  char *w = (char *)ws;
  int32_t *flag = (int32_t *)w;
  w += 256;
  int32_t *owner = (int32_t *)w;
  w += a256((size_t)num_rules * 4);
  int32_t *ufirst = (int32_t *)w;
  w += a256((size_t)S * 4);
  int32_t *blk_u = (int32_t *)w;
  w += a256((size_t)nblk * 4);
  int32_t *blk_r = (int32_t *)w;
  hipLaunchKernelGGL(fill_i32_kernel, dim3(1), dim3(64), 0, stream, flag, 1, 0);
  hipLaunchKernelGGL(fill_i32_kernel, dim3(max(1, min((num_rules + 255) / 256, 4096))), dim3(256), 0, stream, owner,
                     num_rules, 0x7fffffff);
  if (S > 0) {
    hipLaunchKernelGGL(dedupe_owner_kernel, dim3(nblk), dim3(kDedupThreads), 0, stream, span_rule, span_start,
                       span_len, S, num_rules, total_tokens, owner, flag);
    hipLaunchKernelGGL(dedupe_count_kernel, dim3(nblk), dim3(kDedupThreads), 0, stream, span_rule, span_len, S, owner,
                       flag, blk_u, blk_r);
  }
  hipLaunchKernelGGL(dedupe_blocks_kernel, dim3(1), dim3(kDedupThreads), 0, stream, nblk, flag, blk_u, blk_r,
                     uniq_span_offsets, num_uniq, err);
  if (S > 0) {
    hipLaunchKernelGGL(dedupe_place_kernel, dim3(nblk), dim3(kDedupThreads), 0, stream, span_rule, span_len, S, owner,
                       flag, blk_u, blk_r, ufirst, uniq_span, uniq_span_offsets);
    hipLaunchKernelGGL(dedupe_slot_kernel, dim3(nblk), dim3(kDedupThreads), 0, stream, span_rule, span_start, span_len,
                       S, owner, flag, ufirst, uniq_span_offsets, token_ids, span_slot, uniq_row_idx);
  }
  return hipGetLastError() == hipSuccess ? SM_OK : SM_EHIP;
}
