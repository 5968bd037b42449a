// Prefill attention over the paged cache (gfx950).
//
// The prefill pass that prompt compression shortens ("Efficiency Analysis":
// every layer of the prefill runs over the compressed sequence).  Request i
// brings the m_i query rows of the last m_i cached positions of sequence
// s = seq_ids[i]; the row at position p attends causally to entries 0..p:
//   out[row, h] = sum_{j <= p} softmax_j(scale q . K[s, j, g]) V[s, j, g],
//   g = h / G (grouped query).
//
// One workgroup of eight waves per (request, kv head, block of positions).
// It holds 256 query vectors: BQ = 256 / G positions x the G query heads of
// kv head g, so every K/V tile it loads serves all of them.  A wave owns 32
// vectors, the columns of the transposed score blocks
//   S^T (32 keys x 32 queries) = K (32 x D) . Q^T        (v_mfma_f32_32x32x16_bf16)
// and accumulates
//   O^T (D x 32 queries) += V^T (D x 32 keys) . P^T.
// At about 220 registers a wave, two waves share each SIMD, so one wave's
// softmax runs while the other's products occupy the matrix unit.
// In S^T a lane holds 16 keys of one query column, so the softmax row
// statistics need one lane swap per tile.  The K rows of a block are read in
// a permuted order so that the 16 scores a lane holds are exactly the keys
// its PV operand needs (8 contiguous tokens per 16-key step): no shuffle
// between the two products.  K/V tiles of 64 keys go through LDS, the next
// tile's global loads in flight while the current one is multiplied.
//
// Softmax: exp2 of (score x scale log2 e - reference), with the reference
// (a running maximum) moved only when a tile's maximum exceeds it by more
// than 2^8.  Any reference gives the same ratios; keeping it mostly fixed
// skips the rescale of the accumulators on almost every tile.
#include "common.hpp"

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// round-to-nearest-even pair conversion (one v_cvt_pk_bf16_f32 on gfx950)
__device__ __forceinline__ uint32_t cvt_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

namespace sm {

constexpr int kPfVec = 256;                 // query vectors per workgroup
constexpr int kPfWaves = kPfVec / 32;       // one 32-vector column block per wave
constexpr int kPfThreads = 64 * kPfWaves;
constexpr int kPfKeys = 64;                 // keys per tile
constexpr int kPfSub = kPfKeys / 32;        // 32-key score blocks per tile
constexpr int kPfMaxPages = 4096;
constexpr float kPfLog2e = 1.4426950408889634f;

struct PrefillArgs {
  const uint16_t *k_pool;
  const uint16_t *v_pool;
  const int32_t *block_table;
  const int32_t *lengths;
  const int32_t *seq_ids;
  const int32_t *q_offsets;
  const uint16_t *q;
  uint16_t *out;
  int32_t *err;
  int n, total_rows, max_rows, Hkv, Hq, G, BQ, nqb, bs_log2, num_blocks, max_seqs, max_blocks;
  uint32_t page_bytes;  // bytes of one page over all kv heads
  float scale_log2e;    // |scale| log2(e), at least 1e-30
  uint32_t q_sign;      // 0x80008000 when scale < 0: q enters with its sign flipped
};

// Score-block row rho (0..31) holds token tau(rho) of the block: within each
// 16 rows the middle two groups of four swap places, so that the rows a lane
// holds after S^T = K . Q^T ({8 g + 4 h + e}) are tokens 8 h .. 8 h + 7 of
// each 16-key step, in register order.
__device__ __forceinline__ int pf_token_of_row(int rho) {
  const int q = (rho >> 2) & 3;
  const int q2 = q == 1 ? 2 : q == 2 ? 1 : q;
  return (rho & ~15) | (q2 << 2) | (rho & 3);
}

template <int DH>
__global__ __launch_bounds__(kPfThreads, 2) void prefill_bf16(PrefillArgs a) {
  constexpr int KP = DH + 8;        // K tile row pitch (bf16)
  constexpr int VP = kPfKeys + 8;   // V tile row pitch (bf16)
  constexpr int NKS = DH / 16;      // k steps of S^T
  constexpr int NRB = DH / 32;      // 32-dim row blocks of O^T
  constexpr int KCH = DH / 8;       // 16-byte chunks of a K row
  constexpr int VCH = kPfKeys / 8;  // 16-byte chunks of a V row (one dim) in a tile
  constexpr int KTOT = kPfKeys * KCH, VTOT = DH * VCH;    // 16-byte chunks per tile
  constexpr int KU = (KTOT + kPfThreads - 1) / kPfThreads;  // K chunks per thread and tile
  constexpr int VU = (VTOT + kPfThreads - 1) / kPfThreads;  // V chunks per thread and tile
  __shared__ int pages[kPfMaxPages];
  __shared__ int bad_flag;
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[2][kPfKeys * KP];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[2][DH * VP];

  // Workgroup -> (request i, kv head g, block qb).  Workgroups are dealt to
  // the eight XCDs in turn; here the blocks of one (request, head) pair all
  // land on one XCD, so its L2 fetches the pair's K/V once, and eight pairs
  // run side by side.  Within a pair the longest blocks go first.
  const int nqb = a.nqb, P = a.n * a.Hkv, Pfull = P & ~7;
  const int b = blockIdx.x;
  int pair, j;
  if (b < Pfull * nqb) {
    const int k = b >> 3;
    pair = (k / nqb) * 8 + (b & 7);
    j = k - (k / nqb) * nqb;
  } else {
    const int b2 = b - Pfull * nqb;
    pair = Pfull + b2 / nqb;
    j = b2 - (b2 / nqb) * nqb;
  }
  const int qb = nqb - 1 - j, g = pair % a.Hkv, i = pair / a.Hkv;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int c32 = lane & 31, h2 = lane >> 5;
  const int bs_log2 = a.bs_log2, bs = 1 << bs_log2;

  // ---- request checks (uniform) ----
  const int r0 = a.q_offsets[i], r1 = a.q_offsets[i + 1];
  const bool rows_ok = r0 >= 0 && r1 >= r0 && r1 <= a.total_rows;  // before any row is addressed
  const int m = rows_ok ? r1 - r0 : 0;
  const int s = a.seq_ids[i];
  int L = 0;
  bool ok = rows_ok && m <= a.max_rows && s >= 0 && s < a.max_seqs;
  if (ok) {
    L = a.lengths[s];
    ok = L >= 0 && L <= (a.max_blocks << bs_log2) && m <= L;
  }
  if (!ok) {  // block 0 reports the request and zeroes its rows
    if (qb != 0) return;
    if (tid == 0) set_err(a.err, SM_ERR_EINVAL);
    const int per_row = a.G * DH;  // this kv head's query heads
    for (int64_t e = tid; e < (int64_t)m * per_row; e += kPfThreads) {
      const int rr = (int)(e / per_row), k = (int)(e - (int64_t)rr * per_row);
      a.out[((int64_t)(r0 + rr) * a.Hq + g * a.G) * DH + k] = 0;
    }
    return;
  }
  const int q_lo = qb * a.BQ;  // first row of this block within the request
  if (q_lo >= m) return;
  const int nq = min(a.BQ, m - q_lo);
  const int pos0 = L - m + q_lo;  // position of row q_lo
  const int kend = pos0 + nq;     // keys [0, kend) are needed

  // ---- page ids of keys [0, kend) into LDS, range-checked ----
  if (tid == 0) bad_flag = 0;
  __syncthreads();
  const int npg = (kend + bs - 1) >> bs_log2;
  for (int p = tid; p < npg; p += kPfThreads) {
    int blk = a.block_table[(int64_t)s * a.max_blocks + p];
    if (blk < 0 || blk >= a.num_blocks) {
      bad_flag = 1;
      blk = 0;
    }
    pages[p] = blk;
  }
  __syncthreads();
  if (bad_flag) {  // a corrupt block table: this block's rows are zero
    if (tid == 0) set_err(a.err, SM_ERR_EINVAL);
    const int per_row = a.G * DH;
    for (int e = tid; e < nq * per_row; e += kPfThreads) {
      const int rr = e / per_row, k = e - rr * per_row;
      a.out[((int64_t)(r0 + q_lo + rr) * a.Hq + g * a.G) * DH + k] = 0;
    }
    return;
  }

  // ---- this wave's 32 query vectors: v = 32 w + c32 -> query head g G + v / BQ, row q_lo + v % BQ ----
  const int v = 32 * w + c32;
  const int hh = v / a.BQ, rr = v - hh * a.BQ;
  const bool vok = hh < a.G && rr < nq;
  const int vhead = g * a.G + (vok ? hh : 0);
  const int vrow = r0 + q_lo + (vok ? rr : 0);
  const int vpos = vok ? pos0 + rr : -1;  // an idle vector sees no key
  u32x4_t qf[NKS];
  {
    const uint16_t *qp = a.q + ((int64_t)vrow * a.Hq + vhead) * DH + 8 * h2;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      qf[ks] = vok ? *(const u32x4_t *)(qp + 16 * ks) ^ a.q_sign : u32x4_t{0u, 0u, 0u, 0u};
  }
  // wave-wide position range of the valid vectors: tiles past all of them
  // are skipped, tiles before all of them need no mask
  int wave_lo = vok ? vpos : 0x7fffffff, wave_hi = vpos;
#pragma unroll
  for (int sh = 1; sh < 64; sh <<= 1) {
    wave_lo = min(wave_lo, __shfl_xor(wave_lo, sh));
    wave_hi = max(wave_hi, __shfl_xor(wave_hi, sh));
  }
  wave_lo = __builtin_amdgcn_readfirstlane(wave_lo);
  wave_hi = __builtin_amdgcn_readfirstlane(wave_hi);

  // ---- tile loader: 16-byte chunks, K as rows of tokens, V as dim-major runs of 8 tokens ----
  // A chunk's offset within its page is fixed per thread; a tile adds a
  // uniform (t0 mod bs) and its page id.  Tokens past kend re-read page 0.
  const uint64_t page_bytes = a.page_bytes;
  const char *kbase = (const char *)a.k_pool + (int64_t)g * bs * DH * 2;
  const char *vbase = (const char *)a.v_pool + (int64_t)g * bs * DH * 2;
  int ktk[KU], koff[KU], vtk[VU], voff[VU];
#pragma unroll
  for (int u = 0; u < KU; ++u) {
    const int id = min(tid + kPfThreads * u, KTOT - 1);
    ktk[u] = id / KCH;
    koff[u] = ((ktk[u] & (bs - 1)) * DH + (id % KCH) * 8) * 2;
  }
#pragma unroll
  for (int u = 0; u < VU; ++u) {
    const int id = min(tid + kPfThreads * u, VTOT - 1);
    vtk[u] = 8 * (id % VCH);
    voff[u] = ((id / VCH) * bs + (vtk[u] & (bs - 1))) * 2;
  }
  auto fetch = [&](int t0, u32x4_t (&kv)[KU + VU]) {
    const int tin = t0 & (bs - 1);  // 0 when a page is no longer than a tile
#pragma unroll
    for (int u = 0; u < KU; ++u) {
      const int tok = t0 + ktk[u];
      const uint32_t blk = pages[tok < kend ? tok >> bs_log2 : 0];
      kv[u] = *(const u32x4_t *)(kbase + blk * page_bytes + (koff[u] + tin * DH * 2));
    }
#pragma unroll
    for (int u = 0; u < VU; ++u) {
      const int tok = t0 + vtk[u];
      const uint32_t blk = pages[tok < kend ? tok >> bs_log2 : 0];
      kv[KU + u] = *(const u32x4_t *)(vbase + blk * page_bytes + (voff[u] + tin * 2));
    }
    if (t0 + kPfKeys > L) {  // the last tile: V entries past the length may hold anything
#pragma unroll
      for (int u = 0; u < VU; ++u) {
        const int nvalid = L - (t0 + vtk[u]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (2 * e >= nvalid) kv[KU + u][e] = 0u;
          else if (2 * e + 1 >= nvalid) kv[KU + u][e] &= 0xffffu;
        }
      }
    }
  };
  auto stash = [&](int buf, const u32x4_t (&kv)[KU + VU]) {
#pragma unroll
    for (int u = 0; u < KU; ++u) {
      const int id = tid + kPfThreads * u;
      if (KTOT % kPfThreads == 0 || id < KTOT) *(u32x4_t *)(&k_lds[buf][(id / KCH) * KP + (id % KCH) * 8]) = kv[u];
    }
#pragma unroll
    for (int u = 0; u < VU; ++u) {
      const int id = tid + kPfThreads * u;
      if (VTOT % kPfThreads == 0 || id < VTOT) *(u32x4_t *)(&v_lds[buf][(id / VCH) * VP + 8 * (id % VCH)]) = kv[KU + u];
    }
  };

  f32x16_t o[NRB];
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[rb][e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float sl2 = a.scale_log2e;
  const int krow = pf_token_of_row(c32);  // this lane's K row in the S^T operand

  const int ntiles = (kend + kPfKeys - 1) / kPfKeys;
  u32x4_t stage[KU + VU];
  fetch(0, stage);
  stash(0, stage);
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1, t0 = t * kPfKeys;
    if (t + 1 < ntiles) fetch(t0 + kPfKeys, stage);  // in flight during this tile

    if (t0 <= wave_hi) {
      // S^T = K . Q^T, one 32-key block at a time: its fragment reads first, then its products
      f32x16_t sc[kPfSub];
#pragma unroll
      for (int sb = 0; sb < kPfSub; ++sb) {
#pragma unroll
        for (int e = 0; e < 16; ++e) sc[sb][e] = 0.f;
        const uint16_t *kl = &k_lds[buf][(32 * sb + krow) * KP + 8 * h2];
        u32x4_t kf[NKS];
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) kf[ks] = *(const u32x4_t *)(kl + 16 * ks);
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
          sc[sb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kf[ks]), as_bf16x8(qf[ks]), sc[sb], 0, 0, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, NKS, 0);  // LDS reads
        __builtin_amdgcn_sched_group_barrier(0x008, NKS, 0);  // MFMA
      }
      // V fragments of the first block: lane (d, h2) feeds dims 32 rb + d, tokens 16 kst + 8 h2 .. +7
      u32x4_t vf[NRB][2];
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int kst = 0; kst < 2; ++kst)
          vf[rb][kst] = *(const u32x4_t *)(&v_lds[buf][(32 * rb + c32) * VP + 16 * kst + 8 * h2]);

      // online softmax per query column; register r of block sb holds token
      // t0 + 32 sb + tau(8 (r >> 2) + 4 h2 + (r & 3)).  Masked scores become
      // -inf in place: exp2 of -inf is 0 (the multiplier is positive).
      if (t0 + kPfKeys - 1 > wave_lo) {
#pragma unroll
        for (int sb = 0; sb < kPfSub; ++sb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int tok = t0 + 32 * sb + pf_token_of_row(8 * (r >> 2) + 4 * h2 + (r & 3));
            sc[sb][r] = tok <= vpos ? sc[sb][r] : -INFINITY;
          }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int sb = 0; sb < kPfSub; ++sb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[sb][r]);
      float a0, b0;
      swap32(mx, a0, b0);
      mx = fmaxf(a0, b0);
      const float ms = mx == -INFINITY ? -INFINITY : mx * sl2;  // in log2 units
      const bool move = ms > m_run + 8.0f;
      const float m_new = move ? ms : m_run;
      const float mb = m_new == -INFINITY ? 0.f : m_new;  // a column with no key yet
      if (__ballot(move) != 0) {  // rare: rescale before this tile's products are added
        const float alpha = move ? __builtin_amdgcn_exp2f(m_run - mb) : 1.f;
        l_run *= alpha;
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb) o[rb] *= alpha;
      }
      m_run = m_new;
      float ps = 0.f;
      u32x4_t pf[kPfSub][2];
#pragma unroll
      for (int sb = 0; sb < kPfSub; ++sb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          sc[sb][r] = __builtin_amdgcn_exp2f(fmaf(sc[sb][r], sl2, -mb));
          ps += sc[sb][r];
        }
        const f32x16_t &x = sc[sb];
#pragma unroll
        for (int kst = 0; kst < 2; ++kst)
          pf[sb][kst] = u32x4_t{cvt_bf16x2(x[8 * kst + 0], x[8 * kst + 1]), cvt_bf16x2(x[8 * kst + 2], x[8 * kst + 3]),
                                cvt_bf16x2(x[8 * kst + 4], x[8 * kst + 5]), cvt_bf16x2(x[8 * kst + 6], x[8 * kst + 7])};
      }
      l_run += ps;

      // O^T += V^T . P^T
#pragma unroll
      for (int sb = 0; sb < kPfSub; ++sb) {
        if (sb > 0) {
#pragma unroll
          for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
            for (int kst = 0; kst < 2; ++kst)
              vf[rb][kst] = *(const u32x4_t *)(&v_lds[buf][(32 * rb + c32) * VP + 32 * sb + 16 * kst + 8 * h2]);
        }
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
          for (int kst = 0; kst < 2; ++kst)
            o[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vf[rb][kst]), as_bf16x8(pf[sb][kst]), o[rb], 0, 0, 0);
      }
    }

    if (t + 1 < ntiles) stash(buf ^ 1, stage);
    __syncthreads();
  }

  // ---- normalize and store: register 4 gg + e of block rb = dim 32 rb + 8 gg + 4 h2 + e ----
  float a0, b0;
  swap32(l_run, a0, b0);
  const float l_tot = a0 + b0;
  const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
  if (!vok) return;
  uint16_t *op = a.out + ((int64_t)vrow * a.Hq + vhead) * DH + 4 * h2;
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
    for (int gg = 0; gg < 4; ++gg)
      *(uint2 *)(op + 32 * rb + 8 * gg) = make_uint2(cvt_bf16x2(o[rb][4 * gg + 0] * inv, o[rb][4 * gg + 1] * inv),
                                                     cvt_bf16x2(o[rb][4 * gg + 2] * inv, o[rb][4 * gg + 3] * inv));
}

}  // namespace sm

using namespace sm;

SM_API sm_status sm_prefill_attention(const sm_paged_cache *c, const int32_t *seq_ids, int n,
                                      const int32_t *q_offsets, int total_rows, const void *q, int num_q_heads,
                                      float scale, int max_rows, void *out, hipStream_t stream) {
  if (!c || n < 0 || max_rows < 0 || total_rows < 0) return SM_EINVAL;
  if (n == 0) return SM_OK;
  if (!seq_ids || !q_offsets || !q || !out || !c->k_pool || !c->v_pool || !c->block_table || !c->lengths ||
      !c->err)
    return SM_EINVAL;
  if (c->dtype != SM_BF16 || !(fabsf(scale) <= 3.0e38f)) return SM_EINVAL;  // a finite scale
  const int H = c->num_kv_heads, D = c->head_dim, bs = c->block_size;
  if (H <= 0 || num_q_heads <= 0 || num_q_heads % H != 0) return SM_EINVAL;
  const int G = num_q_heads / H;
  if (G > 16 || (D != 64 && D != 128)) return SM_EINVAL;
  if (bs < 16 || (bs & (bs - 1)) != 0 || c->max_blocks_per_seq <= 0 || c->max_blocks_per_seq > kPfMaxPages ||
      c->num_blocks <= 0 || c->max_seqs <= 0)
    return SM_EINVAL;
  if (n > 65535 || (uint64_t)H * bs * D * 2 > 0xffffffffull) return SM_EINVAL;
  PrefillArgs a;
  a.k_pool = (const uint16_t *)c->k_pool;
  a.v_pool = (const uint16_t *)c->v_pool;
  a.block_table = c->block_table;
  a.lengths = c->lengths;
  a.seq_ids = seq_ids;
  a.q_offsets = q_offsets;
  a.q = (const uint16_t *)q;
  a.out = (uint16_t *)out;
  a.err = c->err;
  a.n = n;
  a.total_rows = total_rows;
  a.max_rows = max_rows;
  a.Hkv = H;
  a.Hq = num_q_heads;
  a.G = G;
  a.BQ = kPfVec / G;
  int bl = 0;
  while ((1 << bl) < bs) ++bl;
  a.bs_log2 = bl;
  a.num_blocks = c->num_blocks;
  a.max_seqs = c->max_seqs;
  a.max_blocks = c->max_blocks_per_seq;
  a.page_bytes = (uint32_t)((uint64_t)H * bs * D * 2);
  // A positive multiplier keeps exp2(-inf) = 0 for masked keys.  Below 1e-30
  // every weight rounds to 1 in fp32 either way (|q . k| stays far below 1e30).
  a.scale_log2e = fmaxf(fabsf(scale) * kPfLog2e, 1e-30f);
  a.q_sign = scale < 0.f ? 0x80008000u : 0u;
  const int nqb = max_rows > 0 ? (max_rows + a.BQ - 1) / a.BQ : 1;  // block 0 reports bad requests
  if ((int64_t)nqb * n * H > 0x7fffffff) return SM_EINVAL;
  a.nqb = nqb;
  const dim3 grid(nqb * n * H);
  if (D == 128)
    hipLaunchKernelGGL(prefill_bf16<128>, grid, dim3(kPfThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(prefill_bf16<64>, grid, dim3(kPfThreads), 0, stream, a);
  return hipGetLastError() == hipSuccess ? SM_OK : SM_EHIP;
}
