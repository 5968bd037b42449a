// Prefill attention over the paged cache (gfx950).
//
// The prefill pass that prompt compression shortens ("Efficiency Analysis":
// every layer of the prefill runs over the compressed sequence).  Request i
// brings the m_i query rows of the last m_i cached positions of sequence
// s = seq_ids[i]; the row at position p attends causally to entries 0..p:
//   out[row, h] = sum_{j <= p} softmax_j(scale q . K[s, j, g]) V[s, j, g],
//   g = h / G (grouped query).
//
// One workgroup of four waves per (request, kv head, block of positions).
// It holds 256 query vectors: BQ = 256 / G positions x the G query heads of
// kv head g, so every K/V tile it loads serves all of them.  A wave owns 64
// vectors as two 32-column blocks of the transposed score tile
//   S^T (32 keys x 32 queries) = K (32 x D) . Q^T        (v_mfma_f32_32x32x16_bf16)
// and accumulates
//   O^T (D x 32 queries) += V^T (D x 32 keys) . P^T.
// In S^T a lane holds 16 keys of one query column, so the softmax row
// statistics need one lane swap per tile.  The K rows of a tile are read in
// a permuted order so that the 16 scores a lane holds are exactly the keys
// its PV operand needs (8 contiguous tokens per 16-key step): no shuffle
// between the two products.  K/V tiles of 32 keys go through LDS, the next
// tile's global loads in flight while the current one is multiplied.
#include "common.hpp"

typedef float f32x16_t __attribute__((ext_vector_type(16)));

namespace sm {

constexpr int kPfThreads = 256;
constexpr int kPfVec = 256;   // query vectors per workgroup
constexpr int kPfKeys = 32;   // keys per tile
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
  int n, total_rows, max_rows, Hkv, Hq, G, BQ, bs_log2, num_blocks, max_seqs, max_blocks;
  float scale_log2e;
};

// Score-tile row rho (0..31) holds token tau(rho) of the tile: within each
// 16 rows the middle two groups of four swap places, so that the rows a lane
// holds after S^T = K . Q^T ({8 g + 4 h + e}) are tokens 8 h .. 8 h + 7 of
// each 16-key step, in register order.
__device__ __forceinline__ int pf_token_of_row(int rho) {
  const int q = (rho >> 2) & 3;
  const int q2 = q == 1 ? 2 : q == 2 ? 1 : q;
  return (rho & ~15) | (q2 << 2) | (rho & 3);
}

template <int DH>
__global__ __launch_bounds__(kPfThreads, 1) void prefill_bf16(PrefillArgs a) {
  constexpr int KP = DH + 8;        // K tile row pitch (bf16)
  constexpr int VP = kPfKeys + 8;   // V tile row pitch (bf16)
  constexpr int NKS = DH / 16;      // k steps of S^T
  constexpr int NRB = DH / 32;      // 32-dim row blocks of O^T
  constexpr int KCH = DH / 8;       // 16-byte chunks of a K row
  constexpr int KU = kPfKeys * KCH / kPfThreads;  // K chunks per thread and tile
  constexpr int VU = DH * (kPfKeys / 8) / kPfThreads;  // V chunks per thread and tile
  static_assert(KU * kPfThreads == kPfKeys * KCH && VU * kPfThreads == DH * (kPfKeys / 8), "tile split");
  __shared__ int pages[kPfMaxPages];
  __shared__ int bad_flag;
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[2][kPfKeys * KP];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[2][DH * VP];

  const int qb = gridDim.x - 1 - blockIdx.x;  // longest blocks first
  const int g = blockIdx.y, i = blockIdx.z;
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

  // ---- this wave's 64 query vectors: v = 64 w + 32 cb + c32 ----
  // vector v -> query head g G + v / BQ, row q_lo + v % BQ
  int vpos[2], vrow[2], vhead[2];
  bool vok[2];
  u32x4_t qf[2][NKS];
#pragma unroll
  for (int cb = 0; cb < 2; ++cb) {
    const int v = 64 * w + 32 * cb + c32;
    const int hh = v / a.BQ, rr = v - hh * a.BQ;
    vok[cb] = hh < a.G && rr < nq;
    vhead[cb] = g * a.G + (vok[cb] ? hh : 0);
    vrow[cb] = r0 + q_lo + (vok[cb] ? rr : 0);
    vpos[cb] = vok[cb] ? pos0 + rr : -1;  // an idle vector sees no key
    const uint16_t *qp = a.q + ((int64_t)vrow[cb] * a.Hq + vhead[cb]) * DH + 8 * h2;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      qf[cb][ks] = vok[cb] ? *(const u32x4_t *)(qp + 16 * ks) : u32x4_t{0u, 0u, 0u, 0u};
  }

  // ---- tile loader: 2 K chunks and 2 V chunks of 16 bytes per thread ----
  const int64_t page_elems = (int64_t)bs * DH;
  auto fetch = [&](int t0, u32x4_t (&kv)[KU + VU]) {
#pragma unroll
    for (int u = 0; u < KU; ++u) {
      const int id = tid + kPfThreads * u;
      // K: token id / KCH, 8 dims (id % KCH); tokens past kend re-read token 0
      int tok = t0 + id / KCH;
      if (tok >= kend) tok = 0;
      const int blk = pages[tok >> bs_log2];
      kv[u] = *(const u32x4_t *)(a.k_pool + ((int64_t)blk * a.Hkv + g) * page_elems +
                                 (int64_t)(tok & (bs - 1)) * DH + (id % KCH) * 8);
    }
#pragma unroll
    for (int u = 0; u < VU; ++u) {
      const int id = tid + kPfThreads * u;
      // V: dim id / 4, tokens 8 (id % 4) .. + 7 (one page: bs >= 8)
      const int d = id >> 2;
      int tok = t0 + 8 * (id & 3);
      const int nvalid = min(8, L - tok);  // entries past the length may hold anything
      if (tok >= kend) tok = 0;
      const int blk = pages[tok >> bs_log2];
      u32x4_t x = *(const u32x4_t *)(a.v_pool + ((int64_t)blk * a.Hkv + g) * page_elems + (int64_t)d * bs +
                                     (tok & (bs - 1)));
      if (nvalid < 8) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (2 * e >= nvalid) x[e] = 0u;
          else if (2 * e + 1 >= nvalid) x[e] &= 0xffffu;
        }
      }
      kv[KU + u] = x;
    }
  };
  auto stash = [&](int buf, const u32x4_t (&kv)[KU + VU]) {
#pragma unroll
    for (int u = 0; u < KU; ++u) {
      const int id = tid + kPfThreads * u;
      *(u32x4_t *)(&k_lds[buf][(id / KCH) * KP + (id % KCH) * 8]) = kv[u];
    }
#pragma unroll
    for (int u = 0; u < VU; ++u) {
      const int id = tid + kPfThreads * u;
      *(u32x4_t *)(&v_lds[buf][(id >> 2) * VP + 8 * (id & 3)]) = kv[KU + u];
    }
  };

  f32x16_t o[2][NRB];
#pragma unroll
  for (int cb = 0; cb < 2; ++cb)
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[cb][rb][e] = 0.f;
  float m_run[2] = {-INFINITY, -INFINITY}, l_run[2] = {0.f, 0.f};
  const float sl2 = a.scale_log2e;
  const int krow = pf_token_of_row(c32);  // this lane's K row in the S^T operand
  // every vector of the workgroup sees key t when t <= pos0: no mask below
  const int vpos_min = pos0;

  const int ntiles = (kend + kPfKeys - 1) / kPfKeys;
  u32x4_t stage[KU + VU];
  fetch(0, stage);
  stash(0, stage);
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1, t0 = t * kPfKeys;
    if (t + 1 < ntiles) fetch(t0 + kPfKeys, stage);  // in flight during this tile

    // S^T = K . Q^T for both column blocks
    const uint16_t *kl = &k_lds[buf][krow * KP + 8 * h2];
    f32x16_t sc[2];
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[cb][e] = 0.f;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const u32x4_t kf = *(const u32x4_t *)(kl + 16 * ks);
#pragma unroll
      for (int cb = 0; cb < 2; ++cb)
        sc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kf), as_bf16x8(qf[cb][ks]), sc[cb], 0, 0, 0);
    }

    // online softmax per query column; register 4 gg + e holds token
    // t0 + 8 (gg >> 1) * 2 ... : row 8 gg + 4 h2 + e -> token pf_token_of_row(row)
    const bool need_mask = t0 + kPfKeys - 1 > vpos_min;
    u32x4_t pf[2][2];
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
      float x[16];
      float mx = -INFINITY;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int tok = t0 + pf_token_of_row(8 * (r >> 2) + 4 * h2 + (r & 3));
        const bool valid = !need_mask || tok <= vpos[cb];
        x[r] = valid ? sc[cb][r] * sl2 : -INFINITY;
        mx = fmaxf(mx, x[r]);
      }
      float a0, b0;
      swap32(mx, a0, b0);
      mx = fmaxf(a0, b0);
      const float m_new = fmaxf(m_run[cb], mx);
      const float mb = m_new == -INFINITY ? 0.f : m_new;  // a column with no key yet
      const float alpha = exp2f(m_run[cb] - mb);
      float ps = 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        x[r] = exp2f(x[r] - mb);
        ps += x[r];
      }
      l_run[cb] = l_run[cb] * alpha + ps;
      m_run[cb] = m_new;
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb) o[cb][rb] *= alpha;
#pragma unroll
      for (int kst = 0; kst < 2; ++kst)
        pf[cb][kst] = u32x4_t{pack_bf16x2(x[8 * kst + 0], x[8 * kst + 1]), pack_bf16x2(x[8 * kst + 2], x[8 * kst + 3]),
                              pack_bf16x2(x[8 * kst + 4], x[8 * kst + 5]), pack_bf16x2(x[8 * kst + 6], x[8 * kst + 7])};
    }

    // O^T += V^T . P^T: lane (d, h2) feeds dims 32 rb + d, tokens 16 kst + 8 h2 .. +7
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int kst = 0; kst < 2; ++kst) {
        const u32x4_t vf = *(const u32x4_t *)(&v_lds[buf][(32 * rb + c32) * VP + 16 * kst + 8 * h2]);
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
          o[cb][rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vf), as_bf16x8(pf[cb][kst]), o[cb][rb], 0, 0, 0);
      }

    if (t + 1 < ntiles) stash(buf ^ 1, stage);
    __syncthreads();
  }

  // ---- normalize and store: register 4 gg + e of block rb = dim 32 rb + 8 gg + 4 h2 + e ----
#pragma unroll
  for (int cb = 0; cb < 2; ++cb) {
    float a0, b0;
    swap32(l_run[cb], a0, b0);
    const float l_tot = a0 + b0;
    const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
    if (!vok[cb]) continue;
    uint16_t *op = a.out + ((int64_t)vrow[cb] * a.Hq + vhead[cb]) * DH + 4 * h2;
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int gg = 0; gg < 4; ++gg) {
        const f32x16_t &acc = o[cb][rb];
        *(uint2 *)(op + 32 * rb + 8 * gg) =
            make_uint2(pack_bf16x2(acc[4 * gg + 0] * inv, acc[4 * gg + 1] * inv),
                       pack_bf16x2(acc[4 * gg + 2] * inv, acc[4 * gg + 3] * inv));
      }
  }
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
  if (c->dtype != SM_BF16) return SM_EINVAL;
  const int H = c->num_kv_heads, D = c->head_dim, bs = c->block_size;
  if (H <= 0 || num_q_heads <= 0 || num_q_heads % H != 0) return SM_EINVAL;
  const int G = num_q_heads / H;
  if (G > 16 || (D != 64 && D != 128)) return SM_EINVAL;
  if (bs < 16 || (bs & (bs - 1)) != 0 || c->max_blocks_per_seq <= 0 || c->max_blocks_per_seq > kPfMaxPages ||
      c->num_blocks <= 0 || c->max_seqs <= 0)
    return SM_EINVAL;
  if (n > 65535) return SM_EINVAL;
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
  a.scale_log2e = scale * kPfLog2e;
  const int nqb = max_rows > 0 ? (max_rows + a.BQ - 1) / a.BQ : 1;  // block 0 reports bad requests
  if (nqb > (1 << 30)) return SM_EINVAL;
  const dim3 grid(nqb, H, n);
  if (D == 128)
    hipLaunchKernelGGL(prefill_bf16<128>, grid, dim3(kPfThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(prefill_bf16<64>, grid, dim3(kPfThreads), 0, stream, a);
  return hipGetLastError() == hipSuccess ? SM_OK : SM_EHIP;
}
