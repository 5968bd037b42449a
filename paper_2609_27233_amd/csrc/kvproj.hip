// The K/V state of one input row per request at its compressed position
// (gfx950).
//
// After a decode-time merge the frozen backbone takes the surrogate z_s as
// one input embedding and produces one K/V state per layer for the span
// (appendix "Decoding-time Integration").  For the first attention layer
// that state is
//   K = RoPE_p(W_k RMSNorm(x)),  V = W_v RMSNorm(x),
// with x the step's input row (a surrogate or a plain token embedding), p
// the slot it takes in the cache (the sequence's length after the crop),
// and the norm's gain folded into W_k and W_v.
//
// The projection is a skinny product: a handful of rows against 2 Hkv D x d
// weights (16 MB at d = 4096, Hkv D = 1024), so it is bound by streaming
// the weights once.  RMSNorm is a per-row scalar and commutes with the
// product, so the product runs on the raw rows:
//  1. split-K MFMA partials: a workgroup takes 64 output features x 256 of
//     the d inputs for up to 64 rows (v_mfma_f32_16x16x32_bf16, the rows'
//     slice staged in LDS, the weight fragments loaded straight into the
//     operand registers), 256 x d/256 workgroups for d = 4096;
//  2. one workgroup per (row, 256 output features) sums the partials in a
//     fixed order (the result does not depend on scheduling), scales by
//     1/rms, rotates K by the position (the angle formed and reduced in
//     double precision, then fp32 sin/cos) and writes bf16 rows;
//  3. sm_kv_append_projected then appends those rows (block allocation and
//     all checks of sm_kv_append).
#include "common.hpp"

namespace sm {

constexpr int kPjThreads = 256;
constexpr int kPjRows = 64;   // rows per workgroup
constexpr int kPjFeat = 64;   // output features per workgroup, 16 per wave
constexpr int kPjK = 256;     // inputs per workgroup
constexpr int kPjMaxChunks = 64;  // d <= 64 x 256

struct ProjArgs {
  const uint16_t *x;   // [n][d]
  const uint16_t *Wk;  // [HD][d]
  const uint16_t *Wv;  // [HD][d]
  float *part;         // [d / kPjK][n][2 HD]
  int n, d, HD;
};

__global__ __launch_bounds__(kPjThreads) void kv_proj_partial_kernel(ProjArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t xs[kPjRows][kPjK + 8];
  const int fb = blockIdx.x, kc = blockIdx.y, rg = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int r = lane & 15, q4 = lane >> 4;
  const int f0 = fb * kPjFeat + 16 * w;  // this wave's 16 features: all K (f0 < HD) or all V
  const uint16_t *W = f0 < a.HD ? a.Wk + (int64_t)f0 * a.d : a.Wv + (int64_t)(f0 - a.HD) * a.d;
  const int k0 = kc * kPjK, r0 = rg * kPjRows;
  const int nr = min(kPjRows, a.n - r0);
  // weight fragments: lane (r, q4) holds W[f0 + r][k0 + 32 s + 8 q4 .. +7]
  u32x4_t wf[kPjK / 32];
#pragma unroll
  for (int s = 0; s < kPjK / 32; ++s)
    wf[s] = __builtin_nontemporal_load((const u32x4_t *)(W + (int64_t)r * a.d + k0 + 32 * s + 8 * q4));
  // the rows' slice k0 .. k0 + 255 into LDS (rows past n are zero)
  const int rows16 = (nr + 15) & ~15;  // whole 16-row tiles
  for (int c = tid; c < rows16 * (kPjK / 8); c += kPjThreads) {
    const int row = c / (kPjK / 8), ch = c % (kPjK / 8);
    u32x4_t v = u32x4_t{0u, 0u, 0u, 0u};
    if (row < nr) v = *(const u32x4_t *)(a.x + (int64_t)(r0 + row) * a.d + k0 + 8 * ch);
    *(u32x4_t *)&xs[row][8 * ch] = v;
  }
  __syncthreads();
  const int ntile = (nr + 15) >> 4;
  f32x4_t acc[kPjRows / 16];
#pragma unroll
  for (int t = 0; t < kPjRows / 16; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < kPjK / 32; ++s)
#pragma unroll
    for (int t = 0; t < kPjRows / 16; ++t)
      if (t < ntile) {
        // x operand: lane (r, q4) holds row 16 t + r, inputs 32 s + 8 q4 .. +7
        const u32x4_t xf = *(const u32x4_t *)&xs[16 * t + r][32 * s + 8 * q4];
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(xf), as_bf16x8(wf[s]), acc[t], 0, 0, 0);
      }
  // lane (r, q4), register e: row 16 t + 4 q4 + e, feature f0 + r
#pragma unroll
  for (int t = 0; t < kPjRows / 16; ++t)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int row = 16 * t + 4 * q4 + e;
      if (row < nr) a.part[((int64_t)kc * a.n + r0 + row) * (2 * a.HD) + f0 + r] = acc[t][e];
    }
}

struct ProjEpiArgs {
  const uint16_t *x;
  const float *part;
  const int32_t *seq_ids;
  const int32_t *lengths;
  uint16_t *K, *V;        // [n][HD] bf16
  int32_t *row_offsets;   // [n + 1] (nullable)
  int n, d, HD, D, nkc, max_seqs;
  float rms_eps;
  double inv_freq[64];    // theta^(-2j/D), j < D/2, computed on the host
};

constexpr double kTwoPi = 6.283185307179586476925286766559;

// One workgroup per (block of 256 output features, row): a block covers
// whole heads, so both halves of every rotary pair are at hand.
__global__ __launch_bounds__(kPjThreads) void kv_proj_epilogue_kernel(ProjEpiArgs a) {
  __shared__ float ys[kPjThreads];
  __shared__ float red[16];
  const int fb = blockIdx.x, i = blockIdx.y, tid = threadIdx.x;
  const int f = fb * kPjThreads + tid;  // K features first, then V
  const int s = a.seq_ids[i];
  const double pos = (s >= 0 && s < a.max_seqs) ? (double)a.lengths[s] : 0.0;  // bad ids fail in the append
  // the split-K partials, summed in a fixed order once all are loaded; their
  // loads are in flight while the row's RMSNorm scale is reduced
  float pv[kPjMaxChunks];
#pragma unroll
  for (int kc = 0; kc < kPjMaxChunks; ++kc)
    pv[kc] = kc < a.nkc ? a.part[((int64_t)kc * a.n + i) * (2 * a.HD) + f] : 0.f;
  float ss = 0.f;
  for (int k = 8 * tid; k < a.d; k += 8 * kPjThreads) {
    const u32x4_t v = *(const u32x4_t *)(a.x + (int64_t)i * a.d + k);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = __uint_as_float(v[e] << 16), hi = __uint_as_float(v[e] & 0xffff0000u);
      ss += lo * lo + hi * hi;
    }
  }
  ss = block_sum(ss, red);
  const float inv = rsqrtf(ss / a.d + a.rms_eps);
  float y = 0.f;
#pragma unroll
  for (int kc = 0; kc < kPjMaxChunks; ++kc) y += pv[kc];
  y *= inv;
  ys[tid] = y;
  __syncthreads();
  if (f < a.HD) {
    // rotate-half RoPE: pair (j, j + D/2) turned by pos theta^(-2j/D); the
    // angle is formed and reduced to [-pi, pi] in double precision
    const int half = a.D / 2, jd = f % a.D, j = jd % half;
    const double ang = pos * a.inv_freq[j];
    const float r = (float)(ang - kTwoPi * rint(ang / kTwoPi));
    const float c = cosf(r), sn = sinf(r);
    const float other = ys[jd < half ? tid + half : tid - half];
    const float out = jd < half ? y * c - other * sn : y * c + other * sn;
    a.K[(int64_t)i * a.HD + f] = f32_to_bf16(out);
  } else {
    a.V[(int64_t)i * a.HD + f - a.HD] = f32_to_bf16(y);
  }
  if (a.row_offsets && fb == 0 && tid == 0) {
    a.row_offsets[i] = i;
    if (i == a.n - 1) a.row_offsets[a.n] = a.n;
  }
}

static size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

static size_t part_bytes(int n, int d, int HD) { return align256((size_t)(d / kPjK) * n * 2 * HD * sizeof(float)); }

}  // namespace sm

using namespace sm;

static bool proj_ok(const sm_paged_cache *c, int n, const void *x, const sm_kv_proj_params *p) {
  if (!c || !p || n < 0 || n > SM_MAX_REQUESTS || n > c->max_seqs) return false;
  if (c->dtype != SM_BF16 || (c->head_dim != 64 && c->head_dim != 128) || c->num_kv_heads <= 0) return false;
  const int HD = c->num_kv_heads * c->head_dim;
  if (HD > 2048 || (2 * HD) % kPjThreads != 0) return false;
  if (p->d <= 0 || p->d % kPjK != 0 || p->d > kPjK * kPjMaxChunks || !(p->rope_theta > 0.f) ||
      !(p->rms_eps >= 0.f))
    return false;
  return n == 0 || (x && p->W_k && p->W_v && c->lengths);
}

SM_API size_t sm_kv_project_workspace_bytes(int n, int d, int num_kv_heads, int head_dim) {
  if (n < 0 || d <= 0 || d % kPjK != 0 || d > kPjK * kPjMaxChunks || num_kv_heads <= 0 || head_dim <= 0)
    return 0;
  const int HD = num_kv_heads * head_dim;
  return part_bytes(n, d, HD) + 2 * align256((size_t)n * HD * 2) + align256((size_t)(n + 1) * 4);
}

static sm_status launch_project(const sm_paged_cache *c, const int32_t *seq_ids, int n, const void *x,
                                const sm_kv_proj_params *p, void *K, void *V, int32_t *row_offsets, float *part,
                                hipStream_t stream) {
  const int HD = c->num_kv_heads * c->head_dim;
  ProjArgs a{(const uint16_t *)x, (const uint16_t *)p->W_k, (const uint16_t *)p->W_v, part, n, p->d, HD};
  const dim3 grid(2 * HD / kPjFeat, p->d / kPjK, (n + kPjRows - 1) / kPjRows);
  hipLaunchKernelGGL(kv_proj_partial_kernel, grid, dim3(kPjThreads), 0, stream, a);
  ProjEpiArgs e{(const uint16_t *)x, part, seq_ids, c->lengths, (uint16_t *)K, (uint16_t *)V, row_offsets,
                n, p->d, HD, c->head_dim, p->d / kPjK, c->max_seqs, p->rms_eps, {}};
  for (int j = 0; j < c->head_dim / 2; ++j) e.inv_freq[j] = pow((double)p->rope_theta, -2.0 * j / c->head_dim);
  hipLaunchKernelGGL(kv_proj_epilogue_kernel, dim3(2 * HD / kPjThreads, n), dim3(kPjThreads), 0, stream, e);
  return hipGetLastError() == hipSuccess ? SM_OK : SM_EHIP;
}

SM_API sm_status sm_kv_project(const sm_paged_cache *c, const int32_t *seq_ids, int n, const void *x,
                               const sm_kv_proj_params *p, void *K, void *V, void *ws, size_t ws_bytes,
                               hipStream_t stream) {
  if (!proj_ok(c, n, x, p)) return SM_EINVAL;
  if (n == 0) return SM_OK;
  if (!seq_ids || !K || !V || !ws ||
      ws_bytes < sm_kv_project_workspace_bytes(n, p->d, c->num_kv_heads, c->head_dim))
    return SM_EINVAL;
  return launch_project(c, seq_ids, n, x, p, K, V, nullptr, (float *)ws, stream);
}

SM_API sm_status sm_kv_append_projected(const sm_paged_cache *c, const int32_t *seq_ids, int n, const void *x,
                                        const sm_kv_proj_params *p, void *ws, size_t ws_bytes,
                                        hipStream_t stream) {
  if (!proj_ok(c, n, x, p)) return SM_EINVAL;
  // the append's own synchronous checks first: nothing is enqueued on failure
  if (sm_kv_append(c, seq_ids, nullptr, 0, 0, nullptr, nullptr, stream) != SM_OK) return SM_EINVAL;
  if (n == 0) return SM_OK;
  if (!seq_ids || !ws || ws_bytes < sm_kv_project_workspace_bytes(n, p->d, c->num_kv_heads, c->head_dim))
    return SM_EINVAL;
  const int HD = c->num_kv_heads * c->head_dim;
  char *w = (char *)ws;
  float *part = (float *)w;
  w += part_bytes(n, p->d, HD);
  void *K = w;
  w += align256((size_t)n * HD * 2);
  void *V = w;
  w += align256((size_t)n * HD * 2);
  int32_t *offs = (int32_t *)w;
  const sm_status st = launch_project(c, seq_ids, n, x, p, K, V, offs, part, stream);
  if (st != SM_OK) return st;
  return sm_kv_append(c, seq_ids, offs, n, n, K, V, stream);
}
