// Merge module M_phi over many spans at once (gfx950).
//
// The module (paper Sec. 3.2 Eq. 1 and the appendix "Attention-based Pooling
// Architecture") maps the n static embeddings E_s of a span to one surrogate:
//   P   = LN_kv(GELU(E_s W_kv^T + b_kv))
//   a_i = softmax_j(P[j, head i] . q_i / sqrt(d_h)),   o_i = sum_j a_i[j] P[j, head i]
//   z_s = LN_o(GELU([o_1; ...; o_h] W_o^T + b_o))
//
// All spans of a call, of any length, are processed together (CSR offsets):
//   1. GEMM1  G1 = GELU(emb[row_idx] W_kv^T + b_kv)   row-gathered A operand,
//             bf16 matrix cores (v_mfma_f32_16x16x32_bf16), fp32 accumulate
//   2. pool   one workgroup per span: exact LN_kv row statistics, the h
//             head scores, softmax over the span, pooled row c_s
//   3. GEMM2  Y = GELU(c W_o^T + b_o)                 (fp32 out)
//   4. LN_o   z_s = LN_o(Y_s)
// The fp32 dtype runs the same four steps with a vector-ALU GEMM.
#include "common.hpp"

typedef float f32x16_t __attribute__((ext_vector_type(16)));

namespace sm {

// ---------------------------------------------------------------------------
// bf16 GEMM, C[M][N] = GELU(A[M][K] . B[N][K]^T + bias[N]); A rows optionally
// gathered through `gather`.  128x128 tile per workgroup, K step 64, four
// waves each owning a 64x64 quadrant (4x4 MFMA tiles of 16x16).  The next
// K step is fetched into registers while the current one is multiplied from
// LDS (double-buffered LDS, one barrier per step).

constexpr int kBM = 128, kBN = 128, kBK = 64;
constexpr int kPitch = kBK + 8;  // bf16 elements per LDS row (16-byte pad)

template <typename OutT>
__global__ __launch_bounds__(256, 2) void gemm_bf16_nt_gelu(const uint16_t *__restrict__ A,
                                                            const int32_t *__restrict__ gather,
                                                            int64_t a_rows, const uint16_t *__restrict__ B,
                                                            const uint16_t *__restrict__ bias,
                                                            OutT *__restrict__ C, int M, int N, int K,
                                                            int32_t *err) {
  __shared__ uint16_t As[2][kBM * kPitch];
  __shared__ uint16_t Bs[2][kBN * kPitch];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int r = lane & 15, q4 = lane >> 4;
  const int n0 = blockIdx.x * kBN, m0 = blockIdx.y * kBM;

  // each thread moves four 16-byte pieces of A and of B per K step
  const uint16_t *a_src[4];
  const uint16_t *b_src[4];
  int lds_off[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int id = tid + 256 * u;
    const int row = id >> 3, col = (id & 7) * 8;
    int64_t arow = m0 + row;
    if (gather) {
      int gi = (arow < M) ? gather[arow] : 0;
      if (gi < 0 || gi >= a_rows) {
        set_err(err, SM_ERR_EINVAL);
        gi = 0;
      }
      arow = gi;
    } else if (arow >= M) {
      arow = M - 1;
    }
    a_src[u] = A + arow * K + col;
    b_src[u] = B + (int64_t)(n0 + row) * K + col;
    lds_off[u] = row * kPitch + col;
  }

  f32x4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  u32x4_t ra[4], rb[4];
  const int nk = K / kBK;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    ra[u] = *(const u32x4_t *)(a_src[u]);
    rb[u] = *(const u32x4_t *)(b_src[u]);
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    *(u32x4_t *)(&As[0][lds_off[u]]) = ra[u];
    *(u32x4_t *)(&Bs[0][lds_off[u]]) = rb[u];
  }
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) {
      const int ko = (kt + 1) * kBK;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        ra[u] = *(const u32x4_t *)(a_src[u] + ko);
        rb[u] = *(const u32x4_t *)(b_src[u] + ko);
      }
    }
#pragma unroll
    for (int ks = 0; ks < kBK / 32; ++ks) {
      u32x4_t fa[4], fb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        fa[i] = *(const u32x4_t *)(&As[buf][(wm * 64 + i * 16 + r) * kPitch + ks * 32 + 8 * q4]);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        fb[j] = *(const u32x4_t *)(&Bs[buf][(wn * 64 + j * 16 + r) * kPitch + ks * 32 + 8 * q4]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(fa[i]), as_bf16x8(fb[j]), acc[i][j],
                                                              0, 0, 0);
    }
    if (kt + 1 < nk) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        *(u32x4_t *)(&As[buf ^ 1][lds_off[u]]) = ra[u];
        *(u32x4_t *)(&Bs[buf ^ 1][lds_off[u]]) = rb[u];
      }
    }
    __syncthreads();
  }

  // epilogue: lane (r, q4) of tile (i, j) holds rows 4*q4 + e, column r
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int col = n0 + wn * 64 + j * 16 + r;
    const float bcol = bf16_to_f32(bias[col]);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = m0 + wm * 64 + i * 16 + 4 * q4 + e;
        if (row < M) {
          const float v = gelu_erf(acc[i][j][e] + bcol);
          C[(int64_t)row * N + col] = Elem<OutT>::to_store(v);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Large bf16 GEMM, same contract as above: 256x256 output tile per
// workgroup, four waves in a 2 x 2 grid (128 x 128 each, accumulators in
// the accumulation registers, one wave per SIMD) on
// v_mfma_f32_32x32x16_bf16.  K advances 64 at a time through two LDS
// stages (2 x 64 KB) filled by global_load_lds_dwordx4, which moves 16
// bytes per lane from memory straight into LDS without staging registers.
// A 64-deep k-tile makes each operand row a 128-byte piece, so the L1 asks
// the L2 for whole 128-byte lines (a 32-deep tile sends twice as many
// 64-byte requests, and the L1 keeps only so many in flight).
//
// One k-tile is four k steps of 16 MFMAs.  Each wave holds a whole k-tile
// of fragments in registers (128 VGPRs): during k step 0 it reads those of
// k steps 1-3, then waits for them and passes a barrier, after which the
// stage is free; k steps 1 to 3 load the k-tile after next into it (one
// load every third MFMA, so the CU's requests reach the L2 evenly); before
// k step 3 each wave waits for its own loads of the next k-tile and passes
// a second barrier, and k step 3 reads the next k-tile's first fragments.
// Each load thus has four to six k steps to land.  The waits are explicit
// s_waitcnt and the instruction order is pinned by a scheduling barrier
// after each MFMA.
//
// LDS layout of one operand stage: 256 rows x 128 bytes as 16-byte slots
// row * 8 + (chunk ^ ((row >> 1) & 7)).  A 16-byte LDS read serves 16
// lanes per cycle from 64 banks (256 bytes): the 16 lanes of a fragment
// read take rows r .. r + 15 of one chunk; row parity picks the 128-byte
// half of the bank row and the swizzled chunk the slot within it, so the
// 16 reads hit 16 distinct bank groups.  A direct-to-LDS load writes 64
// consecutive slots (one per lane): lane l of a load covers row
// base + l / 8, slot l % 8, and fetches global chunk (l % 8) ^ swizzle(row).
//
// Tile order: the hardware hands workgroup b to XCD b % 8; XCD x takes the
// logical tiles [x * per_xcd, (x + 1) * per_xcd) in groups of kGroupM row
// tiles, so the 32 tiles in flight on one XCD share A rows and B columns
// in its L2.  Each tile walks K from a rotated start: one k-tile per
// column tile (the 8 column tiles in flight on an XCD are at most 8
// k-tiles apart, so the A rows they share stay in L2) plus an eighth of K
// per XCD, so that the eight XCDs do not ask for the same k offsets of
// their rows, and of W, at the same time (measured 2.5-4% faster than all
// tiles walking K from 0).  The sum over K of one output element thus
// depends on its column tile and on the XCD its tile lands on.

constexpr int kLM = 256, kLN = 256, kLK = 64, kLStages = 2, kLThreads = 256, kGroupM = 4;
constexpr int kLStageBytes = kLM * kLK * 2;  // per operand
constexpr int kLLdsBytes = 2 * kLStages * kLStageBytes;

__device__ __forceinline__ int lds_swz(int row) { return (row >> 1) & 7; }

// s_waitcnt with vmcnt = N, lgkmcnt = 0, expcnt left open
template <int N>
__device__ __forceinline__ void wait_vmcnt_lgkm0() {
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}

__device__ __forceinline__ void load_to_lds16(const uint16_t *src, uint8_t *lds) {
  __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1))) *)src,
                                   (void __attribute__((address_space(3))) *)lds, 16, 0, 0);
}

template <typename OutT>
struct Store4;
template <>
struct Store4<float> {
  static __device__ __forceinline__ void put(float *p, float a, float b, float c, float d) {
    *(f32x4_t *)p = f32x4_t{a, b, c, d};
  }
};
template <>
struct Store4<uint16_t> {
  static __device__ __forceinline__ void put(uint16_t *p, float a, float b, float c, float d) {
    *(uint2 *)p = make_uint2(pack_bf16x2(a, b), pack_bf16x2(c, d));
  }
};

template <typename OutT>
__global__ __launch_bounds__(kLThreads, 1) void gemm256_bf16_nt_gelu(
    const uint16_t *__restrict__ A, const int32_t *__restrict__ gather, int64_t a_rows,
    const uint16_t *__restrict__ B, const uint16_t *__restrict__ bias, OutT *__restrict__ C, int M, int N, int K,
    int tiles_m, int tiles_n, int per_xcd, int staged, int32_t *err) {
  extern __shared__ __attribute__((aligned(1024))) uint8_t lds[];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = w >> 1, wn = w & 1;  // this wave's 128 x 128 block of the tile
  const int xcd = blockIdx.x & 7;
  const int t = xcd * per_xcd + (blockIdx.x >> 3);
  if (t >= tiles_m * tiles_n) return;
  const int gsz = kGroupM * tiles_n;
  const int g0 = (t / gsz) * kGroupM;
  const int gm = min(kGroupM, tiles_m - g0);
  const int tm = g0 + (t % gsz) % gm, tn = (t % gsz) / gm;
  const int m0 = tm * kLM, n0 = tn * kLN;
  const int nk = K / kLK;
  const int rot = (tn + xcd * (nk / 8)) % nk;  // first k-tile of this tile's walk

  // Loads: per k-tile and operand, 32 direct-to-LDS loads of 1 KB (8 rows
  // of 128 bytes); load u of wave w covers rows (4 u + w) * 8 + lane / 8.
  // A rows past M re-read a valid row.
  const uint16_t *pa[8];
  const uint16_t *pb;
  {
    const int lrow = lane >> 3;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int row = (4 * u + w) * 8 + lrow;
      const int chunk = (lane & 7) ^ lds_swz(row);
      int64_t arow = m0 + row;
      if (gather) {
        int gi = (arow < M) ? gather[arow] : 0;
        if (gi < 0 || gi >= a_rows) {
          set_err(err, SM_ERR_EINVAL);
          gi = 0;
        }
        arow = gi;
      } else if (arow >= M) {
        arow = M - 1;
      }
      pa[u] = A + arow * K + chunk * 8;
    }
    // the B rows of load u are those of load 0 plus 32 u (same swizzle)
    const int row0 = w * 8 + lrow;
    pb = B + (int64_t)(n0 + row0) * K + ((lane & 7) ^ lds_swz(row0)) * 8;
  }
  const int64_t bstep = (int64_t)32 * K;
  uint8_t *sa = lds, *sb = lds + kLStages * kLStageBytes;
  auto load_q = [&](int kt, int stage, int q) {  // load q (A 0-7, B 8-15) of the kt-th k-tile of the walk
    const int kr = kt + rot;
    const int ko = (kr >= nk ? kr - nk : kr) * kLK;
    const int u = q & 7;
    if (q < 8) load_to_lds16(pa[u] + ko, sa + stage * kLStageBytes + (4 * u + w) * 1024);
    else load_to_lds16(pb + u * bstep + ko, sb + stage * kLStageBytes + (4 * u + w) * 1024);
  };

  // 32x32x16 operands: lane l feeds row l % 32, k 8 (l / 32) .. +7 of a
  // 16-deep k step ks, i.e. chunk 2 ks + l / 32 of the 128-byte row
  const int r32 = lane & 31, h2 = lane >> 5;
  int fo[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) fo[ks] = r32 * 128 + (((2 * ks + h2) ^ lds_swz(r32)) * 16);
  const int a_off = wm * 128 * 128, b_off = wn * 128 * 128;

  f32x16_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // k-tiles 0 and 1 in stages 0 and 1; the fragments of k step 0
  u32x4_t fa[4][4], fb[4][4];  // [k step][32-row block]
#pragma unroll
  for (int q = 0; q < 16; ++q) load_q(0, 0, q);
#pragma unroll
  for (int q = 0; q < 16; ++q) load_q(1, 1, q);
  wait_vmcnt_lgkm0<16>();
  __builtin_amdgcn_s_barrier();
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    fa[0][i] = *(const u32x4_t *)(sa + a_off + i * 4096 + fo[0]);
    fb[0][i] = *(const u32x4_t *)(sb + b_off + i * 4096 + fo[0]);
  }

  // One k step KS of the k-tile kt in stage ST: 16 MFMAs over the 4 x 4
  // accumulators, each followed by
  //  * k step 0: two of the 24 fragment reads of k steps 1-3 (after MFMAs
  //    0-11);
  //  * k steps 1, 2 and 3: every third MFMA, one of the 16 loads of k-tile
  //    kt + 2 into this (by then free) stage (6, 5 and 5 of them); past the
  //    end of K the last k-tile is loaded again (never read), so that every
  //    wait counts the same loads;
  //  * k step 3: also one of the 8 fragment reads of k step 0 of k-tile
  //    kt + 1 (after MFMAs 0-7), from the other stage.
#define SM_KSTEP(ST, KS)                                                                             \
  {                                                                                                  \
    const int kn2_ = min(kt + 2, nk - 1);                                                            \
    _Pragma("unroll") for (int g = 0; g < 16; ++g) {                                                 \
      const int i = g >> 2, j = g & 3;                                                               \
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(fb[KS][j]), as_bf16x8(fa[KS][i]), \
                                                          acc[i][j], 0, 0, 0);                       \
      if ((KS) == 0) {                                                                               \
        if (g < 12) {                                                                                \
          const int rk_ = 1 + g / 4, rq_ = g & 3;                                                    \
          fa[rk_][rq_] = *(const u32x4_t *)(sa + (ST) * kLStageBytes + a_off + fo[rk_] + rq_ * 4096); \
          fb[rk_][rq_] = *(const u32x4_t *)(sb + (ST) * kLStageBytes + b_off + fo[rk_] + rq_ * 4096); \
        }                                                                                            \
      } else if ((KS) == 1 || (KS) == 2) {                                                           \
        if (g % 3 == 0 && ((KS) == 1 || g < 15)) load_q(kn2_, (ST), ((KS) - 1) * 6 + g / 3);         \
      } else {                                                                                       \
        if (g < 8) {                                                                                 \
          const int o_ = ((ST) ^ 1) * kLStageBytes + fo[0] + (g >> 1) * 4096;                        \
          if (g & 1) fb[0][g >> 1] = *(const u32x4_t *)(sb + b_off + o_);                            \
          else fa[0][g >> 1] = *(const u32x4_t *)(sa + a_off + o_);                                  \
        }                                                                                            \
        if (g % 3 == 1 && g < 15) load_q(kn2_, (ST), 11 + g / 3);                                    \
      }                                                                                              \
      __builtin_amdgcn_sched_barrier(0);                                                             \
    }                                                                                                \
  }
  // A k-tile: k step 0; this wave's fragment reads done, barrier (the stage
  // is free: every wave holds the k-tile in registers); k steps 1 and 2;
  // this wave's loads of k-tile kt + 1 done (the 11 of kt + 2 issued since
  // may still be in flight), barrier (k-tile kt + 1 is in LDS); k step 3.
#define SM_KTILE(ST)                                                                                 \
  {                                                                                                  \
    SM_KSTEP(ST, 0);                                                                                 \
    wait_vmcnt_lgkm0<16>();                                                                          \
    __builtin_amdgcn_s_barrier();                                                                    \
    __builtin_amdgcn_sched_barrier(0);                                                               \
    SM_KSTEP(ST, 1);                                                                                 \
    SM_KSTEP(ST, 2);                                                                                 \
    wait_vmcnt_lgkm0<11>();                                                                          \
    __builtin_amdgcn_s_barrier();                                                                    \
    __builtin_amdgcn_sched_barrier(0);                                                               \
    SM_KSTEP(ST, 3);                                                                                 \
  }
  for (int kt = 0; kt < nk; ++kt) {  // nk is even: stage 0, then stage 1
    SM_KTILE(0);
    ++kt;
    SM_KTILE(1);
  }
#undef SM_KTILE
#undef SM_KSTEP
  wait_vmcnt_lgkm0<0>();

  // 32x32 result layout (swapped): register 4 g + e of tile (i, j) holds
  // C[row 32 i + r32][col 32 j + 8 g + 4 h2 + e]
  if (!staged) {  // straight from the MFMA layout (grids of a few waves of tiles)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int col = n0 + wn * 128 + j * 32 + 8 * g + 4 * h2;
        const uint2 bb = *(const uint2 *)(bias + col);
        const float b0 = __uint_as_float(bb.x << 16), b1 = __uint_as_float(bb.x & 0xffff0000u);
        const float b2 = __uint_as_float(bb.y << 16), b3 = __uint_as_float(bb.y & 0xffff0000u);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = m0 + wm * 128 + i * 32 + r32;
          if (row < M)
            Store4<OutT>::put(C + (int64_t)row * N + col, gelu_erf(acc[i][j][4 * g + 0] + b0),
                              gelu_erf(acc[i][j][4 * g + 1] + b1), gelu_erf(acc[i][j][4 * g + 2] + b2),
                              gelu_erf(acc[i][j][4 * g + 3] + b3));
        }
      }
    }
    return;
  }
  // Epilogue through LDS, free once every wave is past the ring: the tile
  // (bias and GELU applied, in OutT) goes row-major into LDS, HR rows at a
  // time, with the 16-byte chunk c of row r at c ^ (r % CH); then the
  // workgroup stores whole rows, 16 bytes per lane.  Stored straight from
  // the MFMA layout, each lane's 8 or 16 bytes go to 32 rows per
  // instruction, and the partial lines reach memory in pieces (4x the
  // output's bytes written).  The swizzle makes the row reads free of bank
  // conflicts.  Staging serialises the tile's last phase, so it pays when
  // other workgroups' main loops overlap it: grids of many waves of tiles.
  constexpr int CH = kLN * (int)sizeof(OutT) / 16;               // 16-byte chunks per tile row
  constexpr int HR = kLLdsBytes / (kLN * (int)sizeof(OutT));     // tile rows per LDS pass
  constexpr int EPC = 16 / (int)sizeof(OutT);                    // elements per chunk
  __syncthreads();  // every wave's ring reads and loads are done
#pragma unroll
  for (int pass = 0; pass < kLM / HR; ++pass) {
    if (pass > 0) __syncthreads();  // the previous pass's rows are stored
    if (wm * 128 / HR == pass) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int lcol = wn * 128 + j * 32 + 8 * g + 4 * h2;
          const uint2 bb = *(const uint2 *)(bias + n0 + lcol);
          const float b0 = __uint_as_float(bb.x << 16), b1 = __uint_as_float(bb.x & 0xffff0000u);
          const float b2 = __uint_as_float(bb.y << 16), b3 = __uint_as_float(bb.y & 0xffff0000u);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int lrow = wm * 128 + i * 32 + r32 - pass * HR;
            const int c = lcol / EPC;
            uint8_t *dstl = lds + lrow * (CH * 16) + ((c ^ (lrow & (CH - 1))) * 16) + (lcol % EPC) * (int)sizeof(OutT);
            Store4<OutT>::put((OutT *)dstl, gelu_erf(acc[i][j][4 * g + 0] + b0), gelu_erf(acc[i][j][4 * g + 1] + b1),
                              gelu_erf(acc[i][j][4 * g + 2] + b2), gelu_erf(acc[i][j][4 * g + 3] + b3));
          }
        }
      }
    }
    __syncthreads();
#pragma unroll 8
    for (int k = 0; k < HR * CH / kLThreads; ++k) {
      const int q = tid + k * kLThreads, lrow = q / CH, c = q % CH;
      const int row = m0 + pass * HR + lrow;
      const u32x4_t v = *(const u32x4_t *)(lds + lrow * (CH * 16) + ((c ^ (lrow & (CH - 1))) * 16));
      if (row < M) *(u32x4_t *)(C + (int64_t)row * N + n0 + c * EPC) = v;
    }
  }
}

// Output tiles from which the 256-tile GEMM stages a bf16 epilogue through
// LDS.  Measured on the four-wave kernel: GEMM1 of the 70B-shaped batch
// (17,984 tiles) much faster staged (the direct stores wrote 4x the bytes);
// the second projection of the 16 x 4096 prompt batch (624 tiles) about 1%
// faster; so every bf16 output is staged (256 tiles is the kernel's
// minimum).  fp32 output stays direct (two LDS passes measured no better).
constexpr int kStagedMinTiles = 256;

static bool use_gemm256(int M, int N, int K) {
  return N % kLN == 0 && K % (2 * kLK) == 0 && K >= 2 * kLK * kLStages &&
         (int64_t)((M + kLM - 1) / kLM) * (N / kLN) >= 256;
}

template <typename OutT>
static hipError_t launch_gemm256(const uint16_t *A, const int32_t *gather, int64_t a_rows, const uint16_t *B,
                                 const uint16_t *bias, OutT *C, int M, int N, int K, int32_t *err,
                                 hipStream_t stream) {
  // dynamic LDS above 64 KB has to be enabled for the kernel (cheap; done
  // on every launch so that it holds on whichever device is current)
  const hipError_t e = hipFuncSetAttribute((const void *)gemm256_bf16_nt_gelu<OutT>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, kLLdsBytes);
  if (e != hipSuccess) return e;
  const int tiles_m = (M + kLM - 1) / kLM, tiles_n = N / kLN;
  const int per_xcd = (tiles_m * tiles_n + 7) / 8;
  const int staged = sizeof(OutT) == 2 && tiles_m * tiles_n >= kStagedMinTiles;
  hipLaunchKernelGGL(gemm256_bf16_nt_gelu<OutT>, dim3(8 * per_xcd), dim3(kLThreads), kLLdsBytes, stream, A, gather,
                     a_rows, B, bias, C, M, N, K, tiles_m, tiles_n, per_xcd, staged, err);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Skinny bf16 GEMM for M <= 64 rows (a decode-time merge of a few spans):
// C[M][N] = GELU(A[M][K] W[N][K]^T + bias).  One workgroup per 16 output
// columns (N / 16 workgroups, enough to keep every compute unit streaming
// its slice of W), the four waves split K and reduce through LDS.  Operand
// fragments are loaded straight from memory in MFMA layout, U k-steps of 32
// at a time so that U * (1 + m-tiles) 16-byte loads per lane are in flight.

constexpr int kSkinnyMaxM = 64;

template <typename OutT, int U>
__global__ __launch_bounds__(256) void gemm_skinny_bf16_gelu(const uint16_t *__restrict__ A,
                                                             const int32_t *__restrict__ gather, int64_t a_rows,
                                                             const uint16_t *__restrict__ W,
                                                             const uint16_t *__restrict__ bias,
                                                             OutT *__restrict__ C, int M, int N, int K,
                                                             int32_t *err) {
  __shared__ float red[4][kSkinnyMaxM][17];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int r = lane & 15, q4 = lane >> 4;
  const int n0 = blockIdx.x * 16;
  const int mt = (M + 15) >> 4;  // m-tiles (<= 4)
  const uint16_t *arow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = i * 16 + r;
    int64_t idx = 0;
    if (m < M) {
      idx = gather ? gather[m] : m;
      if (idx < 0 || idx >= a_rows) {
        set_err(err, SM_ERR_EINVAL);
        idx = 0;
      }
    }
    arow[i] = A + idx * K + 8 * q4;
  }
  const uint16_t *wrow = W + (int64_t)(n0 + r) * K + 8 * q4;
  const int kw = K >> 2, kbeg = w * kw;
  f32x4_t acc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  for (int k = kbeg; k < kbeg + kw; k += 32 * U) {
    u32x4_t bw[U], fa[U][4];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      bw[u] = *(const u32x4_t *)(wrow + k + 32 * u);
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (i < mt) fa[u][i] = *(const u32x4_t *)(arow[i] + k + 32 * u);
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (i < mt)
          acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(fa[u][i]), as_bf16x8(bw[u]), acc[i], 0, 0, 0);
  }
  // lane (r, q4) of m-tile i holds rows 16 i + 4 q4 + e, column r
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) red[w][i * 16 + 4 * q4 + e][r] = acc[i][e];
  __syncthreads();
  for (int o = tid; o < mt * 16 * 16; o += 256) {
    const int m = o >> 4, n = o & 15;
    if (m >= M) continue;
    const float v = red[0][m][n] + red[1][m][n] + red[2][m][n] + red[3][m][n];
    C[(int64_t)m * N + n0 + n] = Elem<OutT>::to_store(gelu_erf(v + bf16_to_f32(bias[n0 + n])));
  }
}

template <typename OutT>
static void launch_skinny(const uint16_t *A, const int32_t *gather, int64_t a_rows, const uint16_t *W,
                          const uint16_t *bias, OutT *C, int M, int N, int K, int32_t *err, hipStream_t stream) {
  const dim3 grid(N / 16), block(256);
  if ((K / 4) % (32 * 8) == 0)
    hipLaunchKernelGGL((gemm_skinny_bf16_gelu<OutT, 8>), grid, block, 0, stream, A, gather, a_rows, W, bias, C, M,
                       N, K, err);
  else if ((K / 4) % (32 * 4) == 0)
    hipLaunchKernelGGL((gemm_skinny_bf16_gelu<OutT, 4>), grid, block, 0, stream, A, gather, a_rows, W, bias, C, M,
                       N, K, err);
  else
    hipLaunchKernelGGL((gemm_skinny_bf16_gelu<OutT, 2>), grid, block, 0, stream, A, gather, a_rows, W, bias, C, M,
                       N, K, err);
}

// ---------------------------------------------------------------------------
// fp32 GEMM on the vector ALU (64x64 tile, 4x4 outputs per thread), same
// contract as the bf16 one.

constexpr int kFT = 64, kFK = 16;

__global__ __launch_bounds__(256) void gemm_f32_nt_gelu(const float *__restrict__ A,
                                                        const int32_t *__restrict__ gather, int64_t a_rows,
                                                        const float *__restrict__ B,
                                                        const float *__restrict__ bias, float *__restrict__ C,
                                                        int M, int N, int K, int32_t *err) {
  __shared__ float As[kFK][kFT + 4];
  __shared__ float Bs[kFK][kFT + 4];
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  const int n0 = blockIdx.x * kFT, m0 = blockIdx.y * kFT;
  // loader: 64 rows x 16 k per operand = 1024 floats, 4 per thread
  const int lrow = tid >> 2, lk = (tid & 3) * 4;
  int64_t arow = m0 + lrow;
  if (gather) {
    int gi = (arow < M) ? gather[arow] : 0;
    if (gi < 0 || gi >= a_rows) {
      set_err(err, SM_ERR_EINVAL);
      gi = 0;
    }
    arow = gi;
  } else if (arow >= M) {
    arow = M - 1;
  }
  const float *ap = A + arow * K + lk;
  const float *bp = B + (int64_t)(n0 + lrow) * K + lk;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += kFK) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      As[lk + u][lrow] = ap[k0 + u];
      Bs[lk + u][lrow] = bp[k0 + u];
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kFK; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + ty * 4 + i;
    if (row >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = n0 + tx * 4 + j;
      C[(int64_t)row * N + col] = gelu_erf(acc[i][j] + bias[col]);
    }
  }
}

// ---------------------------------------------------------------------------
// Pooling, general form (any d the call accepts): one workgroup per span.
// Thread t owns the 16-byte column groups t, t + 256, ... of every row.

constexpr int kPoolThreads = 256;
constexpr int kMaxSpanLen = 256;
constexpr int kMaxHeads = 16;
constexpr int kMaxD = 8192;

template <typename T>
struct Vec {
  static constexpr int N = 16 / sizeof(T);
};

template <typename T>
__device__ __forceinline__ void load_vec(const T *p, float *x) {
  const u32x4_t u = *(const u32x4_t *)p;
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = __uint_as_float(u[e] << 16);
      x[2 * e + 1] = __uint_as_float(u[e] & 0xffff0000u);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = __uint_as_float(u[e]);
  }
}

template <typename T>
__device__ __forceinline__ void unpack_vec(u32x4_t u, float *x) {
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = __uint_as_float(u[e] << 16);
      x[2 * e + 1] = __uint_as_float(u[e] & 0xffff0000u);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = __uint_as_float(u[e]);
  }
}

template <typename T>
__device__ __forceinline__ void store_vec(T *p, const float *x) {
  u32x4_t u;
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int e = 0; e < 4; ++e) u[e] = pack_bf16x2(x[2 * e], x[2 * e + 1]);
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) u[e] = __float_as_uint(x[e]);
  }
  *(u32x4_t *)p = u;
}

// Row r of the first stage's output: row r of G1, or, with a token table,
// table row gidx[r] (an index outside [0, g_rows) reads row 0 and sets
// EINVAL).
template <typename T>
__device__ __forceinline__ const T *g1_row(const T *G1, const int32_t *gidx, int64_t g_rows, int r, int d,
                                           int32_t *err) {
  int64_t gr = r;
  if (gidx) {
    int v = gidx[r];
    if (v < 0 || v >= g_rows) {
      set_err(err, SM_ERR_EINVAL);
      v = 0;
    }
    gr = v;
  }
  return G1 + gr * d;
}

template <typename T>
__global__ __launch_bounds__(kPoolThreads) void pool_kernel(const T *__restrict__ G1,
                                                            const int32_t *__restrict__ gidx, int64_t g_rows,
                                                            const int32_t *__restrict__ span_offsets,
                                                            int num_spans, int total_rows,
                                                            const T *__restrict__ Q, const T *__restrict__ g_kv,
                                                            const T *__restrict__ beta_kv, float eps, int d,
                                                            int h, T *__restrict__ cout, int32_t *err) {
  constexpr int VN = Vec<T>::N;
  constexpr int kMaxVec = kMaxD / VN / kPoolThreads;
  __shared__ float red[kPoolThreads / 64][kMaxHeads + 2];
  __shared__ float row_mean[kMaxSpanLen], row_inv[kMaxSpanLen];
  __shared__ float alpha[kMaxSpanLen][kMaxHeads];
  const int s = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int nvec = d / VN;
  T *dst = cout + (int64_t)s * d;

  const int r0 = span_offsets[s], r1 = span_offsets[s + 1];
  const int n = r1 - r0;
  bool ok = n >= 1 && n <= kMaxSpanLen && r0 >= 0 && r1 <= total_rows;
  if (s == 0 && r0 != 0) ok = false;
  if (s == num_spans - 1 && r1 != total_rows) ok = false;
  if (!ok) {
    if (tid == 0) set_err(err, SM_ERR_EINVAL);
    const float z[VN] = {};
    for (int v = tid; v < nvec; v += kPoolThreads) store_vec(dst + v * VN, z);
    return;
  }
  const int dh = d / h;
  const float inv_sqrt_dh = 1.0f / sqrtf((float)dh);

  // per-thread copies of gamma, beta, q for the owned columns
  float gv[kMaxVec][VN], bv[kMaxVec][VN], qv[kMaxVec][VN];
#pragma unroll
  for (int u = 0; u < kMaxVec; ++u) {
    const int v = tid + u * kPoolThreads;
    if (v < nvec) {
      load_vec(g_kv + v * VN, gv[u]);
      load_vec(beta_kv + v * VN, bv[u]);
      load_vec(Q + v * VN, qv[u]);  // Q is [h][d_h] = flat [d]
    }
  }

  // pass 1: LN statistics and head scores of every row
  for (int j = 0; j < n; ++j) {
    const T *row = g1_row(G1, gidx, g_rows, r0 + j, d, err);
    float x[kMaxVec][VN];
    float sum = 0.f;
#pragma unroll
    for (int u = 0; u < kMaxVec; ++u) {
      const int v = tid + u * kPoolThreads;
      if (v < nvec) {
        load_vec(row + v * VN, x[u]);
#pragma unroll
        for (int e = 0; e < VN; ++e) sum += x[u][e];
      }
    }
    const float mean = block_sum(sum, &red[0][0]) / d;
    float sq = 0.f;
#pragma unroll
    for (int u = 0; u < kMaxVec; ++u) {
      const int v = tid + u * kPoolThreads;
      if (v < nvec)
#pragma unroll
        for (int e = 0; e < VN; ++e) sq += (x[u][e] - mean) * (x[u][e] - mean);
    }
    const float var = block_sum(sq, &red[0][0]) / d;
    const float inv = 1.0f / sqrtf(var + eps);
    float hs[kMaxHeads];
#pragma unroll
    for (int i = 0; i < kMaxHeads; ++i) hs[i] = 0.f;
#pragma unroll
    for (int u = 0; u < kMaxVec; ++u) {
      const int v = tid + u * kPoolThreads;
      if (v < nvec) {
        const int head = (v * VN) / dh;  // a 16-byte group never straddles heads
        float part = 0.f;
#pragma unroll
        for (int e = 0; e < VN; ++e) part += (gv[u][e] * (x[u][e] - mean) * inv + bv[u][e]) * qv[u][e];
#pragma unroll
        for (int i = 0; i < kMaxHeads; ++i)
          if (i == head) hs[i] += part;
      }
    }
    __syncthreads();
    for (int i = 0; i < h; ++i) {
      const float t = wave_sum(hs[i]);
      if (lane == 0) red[w][i] = t;
    }
    __syncthreads();
    if (tid < h) {
      float t = 0.f;
      for (int ww = 0; ww < kPoolThreads / 64; ++ww) t += red[ww][tid];
      alpha[j][tid] = t * inv_sqrt_dh;  // raw score for now
    }
    if (tid == 0) {
      row_mean[j] = mean;
      row_inv[j] = inv;
    }
  }
  __syncthreads();
  // softmax over the span, per head
  if (tid < h) {
    float m = -INFINITY;
    for (int j = 0; j < n; ++j) m = fmaxf(m, alpha[j][tid]);
    float z = 0.f;
    for (int j = 0; j < n; ++j) {
      const float e = expf(alpha[j][tid] - m);
      alpha[j][tid] = e;
      z += e;
    }
    const float iz = 1.0f / z;
    for (int j = 0; j < n; ++j) alpha[j][tid] *= iz;
  }
  __syncthreads();

  // pass 2: c = sum_j alpha_j P_j  (rows re-read, L2-resident)
  float cacc[kMaxVec][VN];
#pragma unroll
  for (int u = 0; u < kMaxVec; ++u)
#pragma unroll
    for (int e = 0; e < VN; ++e) cacc[u][e] = 0.f;
  for (int j = 0; j < n; ++j) {
    const T *row = g1_row(G1, gidx, g_rows, r0 + j, d, err);
    const float mean = row_mean[j], inv = row_inv[j];
#pragma unroll
    for (int u = 0; u < kMaxVec; ++u) {
      const int v = tid + u * kPoolThreads;
      if (v < nvec) {
        float x[VN];
        load_vec(row + v * VN, x);
        const float a = alpha[j][(v * VN) / dh];
#pragma unroll
        for (int e = 0; e < VN; ++e) cacc[u][e] += a * (gv[u][e] * (x[e] - mean) * inv + bv[u][e]);
      }
    }
  }
#pragma unroll
  for (int u = 0; u < kMaxVec; ++u) {
    const int v = tid + u * kPoolThreads;
    if (v < nvec) store_vec(dst + v * VN, cacc[u]);
  }
}

// Pooling, register form for d = NCH * 64 * (16 / sizeof(T)): one workgroup of
// four waves per span.  Wave w takes rows w, w + 4, ... of the span whole into
// its registers (lane l holds the 16-byte groups l, l + 64, ... of the row), so
// a row's LN statistics and its h head scores cost one load round trip and
// wave reductions only.  The LN_kv gain, bias and the queries are staged once
// in LDS.  The weighted sum then splits the columns over the workgroup and
// re-reads the span's rows (cache hits), four rows per round trip.
constexpr int kPoolWaves = 4;

template <typename T, int NCH>
__global__ __launch_bounds__(kPoolWaves * 64) void pool_rows_kernel(const T *__restrict__ G1,
                                                                    const int32_t *__restrict__ gidx,
                                                                    int64_t g_rows,
                                                                    const int32_t *__restrict__ span_offsets,
                                                                    int num_spans, int total_rows,
                                                                    const T *__restrict__ Q,
                                                                    const T *__restrict__ g_kv,
                                                                    const T *__restrict__ beta_kv, float eps, int d,
                                                                    int h, T *__restrict__ cout, int32_t *err) {
  constexpr int VN = Vec<T>::N;
  constexpr int NT = kPoolWaves * 64, NV = NCH * 64;
  __shared__ float alpha[kMaxSpanLen][kMaxHeads];
  __shared__ float row_mean[kMaxSpanLen], row_inv[kMaxSpanLen];
  __shared__ u32x4_t par[3][NV];  // g_kv, beta_kv, Q as stored
  const int s = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  T *dst = cout + (int64_t)s * d;

  const int r0 = span_offsets[s], r1 = span_offsets[s + 1];
  const int n = r1 - r0;
  bool ok = n >= 1 && n <= kMaxSpanLen && r0 >= 0 && r1 <= total_rows;
  if (s == 0 && r0 != 0) ok = false;
  if (s == num_spans - 1 && r1 != total_rows) ok = false;
  if (!ok) {
    if (tid == 0) set_err(err, SM_ERR_EINVAL);
    for (int v = tid; v < NV; v += NT) ((u32x4_t *)dst)[v] = u32x4_t{0u, 0u, 0u, 0u};
    return;
  }
  const int dh = d / h;
  const float inv_sqrt_dh = 1.0f / sqrtf((float)dh);

  // this wave's first row is requested before the parameters are staged
  u32x4_t xr[NCH];
  if (w < n) {
    const u32x4_t *row = (const u32x4_t *)g1_row(G1, gidx, g_rows, r0 + w, d, err);
#pragma unroll
    for (int u = 0; u < NCH; ++u) xr[u] = row[u * 64 + lane];
  }
  for (int v = tid; v < NV; v += NT) {
    par[0][v] = ((const u32x4_t *)g_kv)[v];
    par[1][v] = ((const u32x4_t *)beta_kv)[v];
    par[2][v] = ((const u32x4_t *)Q)[v];
  }
  int hd[NCH];  // head of this lane's group in chunk u (a group never straddles heads)
#pragma unroll
  for (int u = 0; u < NCH; ++u) hd[u] = ((u * 64 + lane) * VN) / dh;
  __syncthreads();

  for (int j = w; j < n; j += kPoolWaves) {
    // keeps the parameter reads below inside the loop: hoisted, they would
    // hold 3 * NCH * VN floats live across it
    asm volatile("" ::: "memory");
    if (j != w) {
      const u32x4_t *row = (const u32x4_t *)g1_row(G1, gidx, g_rows, r0 + j, d, err);
#pragma unroll
      for (int u = 0; u < NCH; ++u) xr[u] = row[u * 64 + lane];
    }
    float x[NCH][VN];
    float sum = 0.f;
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      unpack_vec<T>(xr[u], x[u]);
#pragma unroll
      for (int e = 0; e < VN; ++e) sum += x[u][e];
    }
    const float mean = wave_sum(sum) / d;
    float sq = 0.f;
#pragma unroll
    for (int u = 0; u < NCH; ++u)
#pragma unroll
      for (int e = 0; e < VN; ++e) sq += (x[u][e] - mean) * (x[u][e] - mean);
    const float inv = 1.0f / sqrtf(wave_sum(sq) / d + eps);
    float part[NCH];
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      float gv[VN], bv[VN], qv[VN];
      unpack_vec<T>(par[0][u * 64 + lane], gv);
      unpack_vec<T>(par[1][u * 64 + lane], bv);
      unpack_vec<T>(par[2][u * 64 + lane], qv);
      float p = 0.f;
#pragma unroll
      for (int e = 0; e < VN; ++e) p += (gv[e] * (x[u][e] - mean) * inv + bv[e]) * qv[e];
      part[u] = p;
    }
#pragma unroll 1
    for (int i = 0; i < h; ++i) {
      float t = 0.f;
#pragma unroll
      for (int u = 0; u < NCH; ++u) t += hd[u] == i ? part[u] : 0.f;
      t = wave_sum(t);
      if (lane == 0) alpha[j][i] = t * inv_sqrt_dh;  // raw score for now
    }
    if (lane == 0) {
      row_mean[j] = mean;
      row_inv[j] = inv;
    }
  }
  __syncthreads();
  // softmax over the span, per head
  if (tid < h) {
    float m = -INFINITY;
    for (int j = 0; j < n; ++j) m = fmaxf(m, alpha[j][tid]);
    float z = 0.f;
    for (int j = 0; j < n; ++j) {
      const float e = expf(alpha[j][tid] - m);
      alpha[j][tid] = e;
      z += e;
    }
    const float iz = 1.0f / z;
    for (int j = 0; j < n; ++j) alpha[j][tid] *= iz;
  }
  __syncthreads();

  // c = sum_j alpha_j P_j over this thread's column groups
  for (int v = tid; v < NV; v += NT) {
    const int col = v * VN, head = col / dh;
    float gv[VN], bv[VN], acc[VN];
    unpack_vec<T>(par[0][v], gv);
    unpack_vec<T>(par[1][v], bv);
#pragma unroll
    for (int e = 0; e < VN; ++e) acc[e] = 0.f;
    for (int j0 = 0; j0 < n; j0 += 4) {
      u32x4_t xq[4];
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        if (j0 + jj < n) xq[jj] = *(const u32x4_t *)(g1_row(G1, gidx, g_rows, r0 + j0 + jj, d, err) + col);
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        if (j0 + jj < n) {
          float x[VN];
          unpack_vec<T>(xq[jj], x);
          const float a = alpha[j0 + jj][head], mean = row_mean[j0 + jj], inv = row_inv[j0 + jj];
#pragma unroll
          for (int e = 0; e < VN; ++e) acc[e] += a * (gv[e] * (x[e] - mean) * inv + bv[e]);
        }
    }
    store_vec(dst + col, acc);
  }
}

// Pooling, column-slice form for d = 4 * 64 * CPL * (16 / sizeof(T)):
// persistent workgroups of four waves, each taking spans blockIdx.x,
// blockIdx.x + gridDim.x, ...  Wave w owns columns [w d/4, (w + 1) d/4);
// lane l holds the 16-byte groups c * 64 + l (c < CPL) of that slice of
// every row.  The slice's score weights q_j g_j, LN_kv gain and bias are
// staged once per workgroup in LDS (each lane reads back only its own), and
// the span's rows are read once: kPoolResident at a time into registers,
// each group scored and folded into the weighted sum by an online softmax
// before the next is loaded.  Only a few sums per row cross waves, through
// LDS.
//
// With the shift K_rw = the slice's first element of row r, wave w forms
//   S1 = sum (x - K),  S2 = sum (x - K)^2,  T_h = sum_{j in head h} q_j g_j (x_j - K)
// over its slice.  The slices' (S1, S2) combine by the pairwise update of
// Chan, Golub and LeVeque into the row's mean mu_r and
// inv_r = 1 / sqrt(var_r + eps), and the score of head h is
//   s_rh = (inv_r sum_w [T_wh + (K_rw - mu_r) C_wh] + D_h) / sqrt(dh),
//   C_wh = sum_{j in h, slice w} q_j g_j,  D_h = sum_{j in h} q_j beta_j,
// i.e. q_h . LN_kv(x_r)_h / sqrt(dh).  With p_rh = exp(s_rh - M_h) (M_h the
// running maximum; earlier terms are rescaled when it moves), Z_h their
// sum and a_rh = p_rh inv_r, the pooled column j is
//   g_j (sum_r a_rh (x_rj - K_rw) - E_wh) / Z_h + beta_j,
//   E_wh = sum_r a_rh (mu_r - K_rw),
// which is sum_r alpha_rh LN_kv(x_r)_j for alpha = softmax_r(s_rh), since
// each head's alphas sum to one.  The shifts keep the sums free of
// cancellation when a row's values sit far from zero.
constexpr int kPoolResident = 4;  // rows per group held in registers
constexpr int kSliceHeads = 5;    // heads meeting one quarter of the columns (h <= 16, d/h a multiple of 64)

template <typename T, int CPL>
__global__ __launch_bounds__(256, CPL <= 2 ? 3 : 2) void pool_slices_kernel(const T *__restrict__ G1, const int32_t *__restrict__ gidx,
                                                          int64_t g_rows, const int32_t *__restrict__ span_offsets,
                                                          int num_spans, int total_rows, const T *__restrict__ Q,
                                                          const T *__restrict__ g_kv, const T *__restrict__ beta_kv,
                                                          float eps, int d, int h, T *__restrict__ cout,
                                                          int32_t *err) {
  constexpr int VN = Vec<T>::N, R = kPoolResident;
  __shared__ float sh_k[R][4], sh_s1[R][4], sh_s2[R][4];  // per row of the group and slice
  __shared__ float sh_t[R][4][kSliceHeads];
  __shared__ float sh_a[R][kMaxHeads], sh_mu[R];
  __shared__ float sh_scale[kMaxHeads], sh_iz[kMaxHeads];
  __shared__ float sh_c[4][kSliceHeads], sh_dq[4][kSliceHeads];
  __shared__ u32x4_t sh_gb[2][4 * 64 * CPL];        // g_kv, beta_kv as stored
  __shared__ f32x4_t sh_wq[4 * 64 * CPL][VN / 4];   // q_j g_j
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int slice = d >> 2, dh = d / h;
  const int hf = (w * slice) / dh, nh = (w * slice + slice - 1) / dh - hf + 1;  // heads meeting this slice
  const int c0 = w * slice + lane * VN;                                             // column of group 0
  int hd[CPL];  // head of group c, counted from hf
#pragma unroll
  for (int c = 0; c < CPL; ++c) hd[c] = (c0 + c * 64 * VN) / dh - hf;

  {
    float cs[kSliceHeads], ds[kSliceHeads];
#pragma unroll
    for (int hs = 0; hs < kSliceHeads; ++hs) cs[hs] = ds[hs] = 0.f;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const int col = c0 + c * 64 * VN;
      const u32x4_t gu = *(const u32x4_t *)(g_kv + col), bu = *(const u32x4_t *)(beta_kv + col);
      sh_gb[0][(w * CPL + c) * 64 + lane] = gu;
      sh_gb[1][(w * CPL + c) * 64 + lane] = bu;
      float qf[VN], gf[VN], bf[VN], wq[VN];
      unpack_vec<T>(*(const u32x4_t *)(Q + col), qf);
      unpack_vec<T>(gu, gf);
      unpack_vec<T>(bu, bf);
      float cc = 0.f, dd = 0.f;
#pragma unroll
      for (int e = 0; e < VN; ++e) {
        wq[e] = qf[e] * gf[e];
        cc += wq[e];
        dd += qf[e] * bf[e];
      }
#pragma unroll
      for (int v = 0; v < VN / 4; ++v)
        sh_wq[(w * CPL + c) * 64 + lane][v] = f32x4_t{wq[4 * v], wq[4 * v + 1], wq[4 * v + 2], wq[4 * v + 3]};
#pragma unroll
      for (int hs = 0; hs < kSliceHeads; ++hs)
        if (hd[c] == hs) {
          cs[hs] += cc;
          ds[hs] += dd;
        }
    }
#pragma unroll
    for (int hs = 0; hs < kSliceHeads; ++hs)
      if (hs < nh) {  // wave-uniform
        const float cw = wave_sum(cs[hs]), dw = wave_sum(ds[hs]);
        if (lane == 0) {
          sh_c[w][hs] = cw;
          sh_dq[w][hs] = dw;
        }
      }
  }
  // scores in base 2 (log2 e folded into 1 / sqrt(dh)): exp2 is one instruction; the
  // softmax is the same.  Divisions by the slice width and d become products.
  const float l2_sqrt_dh = 1.4426950408889634f / sqrtf((float)dh), n_slice = (float)slice;
  const float inv_ns = 1.0f / n_slice, inv_d = 1.0f / (float)d;
  // thread hh < h: the slices head hh meets, its index within each, and
  // its constants C_wh (per slice) and D_h (all slices)
  float hc[4] = {0.f, 0.f, 0.f, 0.f}, hdq = 0.f;
  int hsl[4] = {0, 0, 0, 0}, hwf = 0, hwl = -1;
  __syncthreads();  // sh_c, sh_dq
  if (tid < h) {
    hwf = (tid * dh) / slice;
    hwl = (tid * dh + dh - 1) / slice;
#pragma unroll
    for (int ww = 0; ww < 4; ++ww)
      if (ww >= hwf && ww <= hwl) {
        hsl[ww] = tid - (ww * slice) / dh;
        hc[ww] = sh_c[ww][hsl[ww]];
        hdq += sh_dq[ww][hsl[ww]];
      }
  }

  // the next span's row range is requested a span ahead
  int nx0 = 0, nx1 = 0;
  if ((int)blockIdx.x < num_spans) {
    nx0 = span_offsets[blockIdx.x];
    nx1 = span_offsets[blockIdx.x + 1];
  }
  for (int s = blockIdx.x; s < num_spans; s += gridDim.x) {
    T *dst = cout + (int64_t)s * d;
    const int r0 = nx0, r1 = nx1;
    if (s + (int)gridDim.x < num_spans) {
      nx0 = span_offsets[s + gridDim.x];
      nx1 = span_offsets[s + gridDim.x + 1];
    }
    const int n = r1 - r0;
    bool ok = n >= 1 && n <= kMaxSpanLen && r0 >= 0 && r1 <= total_rows;
    if (s == 0 && r0 != 0) ok = false;
    if (s == num_spans - 1 && r1 != total_rows) ok = false;
    if (!ok) {  // (uniform over the workgroup)
      if (tid == 0) set_err(err, SM_ERR_EINVAL);
#pragma unroll
      for (int c = 0; c < CPL; ++c) *(u32x4_t *)(dst + c0 + c * 64 * VN) = u32x4_t{0u, 0u, 0u, 0u};
      continue;
    }
    float M = -INFINITY, Z = 0.f;  // (thread hh < h: head hh's running maximum and sum)
    float E = 0.f;                 // (lane hs < nh: E of head hf + hs)
    float acc[CPL][VN];
#pragma unroll
    for (int c = 0; c < CPL; ++c)
#pragma unroll
      for (int e = 0; e < VN; ++e) acc[c][e] = 0.f;
    for (int g0 = 0; g0 < n; g0 += R) {
      const int nr = min(R, n - g0);
      u32x4_t xr[R][CPL];
#pragma unroll
      for (int rr = 0; rr < R; ++rr)
        if (rr < nr) {
          const T *row = g1_row(G1, gidx, g_rows, r0 + g0 + rr, d, err) + c0;
#pragma unroll
          for (int c = 0; c < CPL; ++c) xr[rr][c] = *(const u32x4_t *)(row + c * 64 * VN);
        }
      // slice sums of the group's rows
#pragma unroll
      for (int rr = 0; rr < R; ++rr)
        if (rr < nr) {
          float xk[VN];
          unpack_vec<T>(xr[rr][0], xk);
          const float K = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(xk[0])));
          float s1 = 0.f, s2 = 0.f, tc[CPL];
#pragma unroll
          for (int c = 0; c < CPL; ++c) {
            float x[VN], wq[VN];
            unpack_vec<T>(xr[rr][c], x);
#pragma unroll
            for (int v = 0; v < VN / 4; ++v) {
              const f32x4_t q4 = sh_wq[(w * CPL + c) * 64 + lane][v];
#pragma unroll
              for (int e = 0; e < 4; ++e) wq[4 * v + e] = q4[e];
            }
            float t = 0.f;
#pragma unroll
            for (int e = 0; e < VN; ++e) {
              const float dx = x[e] - K;
              s1 += dx;
              s2 = fmaf(dx, dx, s2);
              t = fmaf(wq[e], dx, t);
            }
            tc[c] = t;
          }
          s1 = wave_sum(s1);
          s2 = wave_sum(s2);
#pragma unroll
          for (int hs = 0; hs < kSliceHeads; ++hs)
            if (hs < nh) {
              float t = 0.f;
#pragma unroll
              for (int c = 0; c < CPL; ++c) t += hd[c] == hs ? tc[c] : 0.f;
              t = wave_sum(t);
              if (lane == 0) sh_t[rr][w][hs] = t;
            }
          if (lane == 0) {
            sh_k[rr][w] = K;
            sh_s1[rr][w] = s1;
            sh_s2[rr][w] = s2;
          }
          __builtin_amdgcn_sched_barrier(0);  // one row at a time: bounds the live unpacked values
        }
      lds_barrier();
      // the group's row statistics and scores, folded into the running
      // softmax: thread hh < h takes head hh
      if (tid < h) {
        const int hh = tid;
        float sc[R], iv[R], gmax = -INFINITY;
#pragma unroll
        for (int rr = 0; rr < R; ++rr)
          if (rr < nr) {
            float mw[4], mean = 0.f, m2 = 0.f;
#pragma unroll
            for (int ww = 0; ww < 4; ++ww) {
              const float a1 = sh_s1[rr][ww];
              mw[ww] = sh_k[rr][ww] + a1 * inv_ns;
              mean += mw[ww];
              m2 += sh_s2[rr][ww] - a1 * (a1 * inv_ns);
            }
            mean *= 0.25f;
#pragma unroll
            for (int ww = 0; ww < 4; ++ww) m2 += n_slice * (mw[ww] - mean) * (mw[ww] - mean);
            iv[rr] = __builtin_amdgcn_rsqf(fmaxf(m2, 0.f) * inv_d + eps);
            float t = 0.f;
#pragma unroll
            for (int ww = 0; ww < 4; ++ww)
              if (ww >= hwf && ww <= hwl) t += sh_t[rr][ww][hsl[ww]] + (sh_k[rr][ww] - mean) * hc[ww];
            sc[rr] = (iv[rr] * t + hdq) * l2_sqrt_dh;
            gmax = fmaxf(gmax, sc[rr]);
            if (hh == 0) sh_mu[rr] = mean;
          }
        const float Mn = fmaxf(M, gmax), scale = __builtin_amdgcn_exp2f(M - Mn);  // 0 for the first group
        Z *= scale;
#pragma unroll
        for (int rr = 0; rr < R; ++rr)
          if (rr < nr) {
            const float p = __builtin_amdgcn_exp2f(sc[rr] - Mn);
            Z += p;
            sh_a[rr][hh] = p * iv[rr];
          }
        M = Mn;
        sh_scale[hh] = scale;
        if (g0 + R >= n) sh_iz[hh] = __builtin_amdgcn_rcpf(Z);
      }
      lds_barrier();
      // fold the group into this wave's weighted sum (the rows are unpacked
      // again: an empty asm on the packed registers keeps the compiler from
      // holding the unpacked floats of the score pass across the barriers)
#pragma unroll
      for (int rr = 0; rr < R; ++rr)
#pragma unroll
        for (int c = 0; c < CPL; ++c) asm volatile("" : "+v"(xr[rr][c]));
      if (lane < nh) {
        E *= sh_scale[hf + lane];
        for (int rr = 0; rr < nr; ++rr) E += sh_a[rr][hf + lane] * (sh_mu[rr] - sh_k[rr][w]);
      }
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const float sc = sh_scale[hf + hd[c]];
#pragma unroll
        for (int e = 0; e < VN; ++e) acc[c][e] *= sc;
      }
#pragma unroll
      for (int rr = 0; rr < R; ++rr)
        if (rr < nr) {
          const float K = sh_k[rr][w];
#pragma unroll
          for (int c = 0; c < CPL; ++c) {
            const float a = sh_a[rr][hf + hd[c]];
            float x[VN];
            unpack_vec<T>(xr[rr][c], x);
#pragma unroll
            for (int e = 0; e < VN; ++e) acc[c][e] = fmaf(a, x[e] - K, acc[c][e]);
          }
        }
      // (the next group's sums are written only after every wave has passed
      // this group's second barrier, and read after its own first)
    }
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const float ec = __shfl(E, hd[c]), iz = sh_iz[hf + hd[c]];
      float gf[VN], bf[VN], y[VN];
      unpack_vec<T>(sh_gb[0][(w * CPL + c) * 64 + lane], gf);
      unpack_vec<T>(sh_gb[1][(w * CPL + c) * 64 + lane], bf);
#pragma unroll
      for (int e = 0; e < VN; ++e) y[e] = fmaf(gf[e], (acc[c][e] - ec) * iz, bf[e]);
      store_vec(dst + c0 + c * 64 * VN, y);
    }
  }
}

// Resident workgroups of a pooling kernel over the whole device (looked up
// once per kernel), for the persistent grid.
template <typename K>
static int resident_blocks(K kernel, int threads) {
  static const int nb = [&] {
    int dev = 0, cus = 0, occ = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
      cus = 256;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kernel, threads, 0) != hipSuccess || occ <= 0) occ = 1;
    return cus * occ;
  }();
  return nb;
}

template <typename T>
static hipError_t launch_pool(const T *G1, const int32_t *gidx, int64_t g_rows, const int32_t *span_offsets,
                              int num_spans, int total_rows, const T *Q, const T *g_kv, const T *beta_kv, float eps,
                              int d, int h, T *cout, int32_t *err, hipStream_t stream) {
  constexpr int VN = Vec<T>::N;
  const int cpl = d % (256 * VN) == 0 ? d / (256 * VN) : 0;
#define SM_SLICE_CASE(C)                                                                                         \
  case C: {                                                                                                      \
    const int nb = resident_blocks(pool_slices_kernel<T, C>, 256);                                               \
    hipLaunchKernelGGL((pool_slices_kernel<T, C>), dim3(num_spans < nb ? num_spans : nb), dim3(256), 0, stream,  \
                       G1, gidx, g_rows, span_offsets, num_spans, total_rows, Q, g_kv, beta_kv, eps, d, h, cout,  \
                       err);                                                                                     \
    return hipGetLastError();                                                                                    \
  }
  if (num_spans > 0) switch (cpl) {
      SM_SLICE_CASE(1) SM_SLICE_CASE(2) SM_SLICE_CASE(3) SM_SLICE_CASE(4)
      default:
        break;
    }
#undef SM_SLICE_CASE
  const int nch = d % (64 * VN) == 0 ? d / (64 * VN) : 0;
#define SM_POOL_CASE(C)                                                                                          \
  case C:                                                                                                        \
    hipLaunchKernelGGL((pool_rows_kernel<T, C>), dim3(num_spans), dim3(kPoolWaves * 64), 0, stream, G1, gidx,    \
                       g_rows, span_offsets, num_spans, total_rows, Q, g_kv, beta_kv, eps, d, h, cout, err);     \
    break;
  switch (nch) {
    SM_POOL_CASE(1) SM_POOL_CASE(2) SM_POOL_CASE(3) SM_POOL_CASE(4)
    SM_POOL_CASE(5) SM_POOL_CASE(6) SM_POOL_CASE(7) SM_POOL_CASE(8)
    SM_POOL_CASE(16)
    default:
      hipLaunchKernelGGL(pool_kernel<T>, dim3(num_spans), dim3(kPoolThreads), 0, stream, G1, gidx, g_rows,
                         span_offsets, num_spans, total_rows, Q, g_kv, beta_kv, eps, d, h, cout, err);
  }
#undef SM_POOL_CASE
  return hipGetLastError();
}

// LN_o over fp32 rows Y -> out (storage dtype), one workgroup per row; the
// row, the gain and the bias are all requested before the first reduction.
template <typename T, typename YT = float>
__global__ __launch_bounds__(kPoolThreads) void ln_rows_kernel(const YT *__restrict__ Y,
                                                               const T *__restrict__ g, const T *__restrict__ b,
                                                               float eps, int d, T *__restrict__ out) {
  constexpr int kMaxV = kMaxD / 4 / kPoolThreads;
  __shared__ float red[kPoolThreads / 64];
  const int s = blockIdx.x, tid = threadIdx.x;
  const int nvec = d / 4;
  const YT *row = Y + (int64_t)s * d;
  float x[kMaxV][4], gv[kMaxV][4], bv[kMaxV][4];
#pragma unroll
  for (int u = 0; u < kMaxV; ++u) {
    const int v = tid + u * kPoolThreads;
    if (v < nvec) {
      if constexpr (sizeof(YT) == 2) {
        const uint2 yy = *(const uint2 *)(row + v * 4);
        x[u][0] = __uint_as_float(yy.x << 16);
        x[u][1] = __uint_as_float(yy.x & 0xffff0000u);
        x[u][2] = __uint_as_float(yy.y << 16);
        x[u][3] = __uint_as_float(yy.y & 0xffff0000u);
      } else {
        load_vec<float>((const float *)row + v * 4, x[u]);
      }
      if constexpr (sizeof(T) == 2) {
        const uint2 gg = *(const uint2 *)(g + v * 4), bb = *(const uint2 *)(b + v * 4);
        gv[u][0] = __uint_as_float(gg.x << 16);
        gv[u][1] = __uint_as_float(gg.x & 0xffff0000u);
        gv[u][2] = __uint_as_float(gg.y << 16);
        gv[u][3] = __uint_as_float(gg.y & 0xffff0000u);
        bv[u][0] = __uint_as_float(bb.x << 16);
        bv[u][1] = __uint_as_float(bb.x & 0xffff0000u);
        bv[u][2] = __uint_as_float(bb.y << 16);
        bv[u][3] = __uint_as_float(bb.y & 0xffff0000u);
      } else {
        load_vec<float>((const float *)g + v * 4, gv[u]);
        load_vec<float>((const float *)b + v * 4, bv[u]);
      }
    }
  }
  float sum = 0.f;
#pragma unroll
  for (int u = 0; u < kMaxV; ++u)
    if (tid + u * kPoolThreads < nvec)
#pragma unroll
      for (int e = 0; e < 4; ++e) sum += x[u][e];
  const float mean = block_sum(sum, red) / d;
  float sq = 0.f;
#pragma unroll
  for (int u = 0; u < kMaxV; ++u)
    if (tid + u * kPoolThreads < nvec)
#pragma unroll
      for (int e = 0; e < 4; ++e) sq += (x[u][e] - mean) * (x[u][e] - mean);
  const float inv = 1.0f / sqrtf(block_sum(sq, red) / d + eps);
#pragma unroll
  for (int u = 0; u < kMaxV; ++u) {
    const int v = tid + u * kPoolThreads;
    if (v < nvec) {
      float y[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) y[e] = gv[u][e] * (x[u][e] - mean) * inv + bv[u][e];
      if constexpr (sizeof(T) == 2)
        *(uint2 *)(out + (int64_t)s * d + v * 4) = make_uint2(pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3]));
      else
        *(f32x4_t *)(out + (int64_t)s * d + v * 4) = f32x4_t{y[0], y[1], y[2], y[3]};
    }
  }
}

// LN_o over bf16 rows of d = NV * 2048 (256 threads x NV 16-byte groups),
// for large batches: persistent workgroups take rows blockIdx.x,
// blockIdx.x + gridDim.x, ...; each loads the gain and bias once (one
// workgroup per row re-read them from L2 for every row, as many bytes as
// the row itself) and issues the next row's loads before this row's two
// reductions.  The arithmetic is that of ln_rows_kernel: mean, then the
// mean of squared deviations, in fp32; bf16 out, rounded to nearest even.
template <int NV>
__global__ __launch_bounds__(kPoolThreads) void ln_rows_bf16_kernel(const uint16_t *__restrict__ Y,
                                                                    const uint16_t *__restrict__ g,
                                                                    const uint16_t *__restrict__ b, float eps,
                                                                    int d, int rows, uint16_t *__restrict__ out) {
  __shared__ float red[kPoolThreads / 64];
  const int tid = threadIdx.x;
  u32x4_t gq[NV], bq[NV], xq[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int col = (tid + v * kPoolThreads) * 8;
    gq[v] = *(const u32x4_t *)(g + col);
    bq[v] = *(const u32x4_t *)(b + col);
    xq[v] = *(const u32x4_t *)(Y + (int64_t)blockIdx.x * d + col);
  }
  for (int s = blockIdx.x; s < rows; s += gridDim.x) {
    const int sn = min(s + (int)gridDim.x, rows - 1);  // (the last row's loads are repeated, never used)
    u32x4_t nq[NV];
#pragma unroll
    for (int v = 0; v < NV; ++v) nq[v] = *(const u32x4_t *)(Y + (int64_t)sn * d + (tid + v * kPoolThreads) * 8);
    float x[NV][8];
    float sum = 0.f;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      unpack_vec<uint16_t>(xq[v], x[v]);
#pragma unroll
      for (int e = 0; e < 8; ++e) sum += x[v][e];
    }
    const float mean = block_sum(sum, red) / d;
    float sq = 0.f;
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < 8; ++e) sq += (x[v][e] - mean) * (x[v][e] - mean);
    const float inv = 1.0f / sqrtf(block_sum(sq, red) / d + eps);
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      float gf[8], bf[8], y[8];
      unpack_vec<uint16_t>(gq[v], gf);
      unpack_vec<uint16_t>(bq[v], bf);
#pragma unroll
      for (int e = 0; e < 8; ++e) y[e] = gf[e] * (x[v][e] - mean) * inv + bf[e];
      store_vec<uint16_t>(out + (int64_t)s * d + (tid + v * kPoolThreads) * 8, y);
      xq[v] = nq[v];
    }
  }
}

// LN_o of bf16 rows: the persistent form where d allows it (rows > 0)
static hipError_t launch_ln_bf16(const uint16_t *Y, const uint16_t *g, const uint16_t *b, float eps, int d,
                                 int rows, uint16_t *out, hipStream_t stream) {
  const int nv = d % (8 * kPoolThreads) == 0 ? d / (8 * kPoolThreads) : 0;
#define SM_LN_CASE(NV)                                                                                   \
  case NV: {                                                                                             \
    const int nb = resident_blocks(ln_rows_bf16_kernel<NV>, kPoolThreads);                               \
    hipLaunchKernelGGL(ln_rows_bf16_kernel<NV>, dim3(rows < nb ? rows : nb), dim3(kPoolThreads), 0, stream, Y, g, \
                       b, eps, d, rows, out);                                                            \
    return hipGetLastError();                                                                            \
  }
  switch (nv) {
    SM_LN_CASE(1) SM_LN_CASE(2) SM_LN_CASE(3) SM_LN_CASE(4)
    default:
      break;
  }
#undef SM_LN_CASE
  hipLaunchKernelGGL((ln_rows_kernel<uint16_t, uint16_t>), dim3(rows), dim3(kPoolThreads), 0, stream, Y, g, b, eps,
                     d, out);
  return hipGetLastError();
}

}  // namespace sm

using namespace sm;

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }


// ---------------------------------------------------------------------------
// Row order of a large first stage.  The gathered rows are token ids in span
// order, scattered over the embedding table, and the 256-tile GEMM reads
// each of a tile's 256 rows once per 64-deep k-tile: rows from all over the
// table cost address translations and DRAM pages at every k-tile, and a
// repeated token is fetched by as many tiles as it has occurrences.  A
// stable counting sort of the rows by token-id bucket (kSortBuckets
// buckets of consecutive ids) puts nearby and repeated ids in the same
// tiles.  The GEMM then writes G1 in sorted order, and the pooling kernel
// reads CSR row r as G1 row inv[r].  Three launches: per-chunk bucket
// counts, their exclusive scan in (bucket, chunk) order, and a per-chunk
// scatter that keeps the rows of one bucket in their CSR order, so the
// permutation is the same on every run.
constexpr int kSortBuckets = 4096, kSortChunk = 4096;

__device__ __forceinline__ int sort_bucket(int32_t t, int64_t vocab) {
  if (t < 0) return 0;
  if (t >= vocab) return kSortBuckets - 1;  // (the GEMM flags the id)
  return (int)((int64_t)t * kSortBuckets / vocab);
}

// grid: one workgroup of 256 per chunk of kSortChunk rows
__global__ __launch_bounds__(256) void sort_count_kernel(const int32_t *__restrict__ tok, int n, int64_t vocab,
                                                         int32_t *__restrict__ hist) {
  __shared__ int h[kSortBuckets];
  for (int i = threadIdx.x; i < kSortBuckets; i += 256) h[i] = 0;
  __syncthreads();
  const int r0 = blockIdx.x * kSortChunk, r1 = min(n, r0 + kSortChunk);
  for (int r = r0 + (int)threadIdx.x; r < r1; r += 256) atomicAdd(&h[sort_bucket(tok[r], vocab)], 1);
  __syncthreads();
  for (int i = threadIdx.x; i < kSortBuckets; i += 256) hist[(int64_t)blockIdx.x * kSortBuckets + i] = h[i];
}

// one workgroup of 1024: hist[c][b] becomes the first sorted position of
// chunk c's rows in bucket b (buckets in order, chunks in order within one)
__global__ __launch_bounds__(1024) void sort_scan_kernel(int32_t *__restrict__ hist, int nchunks) {
  __shared__ int red[16];
  constexpr int BPT = kSortBuckets / 1024;  // buckets per thread
  const int b0 = threadIdx.x * BPT;
  static_assert(BPT == 4, "one 16-byte group of buckets per thread");
  // (the chunks are taken 8 at a time, so that 8 loads are in flight)
  int tot[BPT] = {0, 0, 0, 0}, sum = 0;
  for (int c0 = 0; c0 < nchunks; c0 += 8) {
    int4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      v[u] = c0 + u < nchunks ? *(const int4 *)&hist[(int64_t)(c0 + u) * kSortBuckets + b0] : make_int4(0, 0, 0, 0);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      tot[0] += v[u].x;
      tot[1] += v[u].y;
      tot[2] += v[u].z;
      tot[3] += v[u].w;
    }
  }
#pragma unroll
  for (int k = 0; k < BPT; ++k) sum += tot[k];
  int total;
  const int base = block_inclusive_scan(sum, red, &total) - sum;
  int run[BPT];
  run[0] = base;
#pragma unroll
  for (int k = 1; k < BPT; ++k) run[k] = run[k - 1] + tot[k - 1];
  for (int c0 = 0; c0 < nchunks; c0 += 8) {
    int4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      v[u] = c0 + u < nchunks ? *(const int4 *)&hist[(int64_t)(c0 + u) * kSortBuckets + b0] : make_int4(0, 0, 0, 0);
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (c0 + u < nchunks) {
        *(int4 *)&hist[(int64_t)(c0 + u) * kSortBuckets + b0] = make_int4(run[0], run[1], run[2], run[3]);
        run[0] += v[u].x;
        run[1] += v[u].y;
        run[2] += v[u].z;
        run[3] += v[u].w;
      }
  }
}

// grid: one workgroup of 256 per chunk.  The chunk's ids and cursors are
// staged in LDS by the whole workgroup; then wave 0 takes the ids 64 at a
// time in CSR order: the lanes that share a bucket find each other through
// one ballot per bucket bit, take consecutive positions in lane order, and
// the lowest of them advances the bucket's cursor.
__global__ __launch_bounds__(256) void sort_scatter_kernel(const int32_t *__restrict__ tok, int n, int64_t vocab,
                                                          const int32_t *__restrict__ first,
                                                          int32_t *__restrict__ sorted_tok, int32_t *__restrict__ inv) {
  __shared__ __attribute__((aligned(16))) int cur[kSortBuckets];
  __shared__ __attribute__((aligned(16))) int32_t ids[kSortChunk];
  const int lane = threadIdx.x & 63;
  const int r0 = blockIdx.x * kSortChunk, r1 = min(n, r0 + kSortChunk);
  {
    static_assert(kSortBuckets == 4 * 4 * 256 && kSortChunk == 4 * 4 * 256, "4 x 16 bytes per thread");
    int4 cv[4], iv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = 4 * (threadIdx.x + 256 * u);
      cv[u] = *(const int4 *)&first[(int64_t)blockIdx.x * kSortBuckets + i];
      iv[u] = make_int4(r0 + i < r1 ? tok[r0 + i] : 0, r0 + i + 1 < r1 ? tok[r0 + i + 1] : 0,
                        r0 + i + 2 < r1 ? tok[r0 + i + 2] : 0, r0 + i + 3 < r1 ? tok[r0 + i + 3] : 0);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = 4 * (threadIdx.x + 256 * u);
      *(int4 *)&cur[i] = cv[u];
      *(int4 *)&ids[i] = iv[u];
    }
  }
  __syncthreads();
  if (threadIdx.x >= 64) return;
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));  // lanes below this one
  for (int base = r0; base < r1; base += 64) {
    const int r = base + lane;
    const bool valid = r < r1;
    const int32_t t = valid ? ids[r - r0] : 0;
    const int b = sort_bucket(t, vocab);
    uint64_t same = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 12; ++bit) {  // kSortBuckets = 2^12
      const bool on = (b >> bit) & 1;
      const uint64_t m = __ballot(on);
      same &= on ? m : ~m;
    }
    const int rank = __popcll(same & lt), cnt = __popcll(same);
    const int pos = cur[b] + rank;  // every lane reads before the leaders write (in order within the wave)
    if (valid) {
      sorted_tok[pos] = t;
      inv[r] = pos;
      if (rank == 0) cur[b] = pos + cnt;
    }
  }
}

static size_t sort_ws_bytes(int total_rows) {
  const size_t nchunks = ((size_t)total_rows + kSortChunk - 1) / kSortChunk;
  return 2 * align256((size_t)total_rows * 4) + align256(nchunks * kSortBuckets * 4);
}

SM_API size_t sm_merge_workspace_bytes(int total_rows, int num_spans, int d, sm_dtype dt) {
  if (total_rows < 0 || num_spans < 0 || d <= 0) return 0;
  const size_t es = dt == SM_BF16 ? 2 : 4;
  return align256((size_t)total_rows * d * es) + align256((size_t)num_spans * d * es) +
         align256((size_t)num_spans * d * 4) + sort_ws_bytes(total_rows);
}

// Argument checks shared by the merge entry points.
static sm_status merge_param_check(const sm_merge_params *p, sm_dtype dt) {
  if (!p) return SM_EINVAL;
  if (dt != SM_F32 && dt != SM_BF16) return SM_EINVAL;
  const int d = p->d, h = p->h;
  if (d <= 0 || d > kMaxD || d % 256 != 0 || h <= 0 || h > kMaxHeads || d % h != 0 || (d / h) % 64 != 0)
    return SM_EINVAL;
  if (!p->Q || !p->W_kv || !p->b_kv || !p->g_kv || !p->beta_kv || !p->W_o || !p->b_o || !p->g_o || !p->beta_o)
    return SM_EINVAL;
  return SM_OK;
}

// First stage: C[M][d] = GELU(A[rows][d] W_kv^T + b_kv), the A rows gathered
// through `gather` when given (else rows 0 .. M-1).
static sm_status first_stage(const void *A, const int32_t *gather, int64_t a_rows, int M, const sm_merge_params *p,
                             sm_dtype dt, void *C, int32_t *err, hipStream_t stream) {
  const int d = p->d;
  if (dt == SM_BF16) {
    if (M <= kSkinnyMaxM)
      launch_skinny<uint16_t>((const uint16_t *)A, gather, a_rows, (const uint16_t *)p->W_kv,
                              (const uint16_t *)p->b_kv, (uint16_t *)C, M, d, d, err, stream);
    else if (use_gemm256(M, d, d)) {
      if (launch_gemm256<uint16_t>((const uint16_t *)A, gather, a_rows, (const uint16_t *)p->W_kv,
                                   (const uint16_t *)p->b_kv, (uint16_t *)C, M, d, d, err, stream) != hipSuccess)
        return SM_EHIP;
    } else
      hipLaunchKernelGGL(gemm_bf16_nt_gelu<uint16_t>, dim3(d / kBN, (M + kBM - 1) / kBM), dim3(256), 0, stream,
                         (const uint16_t *)A, gather, a_rows, (const uint16_t *)p->W_kv, (const uint16_t *)p->b_kv,
                         (uint16_t *)C, M, d, d, err);
  } else {
    hipLaunchKernelGGL(gemm_f32_nt_gelu, dim3(d / kFT, (M + kFT - 1) / kFT), dim3(256), 0, stream, (const float *)A,
                       gather, a_rows, (const float *)p->W_kv, (const float *)p->b_kv, (float *)C, M, d, d, err);
  }
  return hipGetLastError() == hipSuccess ? SM_OK : SM_EHIP;
}

// Pooling, second projection and LN_o over the first-stage rows G1 (row r
// of the CSR list is G1 row gidx[r] when gidx is given, else row r).
static sm_status pool_and_project(const void *G1, const int32_t *gidx, int64_t g_rows, int total_rows,
                                  const int32_t *span_offsets, int num_spans, const sm_merge_params *p, sm_dtype dt,
                                  void *cbuf, float *ybuf, void *out, int32_t *err, hipStream_t stream) {
  const int d = p->d, h = p->h;
  if (dt == SM_BF16) {
    if (launch_pool<uint16_t>((const uint16_t *)G1, gidx, g_rows, span_offsets, num_spans, total_rows,
                              (const uint16_t *)p->Q, (const uint16_t *)p->g_kv, (const uint16_t *)p->beta_kv,
                              p->ln_eps, d, h, (uint16_t *)cbuf, err, stream) != hipSuccess)
      return SM_EHIP;
    if (num_spans <= kSkinnyMaxM)
      launch_skinny<float>((const uint16_t *)cbuf, (const int32_t *)nullptr, (int64_t)num_spans,
                           (const uint16_t *)p->W_o, (const uint16_t *)p->b_o, ybuf, num_spans, d, d, err, stream);
    else if (use_gemm256(num_spans, d, d)) {
      if (launch_gemm256<uint16_t>((const uint16_t *)cbuf, (const int32_t *)nullptr, (int64_t)num_spans,
                                   (const uint16_t *)p->W_o, (const uint16_t *)p->b_o, (uint16_t *)ybuf, num_spans, d,
                                   d, err, stream) != hipSuccess)
        return SM_EHIP;
      return launch_ln_bf16((const uint16_t *)ybuf, (const uint16_t *)p->g_o, (const uint16_t *)p->beta_o,
                            p->ln_eps, d, num_spans, (uint16_t *)out, stream) == hipSuccess
                 ? SM_OK
                 : SM_EHIP;
    } else
      hipLaunchKernelGGL(gemm_bf16_nt_gelu<float>, dim3(d / kBN, (num_spans + kBM - 1) / kBM), dim3(256), 0,
                         stream, (const uint16_t *)cbuf, (const int32_t *)nullptr, (int64_t)num_spans,
                         (const uint16_t *)p->W_o, (const uint16_t *)p->b_o, ybuf, num_spans, d, d, err);
    if (hipGetLastError() != hipSuccess) return SM_EHIP;
    hipLaunchKernelGGL(ln_rows_kernel<uint16_t>, dim3(num_spans), dim3(kPoolThreads), 0, stream, ybuf,
                       (const uint16_t *)p->g_o, (const uint16_t *)p->beta_o, p->ln_eps, d, (uint16_t *)out);
  } else {
    if (launch_pool<float>((const float *)G1, gidx, g_rows, span_offsets, num_spans, total_rows,
                           (const float *)p->Q, (const float *)p->g_kv, (const float *)p->beta_kv, p->ln_eps, d, h,
                           (float *)cbuf, err, stream) != hipSuccess)
      return SM_EHIP;
    hipLaunchKernelGGL(gemm_f32_nt_gelu, dim3(d / kFT, (num_spans + kFT - 1) / kFT), dim3(256), 0, stream,
                       (const float *)cbuf, (const int32_t *)nullptr, (int64_t)num_spans, (const float *)p->W_o,
                       (const float *)p->b_o, ybuf, num_spans, d, d, err);
    if (hipGetLastError() != hipSuccess) return SM_EHIP;
    hipLaunchKernelGGL(ln_rows_kernel<float>, dim3(num_spans), dim3(kPoolThreads), 0, stream, ybuf,
                       (const float *)p->g_o, (const float *)p->beta_o, p->ln_eps, d, (float *)out);
  }
  return hipGetLastError() == hipSuccess ? SM_OK : SM_EHIP;
}

SM_API sm_status sm_merge_spans(const void *emb, int64_t emb_rows, const int32_t *row_idx, int total_rows,
                                const int32_t *span_offsets, int num_spans, const sm_merge_params *p,
                                sm_dtype dt, void *out, void *ws, size_t ws_bytes, int32_t *err,
                                hipStream_t stream) {
  if (total_rows < 0 || num_spans < 0) return SM_EINVAL;
  const sm_status pst = merge_param_check(p, dt);
  if (pst != SM_OK) return pst;
  const int d = p->d;
  if (num_spans == 0) return total_rows == 0 ? SM_OK : SM_EINVAL;
  if (total_rows < num_spans) return SM_EINVAL;
  if (!emb || emb_rows <= 0 || !row_idx || !span_offsets || !out || !ws || !err) return SM_EINVAL;
  if (ws_bytes < sm_merge_workspace_bytes(total_rows, num_spans, d, dt)) return SM_EINVAL;
  if ((total_rows + kBM - 1) / kBM > 65535 || (num_spans + kBM - 1) / kBM > 65535) return SM_EINVAL;

  const size_t es = dt == SM_BF16 ? 2 : 4;
  char *wsb = (char *)ws;
  void *g1 = wsb;
  void *cbuf = wsb + align256((size_t)total_rows * d * es);
  float *ybuf = (float *)(wsb + align256((size_t)total_rows * d * es) + align256((size_t)num_spans * d * es));
  if (dt == SM_BF16 && total_rows > kSkinnyMaxM && use_gemm256(total_rows, d, d)) {
    // the first stage in token-id order (see sort_count_kernel)
    char *sw = (char *)ybuf + align256((size_t)num_spans * d * 4);
    int32_t *sorted_tok = (int32_t *)sw;
    int32_t *inv = (int32_t *)(sw + align256((size_t)total_rows * 4));
    int32_t *hist = (int32_t *)(sw + 2 * align256((size_t)total_rows * 4));
    const int nchunks = (total_rows + kSortChunk - 1) / kSortChunk;
    hipLaunchKernelGGL(sort_count_kernel, dim3(nchunks), dim3(256), 0, stream, row_idx, total_rows, emb_rows, hist);
    hipLaunchKernelGGL(sort_scan_kernel, dim3(1), dim3(1024), 0, stream, hist, nchunks);
    hipLaunchKernelGGL(sort_scatter_kernel, dim3(nchunks), dim3(256), 0, stream, row_idx, total_rows, emb_rows,
                       (const int32_t *)hist, sorted_tok, inv);
    if (hipGetLastError() != hipSuccess) return SM_EHIP;
    const sm_status st = first_stage(emb, sorted_tok, emb_rows, total_rows, p, dt, g1, err, stream);
    if (st != SM_OK) return st;
    return pool_and_project(g1, inv, total_rows, total_rows, span_offsets, num_spans, p, dt, cbuf, ybuf, out, err,
                            stream);
  }
  const sm_status st = first_stage(emb, row_idx, emb_rows, total_rows, p, dt, g1, err, stream);
  if (st != SM_OK) return st;
  return pool_and_project(g1, nullptr, total_rows, total_rows, span_offsets, num_spans, p, dt, cbuf, ybuf, out, err,
                          stream);
}

SM_API sm_status sm_merge_token_table(const void *emb, int64_t emb_rows, const sm_merge_params *p, sm_dtype dt,
                                      void *table, int32_t *err, hipStream_t stream) {
  const sm_status pst = merge_param_check(p, dt);
  if (pst != SM_OK) return pst;
  if (emb_rows <= 0 || emb_rows > INT32_MAX || !emb || !table || !err) return SM_EINVAL;
  if ((emb_rows + kBM - 1) / kBM > 65535) return SM_EINVAL;
  return first_stage(emb, nullptr, emb_rows, (int)emb_rows, p, dt, table, err, stream);
}

SM_API sm_status sm_merge_spans_tabled(const void *table, int64_t table_rows, const int32_t *row_idx,
                                       int total_rows, const int32_t *span_offsets, int num_spans,
                                       const sm_merge_params *p, sm_dtype dt, void *out, void *ws, size_t ws_bytes,
                                       int32_t *err, hipStream_t stream) {
  if (total_rows < 0 || num_spans < 0) return SM_EINVAL;
  const sm_status pst = merge_param_check(p, dt);
  if (pst != SM_OK) return pst;
  const int d = p->d;
  if (num_spans == 0) return total_rows == 0 ? SM_OK : SM_EINVAL;
  if (total_rows < num_spans) return SM_EINVAL;
  if (!table || table_rows <= 0 || !row_idx || !span_offsets || !out || !ws || !err) return SM_EINVAL;
  if (ws_bytes < sm_merge_workspace_bytes(0, num_spans, d, dt)) return SM_EINVAL;
  if ((num_spans + kBM - 1) / kBM > 65535) return SM_EINVAL;

  const size_t es = dt == SM_BF16 ? 2 : 4;
  char *wsb = (char *)ws;
  void *cbuf = wsb;
  float *ybuf = (float *)(wsb + align256((size_t)num_spans * d * es));
  return pool_and_project(table, row_idx, table_rows, total_rows, span_offsets, num_spans, p, dt, cbuf, ybuf, out,
                          err, stream);
}

SM_API const char *sm_status_string(sm_status s) {
  switch (s) {
    case SM_OK: return "ok";
    case SM_EINVAL: return "invalid argument";
    case SM_ERANGE: return "length or capacity out of range";
    case SM_ENOMEM: return "not enough free KV blocks";
    case SM_EHIP: return "HIP launch failed";
  }
  return "unknown status";
}
