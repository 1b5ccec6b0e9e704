// Causal GQA flash-attention forward for gfx950 (one head chunk per launch).
//
// Computes, for each query row i of each head of the chunk, the softmax of
// the scaled scores q_i.k_j/sqrt(d) over the visible keys and its weighted
// sum of values (paper Section 2.1), plus the row log-sum-exp (Section 3,
// "the final log-sum-exponent").  Online softmax over key tiles keeps HBM
// traffic at O(S d) per head (flash attention, cited in Section 2.3).
//
// Work decomposition
//   workgroup = 4 waves x 32 query rows = one 128-row query block of one head
//   key/value tile = 64 keys, double-buffered in LDS (K rows 16 KB, V^T 16 KB)
//   per wave per tile: S^T = K . Q^T   (2 x 8 MFMA 32x32x16, keys on rows)
//                      O^T += V^T . P^T (4 x 4 MFMA)
// Computing S^T (keys x queries) puts one query column in each lane: the 32
// scores of a lane pair form the row, so the running max/sum need a single
// cross-half exchange per tile, and the C tile converts in registers into the
// B operand of the P.V product (V^T is stored in MFMA order, see common.h).
// Query blocks are dispatched longest-first (causal work grows with the block
// index), interleaving the chunk's heads.
#include "common.h"
#include "kernels.h"

namespace upipe {

namespace {

constexpr int BQ = 128;        // query rows per workgroup
constexpr int BK = 64;         // keys per tile
constexpr int K_TILE_BYTES = BK * HEAD_DIM * 2;   // [64][128] bf16
constexpr int V_TILE_BYTES = HEAD_DIM * BK * 2;   // [128][64] bf16
constexpr int STAGE_BYTES = K_TILE_BYTES + V_TILE_BYTES;

// K tile: row r (key) is 256 B = 16 chunks of 16 B; chunk c stored at
// c ^ (r & 15) so the 16 lanes of one LDS cycle hit distinct banks.
__device__ __forceinline__ uint32_t k_off(int row, int chunk) {
  return row * 256 + ((chunk ^ (row & 15)) << 4);
}
// V^T tile: row r (head dim) is 128 B = 8 chunks; chunk c at c ^ (r & 7).
__device__ __forceinline__ uint32_t v_off(int row, int chunk) {
  return K_TILE_BYTES + row * 128 + ((chunk ^ (row & 7)) << 4);
}

struct TileRegs {
  u32x4 k[4];
  u32x4 v[4];
};

__device__ __forceinline__ void load_tile(TileRegs& r, const bf16* __restrict__ Kh,
                                          const bf16* __restrict__ Vth,
                                          int64_t Sp, int64_t kb, int t) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int pi = t + 256 * i;
    const int row = pi >> 4, chunk = pi & 15;
    r.k[i] = *reinterpret_cast<const u32x4*>(Kh + (kb + row) * HEAD_DIM + chunk * 8);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int pi = t + 256 * i;
    const int row = pi >> 3, chunk = pi & 7;
    r.v[i] = *reinterpret_cast<const u32x4*>(Vth + (int64_t)row * Sp + kb + chunk * 8);
  }
}

__device__ __forceinline__ void store_tile(const TileRegs& r, char* buf, int t) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int pi = t + 256 * i;
    lds_write_b128(buf, k_off(pi >> 4, pi & 15), r.k[i]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int pi = t + 256 * i;
    lds_write_b128(buf, v_off(pi >> 3, pi & 7), r.v[i]);
  }
}

template <bool CAUSAL>
__global__ __launch_bounds__(256, 2) void attn_fwd_kernel(
    const bf16* __restrict__ Qc, const bf16* __restrict__ Kp,
    const bf16* __restrict__ Vt, bf16* __restrict__ Oc, float* __restrict__ lse,
    int64_t S, int64_t Sp, int U, int h0, int G, int nqb) {
  __shared__ __attribute__((aligned(16))) char smem[2 * STAGE_BYTES];
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  const int r32 = lane & 31, g = lane >> 5;
  const int L = blockIdx.x;
  const int qb = nqb - 1 - L / U;
  const int u = L % U;
  const int kvh = (h0 + u) / G;
  const int64_t q0 = (int64_t)qb * BQ;
  const int64_t qw = q0 + 32 * w;          // first query row of this wave
  const int64_t myq = qw + r32;            // this lane's query row

  const bf16* Kh = Kp + (int64_t)kvh * Sp * HEAD_DIM;
  const bf16* Vth = Vt + (int64_t)kvh * HEAD_DIM * Sp;

  // Q^T B-operand fragments for the whole key loop: lane = query column,
  // k-group g covers head-dim [16s + 8g, 16s + 8g + 8).
  bf16x8 qf[8];
  {
    const bf16* qp = Qc + ((int64_t)u * Sp + myq) * HEAD_DIM + 8 * g;
#pragma unroll
    for (int s = 0; s < 8; ++s) qf[s] = *reinterpret_cast<const bf16x8*>(qp + 16 * s);
  }

  f32x16 oacc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[dt][i] = 0.f;
  float m_run = -INFINITY;   // running max of scaled scores, log2 domain
  float l_run = 0.f;         // this lane's partial row sum (16+16 keys/tile)
  const float sl2 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e)/sqrt(128)

  const int ntiles = CAUSAL ? (int)((q0 + BQ) / BK) : (int)(Sp / BK);

  TileRegs regs;
  load_tile(regs, Kh, Vth, Sp, 0, t);
  store_tile(regs, smem, t);
  __syncthreads();

  for (int j = 0; j < ntiles; ++j) {
    const int64_t kb = (int64_t)j * BK;
    char* buf = smem + (j & 1) * STAGE_BYTES;
    const bool more = j + 1 < ntiles;
    if (more) load_tile(regs, Kh, Vth, Sp, kb + BK, t);

    const bool needed = !CAUSAL || kb <= qw + 31;
    if (needed) {
      f32x16 st[2];
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
#pragma unroll
        for (int i = 0; i < 16; ++i) st[tt][i] = 0.f;
        const int row = 32 * tt + r32;
#pragma unroll
        for (int s = 0; s < 8; ++s)
          st[tt] = mfma32x32x16(lds_read_b128(buf, k_off(row, 2 * s + g)), qf[s], st[tt]);
      }
      // Mask: causal keys beyond the query row; keys past S when not causal.
      const bool diag = CAUSAL ? (kb + BK - 1 > qw) : (kb + BK > S);
      if (diag) {
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int64_t key = kb + 32 * tt + 8 * (i >> 2) + 4 * g + (i & 3);
            const bool vis = CAUSAL ? (key <= myq) : (key < S);
            if (!vis) st[tt][i] = -INFINITY;
          }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, st[tt][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx * sl2);
      const float alpha = fast_exp2(m_run - m_new);
      m_run = m_new;
      float rs = 0.f;
      bf16x8 pf[2][2];
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float p = fast_exp2(fmaf(st[tt][i], sl2, -m_new));
          rs += p;
          pf[tt][i >> 3][i & 7] = (bf16)p;
        }
      l_run = fmaf(l_run, alpha, rs);
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[dt][i] *= alpha;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const int drow = 32 * dt + r32;
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
          for (int kt = 0; kt < 2; ++kt)
            oacc[dt] = mfma32x32x16(lds_read_b128(buf, v_off(drow, 4 * tt + 2 * kt + g)),
                                    pf[tt][kt], oacc[dt]);
      }
    }
    if (more) store_tile(regs, smem + ((j + 1) & 1) * STAGE_BYTES, t);
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = 1.f / l_tot;
  bf16* op = Oc + ((int64_t)u * Sp + myq) * HEAD_DIM + 4 * g;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      bf16x4 ov;
#pragma unroll
      for (int b = 0; b < 4; ++b) ov[b] = (bf16)(oacc[dt][4 * a + b] * inv);
      *reinterpret_cast<bf16x4*>(op + 32 * dt + 8 * a) = ov;
    }
  if (g == 0 && myq < S)
    lse[(int64_t)(h0 + u) * S + myq] = (m_run + __log2f(l_tot)) * 0.6931471805599453f;
}

}  // namespace

hipError_t launch_attn_fwd(const bf16* Qc, const bf16* Kp, const bf16* Vt,
                           bf16* Oc, float* lse, int64_t S, int64_t Sp, int U,
                           int h0, int G, int causal, hipStream_t st) {
  const int nqb = (int)(Sp / BQ);
  dim3 grid((unsigned)(nqb * U));
  if (causal)
    hipLaunchKernelGGL(attn_fwd_kernel<true>, grid, dim3(256), 0, st, Qc, Kp,
                       Vt, Oc, lse, S, Sp, U, h0, G, nqb);
  else
    hipLaunchKernelGGL(attn_fwd_kernel<false>, grid, dim3(256), 0, st, Qc, Kp,
                       Vt, Oc, lse, S, Sp, U, h0, G, nqb);
  return hipGetLastError();
}

}  // namespace upipe
