// Causal GQA flash-attention forward for gfx950 (one head chunk per launch).
//
// Computes, for each query row i of each head of the chunk, the softmax of
// the scaled scores q_i.k_j/sqrt(d) over the visible keys and its weighted
// sum of values (paper Section 2.1), plus the row log-sum-exp (Section 2.3,
// "the final log-sum-exponent").  Online softmax over key tiles keeps HBM
// traffic at O(S d) per head.
//
// Work decomposition
//   workgroup = 4 waves x 32 query rows = one 128-row query block of one head
//   key/value tile = 64 keys, double-buffered in LDS (K rows 16 KB, V^T 16 KB)
//   filled by direct global->LDS copies issued one tile ahead
//   per wave per tile: S^T = K . Q^T   (2 x 8 MFMA 32x32x16, keys on rows)
//                      O^T += V^T . P^T (4 x 4 MFMA)
// Computing S^T (keys x queries) puts one query column in each lane: the 64
// scores of a row sit in one lane pair, so the running max needs a single
// cross-half exchange per tile, and the C tile converts in registers into the
// B operand of the P.V product (V^T is stored in MFMA order, see common.h).
//
// Lazy rescaling: the reference max m of a row only moves when a tile's max
// exceeds it by more than 2^8 (decided per wave), so most tiles skip the
// rescale of the 64 accumulator registers; probabilities stay <= 2^8 and the
// final O = acc / l and lse = m + log l are exact for any reference m.
// Query blocks are dispatched longest-first (causal work grows with the block
// index), interleaving the chunk's heads.
#include "common.h"
#include "kernels.h"

namespace upipe {

namespace {

constexpr int BQ = 128;        // query rows per workgroup
constexpr int BK = 64;         // keys per tile
constexpr int K_TILE = BK * HEAD_DIM * 2;        // [64][128] bf16 = 16 KB
constexpr int V_TILE = HEAD_DIM * BK * 2;        // [128][64] bf16 = 16 KB
constexpr int STAGE = K_TILE + V_TILE;
constexpr float kTau = 8.f;    // lazy-rescale threshold (log2 domain)

// Issue this wave's share of the copies of key tile `kb` into `buf`:
// 4 blocks of 1 KB of K rows (4 rows each) and 4 blocks of V^T rows (8 each).
__device__ __forceinline__ void issue_tile(const char* Kh, const char* Vth, uint32_t vt_row_bytes,
                                           uint32_t kb, char* buf, int w, int lane) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int blk = 4 * w + i;
    const int row = 4 * blk + (lane >> 4);
    const int c = (lane & 15) ^ (row & 15);
    dma_b128(Kh + (kb + row) * 256u + c * 16u, buf + blk * 1024);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int blk = 4 * w + i;
    const int row = 8 * blk + (lane >> 3);
    const int c = (lane & 7) ^ (row & 7) ^ ((row >> 3) & 1);
    dma_b128(Vth + row * vt_row_bytes + kb * 2u + c * 16u, buf + K_TILE + blk * 1024);
  }
}

template <bool CAUSAL>
__global__ __launch_bounds__(256, 2) void attn_fwd_kernel(
    const bf16* __restrict__ Qc, const bf16* __restrict__ Kp, const bf16* __restrict__ Vt,
    bf16* __restrict__ Oc, float* __restrict__ lse, int64_t S, int64_t Sp, int U, int h0, int G,
    int nqb) {
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  const int r32 = lane & 31, g = lane >> 5;
  const int L = blockIdx.x;
  const int qb = nqb - 1 - L / U;
  const int u = L % U;
  const int kvh = (h0 + u) / G;
  const uint32_t q0 = (uint32_t)qb * BQ;
  const uint32_t qw = q0 + 32 * w;          // first query row of this wave
  const uint32_t myq = qw + r32;            // this lane's query row
  const uint32_t Sv = (uint32_t)S;

  const char* Kh = reinterpret_cast<const char*>(Kp + (int64_t)kvh * Sp * HEAD_DIM);
  const char* Vth = reinterpret_cast<const char*>(Vt + (int64_t)kvh * HEAD_DIM * Sp);
  const uint32_t vt_row_bytes = (uint32_t)Sp * 2u;

  const int ntiles = CAUSAL ? (int)((q0 + BQ) / BK) : (int)(Sp / BK);
  issue_tile(Kh, Vth, vt_row_bytes, 0, smem, w, lane);

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
  float m_ref = -INFINITY;   // reference max of scaled scores, log2 domain
  float l_run = 0.f;         // this lane's partial row sum
  const float sl2 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e)/sqrt(128)

  for (int j = 0; j < ntiles; ++j) {
    const uint32_t kb = (uint32_t)j * BK;
    char* buf = smem + (j & 1) * STAGE;
    wait_vmem();
    __syncthreads();   // tile j landed for all waves; tile j-1's buffer is free
    if (j + 1 < ntiles) issue_tile(Kh, Vth, vt_row_bytes, kb + BK, smem + ((j + 1) & 1) * STAGE, w, lane);

    if (CAUSAL && kb > qw + 31) continue;   // whole tile masked for this wave
    f32x16 st[2];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
#pragma unroll
      for (int i = 0; i < 16; ++i) st[tt][i] = 0.f;
      const int row = 32 * tt + r32;
#pragma unroll
      for (int s = 0; s < 8; ++s)
        st[tt] = mfma32x32x16(lds_read_b128(buf, swz256(row, 2 * s + g)), qf[s], st[tt]);
    }
    // Mask: causal keys beyond the query row; keys past S when not causal.
    const bool diag = CAUSAL ? (kb + BK - 1 > qw) : (kb + BK > Sv);
    if (diag) {
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const uint32_t key = kb + 32 * tt + 8 * (i >> 2) + 4 * g + (i & 3);
          const bool vis = CAUSAL ? (key <= myq) : (key < Sv);
          if (!vis) st[tt][i] = -INFINITY;
        }
    }
    float mx = st[0][0];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, st[tt][i]);
    mx = fmaxf(mx, __shfl_xor(mx, 32)) * sl2;
    if (__builtin_amdgcn_ballot_w64(mx > m_ref + kTau) != 0) {
      const float m_new = fmaxf(m_ref, mx);
      const float alpha = fast_exp2(m_ref - m_new);
      m_ref = m_new;
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[dt][i] *= alpha;
    }
    bf16x8 pf[2][2];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float p = fast_exp2(fmaf(st[tt][i], sl2, -m_ref));
        l_run += p;
        pf[tt][i >> 3][i & 7] = (bf16)p;
      }
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const int drow = 32 * dt + r32;
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
          oacc[dt] = mfma32x32x16(lds_read_b128(buf + K_TILE, swz128(drow, 4 * tt + 2 * kt + g)),
                                  pf[tt][kt], oacc[dt]);
    }
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
  if (g == 0 && myq < Sv)
    lse[(int64_t)(h0 + u) * S + myq] = (m_ref + __log2f(l_tot)) * 0.6931471805599453f;
}

}  // namespace

hipError_t launch_attn_fwd(const bf16* Qc, const bf16* Kp, const bf16* Vt, bf16* Oc, float* lse,
                           int64_t S, int64_t Sp, int U, int h0, int G, int causal,
                           hipStream_t st) {
  const int nqb = (int)(Sp / BQ);
  dim3 grid((unsigned)(nqb * U));
  if (causal)
    hipLaunchKernelGGL(attn_fwd_kernel<true>, grid, dim3(256), 0, st, Qc, Kp, Vt, Oc, lse, S, Sp,
                       U, h0, G, nqb);
  else
    hipLaunchKernelGGL(attn_fwd_kernel<false>, grid, dim3(256), 0, st, Qc, Kp, Vt, Oc, lse, S, Sp,
                       U, h0, G, nqb);
  return hipGetLastError();
}

}  // namespace upipe
