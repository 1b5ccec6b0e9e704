// Causal GQA flash-attention forward for gfx950 (one head chunk per launch).
//
// Computes, for each query row i of each head of the chunk, the softmax of
// the scaled scores q_i.k_j/sqrt(d) over the visible keys and its weighted
// sum of values (paper Section 2.1), plus the row log-sum-exp (Section 2.3,
// "the final log-sum-exponent").  Online softmax over key stages keeps HBM
// traffic at O(S d) per head.
//
// Work decomposition
//   workgroup = 8 waves x 32 query rows = one 256-row query block of one head
//               (two waves per SIMD, one workgroup per CU)
//   key stage = 128 keys, double-buffered in LDS (K rows 32 KB, V rows 32 KB),
//               filled by buffer->LDS copies issued one stage ahead
//   per wave per stage: S^T = K . Q^T    (4 x 8 MFMA 32x32x16, keys on rows)
//                       O^T += V^T . P^T (8 x 4 MFMA)
// Computing S^T (keys x queries) puts one query column in each lane: the
// scores of a row sit in one lane pair, and the C tile converts in registers
// into the B operand of the P.V product, whose V^T operand is read out of
// the V rows with transposing LDS reads (tr_operand, common.h).  A stage of
// 128 keys per barrier halves the copies and barriers per product against
// 64-key tiles, and 256 rows per workgroup halve the L2->LDS traffic per
// query.
//
// Lazy rescaling: probabilities are taken against a reference max m_ref that
// moves only when needed.  A lane's sum of its stage probabilities bounds
// each of them, so the row max is computed only when that sum exceeds 2^8 (or
// is not a number, as on the first stage); O = acc / l and lse = m_ref + log l
// are exact for any reference.  Row sums add the bf16-rounded probabilities
// that enter the P.V product (v_dot2_f32_bf16), so O is normalised by the
// weights it was built from.  Query blocks are dispatched longest-first.
#include "common.h"
#include "kernels.h"

namespace upipe {

namespace {

constexpr int BQ = 256;        // query rows per workgroup (8 waves x 32)
constexpr int BKS = 128;       // keys per LDS stage
constexpr int K_TILE = BKS * HEAD_DIM * 2;       // [128][128] bf16 = 32 KB
constexpr int V_TILE = HEAD_DIM * BKS * 2;       // [128][128] bf16 = 32 KB
constexpr int STAGE = K_TILE + V_TILE;
constexpr float kSumMax = 256.f;   // lazy-rescale bound on a lane's stage sum (2^8)

// This wave's share of the copies of the 128-key stage at `kb`: 4 blocks of
// 1 KB of K rows and 4 of V rows (4 rows of 256 B each, V in the swizzle of
// transposing reads).  The lane offsets
// inside a stage are fixed; the stage offset is uniform.
__device__ __forceinline__ void issue_tile(buf_rsrc rk, buf_rsrc rv, const uint32_t (&offk)[4],
                                           const uint32_t (&offv)[4], uint32_t kb, char* buf, int w) {
#pragma unroll
  for (int i = 0; i < 4; ++i) dma_buf_b128(rk, offk[i], kb * 256u, buf + (4 * w + i) * 1024);
#pragma unroll
  for (int i = 0; i < 4; ++i) dma_buf_b128(rv, offv[i], kb * 256u, buf + K_TILE + (4 * w + i) * 1024);
}

__device__ __forceinline__ float tile_probs4(const f32x16 (&st)[4], bf16x8 (&pf)[4][2], float m_ref,
                                             float sl2) {
  float ls = 0.f;
  const bf16x2 one = {(bf16)1.f, (bf16)1.f};
#pragma unroll
  for (int tt = 0; tt < 4; ++tt)
#pragma unroll
    for (int i = 0; i < 16; i += 2) {
      bf16x2 pr;
      pr[0] = (bf16)fast_exp2(fmaf(st[tt][i], sl2, -m_ref));
      pr[1] = (bf16)fast_exp2(fmaf(st[tt][i + 1], sl2, -m_ref));
      pf[tt][i >> 3][i & 7] = pr[0];
      pf[tt][i >> 3][(i & 7) + 1] = pr[1];
      ls = __builtin_amdgcn_fdot2_f32_bf16(pr, one, ls, false);
    }
  return ls;
}

// One query block of one head against the key/value rows of its kv head.
// Query row i (of Sq, padded to Sqp) may see key j (of Skv, padded to Skvp)
// iff j <= i + delta (causal) -- delta = 0 and Skv = Sq is plain causal
// self-attention; other offsets are one ring step of context-parallel
// attention -- and always j < Skv.  A row that sees no key gets O = 0 and
// lse = -inf, the neutral element of the log-sum-exp merge.
template <bool CAUSAL>
__global__ __launch_bounds__(512, 1) void attn_fwd_kernel(
    const bf16* __restrict__ Qc, const bf16* __restrict__ Kp, const bf16* __restrict__ Vp,
    bf16* __restrict__ Oc, float* __restrict__ lse, int Sq, int Sqp, int Skv, int Skvp, int delta,
    int U, int h0, int G, int nqb, int ns, int lse_h0, int lse_ld, int lse_rows) {
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const int r32 = lane & 31, g = lane >> 5;
  // Workgroup -> (query block, head, key split), longest blocks first.
  const int L = blockIdx.x;
  const int qb = nqb - 1 - L / (U * ns);
  const int u = (L % (U * ns)) / ns;
  const int sp = L % ns;
  const int kvh = (h0 + u) / G;
  const int q0 = qb * BQ;
  const int qw = q0 + 32 * w;               // first query row of this wave
  const int myq = qw + r32;                 // this lane's query row
  const bool rows_ok = qw < Sqp;            // the last block may hold 128 rows only

  // One head's K and V rows [Skvp][128], 32-bit addressed.
  const buf_rsrc rk = make_rsrc(Kp + (int64_t)kvh * Skvp * HEAD_DIM, (uint32_t)Skvp * 256u);
  const buf_rsrc rv = make_rsrc(Vp + (int64_t)kvh * Skvp * HEAD_DIM, (uint32_t)Skvp * 256u);
  uint32_t offk[4], offv[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int blk = 4 * w + i;
    const int r = 4 * blk + (lane >> 4);       // stage row, 16 lanes per row
    const uint32_t c = (uint32_t)((lane & 15) ^ (r & 15)) << 4;
    offk[i] = r * 256u + c;
    offv[i] = r * 256u + (((lane & 15) ^ tsw(r)) << 4);
  }

  // Stages of the workgroup (up to the last key its last row may see) and
  // the leading ones holding a key visible to this wave.
  const int max_st = Skvp / BKS;
  const int nst = CAUSAL ? max(0, min(max_st, (min(q0 + BQ, Sqp) + delta + BKS - 1) / BKS)) : max_st;
  const int nw = !rows_ok ? 0 : CAUSAL ? max(0, min(nst, (qw + 32 + delta + BKS - 1) / BKS)) : nst;
  // Last visible key of this lane's row and of the wave's first row.
  const int lim = CAUSAL ? min(myq + delta, Skv - 1) : Skv - 1;
  const int lim_w = CAUSAL ? min(qw + delta, Skv - 1) : Skv - 1;
  // This split's stages [j0, j1) of the block's nst (all of them when ns = 1).
  const int per = (nst + ns - 1) / ns;
  const int j0 = min(nst, sp * per), j1 = min(nst, j0 + per);
  if (j0 < j1) issue_tile(rk, rv, offk, offv, j0 * BKS, smem + (j0 & 1) * STAGE, w);

  // Q^T B-operand fragments for the whole key loop: lane = query column,
  // k-group g covers head-dim [16s + 8g, 16s + 8g + 8).
  bf16x8 qf[8];
#pragma unroll
  for (int s = 0; s < 8; ++s)
#pragma unroll
    for (int e = 0; e < 8; ++e) qf[s][e] = (bf16)0.f;
  if (rows_ok) {
    const bf16* qp = Qc + ((int64_t)u * Sqp + myq) * HEAD_DIM + 8 * g;
#pragma unroll
    for (int s = 0; s < 8; ++s) qf[s] = *reinterpret_cast<const bf16x8*>(qp + 16 * s);
  }

  f32x16 oacc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[dt][i] = 0.f;
  // Reference max of the scaled scores (log2 domain): a finite stand-in for
  // -inf, so that a stage whose keys are all masked for a row leaves it at
  // p = 0 rather than producing 0 * inf.
  float m_ref = -1e30f;
  float l_run = 0.f;         // this lane's partial row sum
  const float sl2 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e)/sqrt(128)

  for (int j = j0; j < j1; ++j) {
    const int ks = j * BKS;
    char* buf = smem + (j & 1) * STAGE;
    wait_vmem();
    __syncthreads();   // stage j landed for all waves; stage j-1's buffer is free
    if (j + 1 < j1) issue_tile(rk, rv, offk, offv, ks + BKS, smem + ((j + 1) & 1) * STAGE, w);
    if (j >= nw) continue;                  // whole stage masked for this wave
    {
      const int kb = ks;
      f32x16 st[4];
#pragma unroll
      for (int tt = 0; tt < 4; ++tt)
#pragma unroll
        for (int i = 0; i < 16; ++i) st[tt][i] = 0.f;
#pragma unroll
      for (int s = 0; s < 8; ++s)
#pragma unroll
        for (int tt = 0; tt < 4; ++tt)
          st[tt] = mfma32x32x16(lds_read_b128(buf, swz256(32 * tt + r32, 2 * s + g)), qf[s], st[tt]);
      // Keep six K fragment reads in flight ahead of the MFMAs: left alone,
      // the scheduler reads two, waits for them and multiplies, exposing the
      // LDS latency every two MFMAs.
      __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
#pragma unroll
      for (int i = 0; i < 26; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 6, 0);
      // Mask keys past the row's last visible key (wave-uniform test first).
      if (kb + BKS - 1 > lim_w) {
#pragma unroll
        for (int tt = 0; tt < 4; ++tt)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int key = kb + 32 * tt + 8 * (i >> 2) + 4 * g + (i & 3);
            if (key > lim) st[tt][i] = -INFINITY;
          }
      }
      bf16x8 pf[4][2];
      float ls = tile_probs4(st, pf, m_ref, sl2);
      if (__builtin_amdgcn_ballot_w64(!(ls <= kSumMax)) != 0) {
        float mx = st[0][0];
#pragma unroll
        for (int tt = 0; tt < 4; ++tt)
#pragma unroll
          for (int i = 0; i < 16; ++i) mx = fmaxf(mx, st[tt][i]);
        mx = fmaxf(mx, __shfl_xor(mx, 32)) * sl2;
        const float m_new = fmaxf(m_ref, mx);
        const float alpha = fast_exp2(m_ref - m_new);
        m_ref = m_new;
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int i = 0; i < 16; ++i) oacc[dt][i] *= alpha;
        ls = tile_probs4(st, pf, m_ref, sl2);
      }
      l_run += ls;
#pragma unroll
      for (int c = 0; c < 8; ++c)
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
          oacc[dt] = mfma32x32x16(tr_operand(buf + K_TILE, 16 * c, 32 * dt, lane), pf[c >> 1][c & 1],
                                  oacc[dt]);
      // Stream the V^T fragments: four (eight transposing reads) ahead, then
      // two reads per MFMA (the default schedule issued bursts of eight
      // reads and waited between them).
      __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
      for (int i = 0; i < 28; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
    }
  }

  if (!rows_ok) return;
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;   // no visible key: O = 0
  bf16* op = Oc + ((int64_t)(sp * U + u) * Sqp + myq) * HEAD_DIM + 4 * g;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      bf16x4 ov;
#pragma unroll
      for (int b = 0; b < 4; ++b) ov[b] = (bf16)(oacc[dt][4 * a + b] * inv);
      *reinterpret_cast<bf16x4*>(op + 32 * dt + 8 * a) = ov;
    }
  if (g == 0 && myq < lse_rows)
    lse[(int64_t)(lse_h0 + sp * U + u) * lse_ld + myq] =
        l_tot > 0.f ? (m_ref + __log2f(l_tot)) * 0.6931471805599453f : -INFINITY;
}

}  // namespace

hipError_t launch_attn_fwd_split(const bf16* Qc, const bf16* Kp, const bf16* Vp, bf16* Oc,
                                 float* lse, int64_t Sq, int64_t Sqp, int64_t Skv, int64_t Skvp,
                                 int64_t delta, int U, int h0, int G, int causal, int ns,
                                 int lse_h0, int64_t lse_ld, int64_t lse_rows, hipStream_t st) {
  const int nqb = (int)((Sqp + BQ - 1) / BQ);
  // Offsets beyond either length change nothing: clamp into int range.
  const int dl = (int)(delta < -Sq ? -Sq : delta > Skv ? Skv : delta);
  dim3 grid((unsigned)(nqb * U * ns));
  if (causal)
    hipLaunchKernelGGL(attn_fwd_kernel<true>, grid, dim3(512), 0, st, Qc, Kp, Vp, Oc, lse, (int)Sq,
                       (int)Sqp, (int)Skv, (int)Skvp, dl, U, h0, G, nqb, ns, lse_h0, (int)lse_ld,
                       (int)lse_rows);
  else
    hipLaunchKernelGGL(attn_fwd_kernel<false>, grid, dim3(512), 0, st, Qc, Kp, Vp, Oc, lse, (int)Sq,
                       (int)Sqp, (int)Skv, (int)Skvp, dl, U, h0, G, nqb, ns, lse_h0, (int)lse_ld,
                       (int)lse_rows);
  return hipGetLastError();
}

hipError_t launch_attn_fwd(const bf16* Qc, const bf16* Kp, const bf16* Vp, bf16* Oc, float* lse,
                           int64_t Sq, int64_t Sqp, int64_t Skv, int64_t Skvp, int64_t delta, int U,
                           int h0, int G, int causal, hipStream_t st) {
  return launch_attn_fwd_split(Qc, Kp, Vp, Oc, lse, Sq, Sqp, Skv, Skvp, delta, U, h0, G, causal, 1,
                               h0, Sq, Sq, st);
}

int attn_fwd_key_splits(int64_t Sqp, int64_t Skvp) {
  // Fewer 256-row query blocks than half the CUs leave CUs idle at U = 1:
  // split the key range of every block in two (a function of the lengths
  // only, so that every chunk size U gives the same results).
  return ((Sqp + BQ - 1) / BQ <= 128 && Skvp / BKS >= 2) ? 2 : 1;
}

}  // namespace upipe
