// Causal GQA flash-attention backward for gfx950 (one head chunk per launch).
//
// Analytic gradient of softmax attention (paper Section 2.1), with the
// probabilities rebuilt from the saved row log-sum-exp:
//   P_ij  = exp(q_i.k_j/sqrt d - lse_i),   D_i = dO_i . O_i
//   dS_ij = P_ij (dO_i . v_j - D_i)
//   dV_j += sum_i P_ij dO_i,   dK_j += sum_i dS_ij q_i / sqrt d,
//   dQ_i  = sum_j dS_ij k_j / sqrt d.
// Two kernels, no atomics, one fixed summation order:
//   dkdv: a workgroup owns 128 keys of one key/value head (4 waves x 32 keys,
//         K and V fragments in registers) and walks the chunk's query heads in
//         ascending order and, within a head, the 64-row query tiles from the
//         last one down to its diagonal (the two 32-row halves of a tile in
//         ascending order), so that all resident workgroups read
//         the same query tiles at about the same time (shared L2 lines).  Its
//         fp32 dK/dV accumulators start from the values the previous chunk
//         left in the workspace (UPipe keeps per-group dK/dV accumulators alive
//         across stages, Appendix A), so any chunk size U gives bit-identical
//         sums.
//   dq:   a workgroup owns 128 query rows of one head and walks 32-key tiles
//         in ascending order, recomputing P and dS.
// Tiles reach LDS through direct global->LDS copies issued one tile ahead.
// Transposed operands come from the MFMA-ordered [d][S] copies (common.h).
#include "common.h"
#include "kernels.h"

namespace upipe {

namespace {

constexpr float kSl2 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e)/sqrt(128)
constexpr float kScale = 0.08838834764831845f;                      // 1/sqrt(128)

// ------------------------------------------------------------------ dK / dV
// LDS stage for one 64-row query tile (two 32-row subtiles): Q [64][128] and
// dO [64][128] (256-B rows), Q^T and dO^T [128][64] in MFMA order (128-B
// rows), lse and D [64].  Two subtiles per stage let one subtile's softmax
// gradient (VALU) overlap the other's products (MFMA) within a wave.
constexpr int QT = 64;
constexpr int ROWT = QT * HEAD_DIM * 2;   // 16 KB
constexpr int OFF_Q = 0, OFF_DO = ROWT, OFF_QT = 2 * ROWT, OFF_DOT = 3 * ROWT,
              OFF_LSE = 4 * ROWT, OFF_D = OFF_LSE + QT * 4;
constexpr int KV_STAGE = 4 * ROWT + 1024;   // lse/D block padded to 1 KB

struct QTilePtrs {
  const char *q, *dO, *qt, *dOt, *lse, *D;   // head bases (bytes)
  uint32_t col_bytes;                          // row stride of the [d][Sp] copies
};

// Wave w copies four 1 KB blocks of each of Q, dO (4 rows of 256 B per block)
// and Q^T, dO^T (8 rows of 128 B per block); wave 0 also copies lse and D.
__device__ __forceinline__ void issue_qtile(const QTilePtrs& p, uint32_t qb, char* buf, int w,
                                            int lane) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int blk = 4 * w + i;
    const int row = 4 * blk + (lane >> 4);
    const uint32_t off = (qb + row) * 256u + (((lane & 15) ^ (row & 15)) << 4);
    dma_b128(p.q + off, buf + OFF_Q + blk * 1024);
    dma_b128(p.dO + off, buf + OFF_DO + blk * 1024);
    const int crow = 8 * blk + (lane >> 3);
    const uint32_t coff = crow * p.col_bytes + qb * 2u +
                          (((lane & 7) ^ (crow & 7) ^ ((crow >> 3) & 1)) << 4);
    dma_b128(p.qt + coff, buf + OFF_QT + blk * 1024);
    dma_b128(p.dOt + coff, buf + OFF_DOT + blk * 1024);
  }
  if (w == 0 && lane < 32) {
    const char* src = lane < 16 ? p.lse + qb * 4u + lane * 16u : p.D + qb * 4u + (lane - 16) * 16u;
    dma_b128(src, buf + OFF_LSE);
  }
}

// One 32-row query subtile: rows qs..qs+31 at offset `sub` (0 or 32) in the
// stage.  Returns the bf16 P and dS fragments for the dV / dK products.
template <bool CAUSAL>
__device__ __forceinline__ void subtile_scores(const char* buf, int sub, uint32_t qs,
                                               uint32_t mykey, bool diag, int r32, int g,
                                               const bf16x8 (&kf)[8], const bf16x8 (&vf)[8],
                                               bf16x8 (&pf)[2], bf16x8 (&sf)[2]) {
  f32x16 sacc, pacc;
#pragma unroll
  for (int i = 0; i < 16; ++i) { sacc[i] = 0.f; pacc[i] = 0.f; }
  const int row = sub + r32;
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    sacc = mfma32x32x16(lds_read_b128(buf + OFF_Q, swz256(row, 2 * s + g)), kf[s], sacc);
    pacc = mfma32x32x16(lds_read_b128(buf + OFF_DO, swz256(row, 2 * s + g)), vf[s], pacc);
  }
  const float* lsel = reinterpret_cast<const float*>(buf + OFF_LSE) + sub;
  const float* Dl = reinterpret_cast<const float*>(buf + OFF_D) + sub;
  float p[16];
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    const f32x4 l4 = *reinterpret_cast<const f32x4*>(lsel + 8 * a + 4 * g);
#pragma unroll
    for (int b = 0; b < 4; ++b) p[4 * a + b] = fast_exp2(fmaf(sacc[4 * a + b], kSl2, -l4[b]));
  }
  if (CAUSAL && diag) {   // wave-uniform: only tiles that cross the diagonal
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (mykey > qs + 8 * (i >> 2) + 4 * g + (i & 3)) p[i] = 0.f;
  }
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    const f32x4 d4 = *reinterpret_cast<const f32x4*>(Dl + 8 * a + 4 * g);
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int i = 4 * a + b;
      pf[i >> 3][i & 7] = (bf16)p[i];
      sf[i >> 3][i & 7] = (bf16)(p[i] * (pacc[i] - d4[b]));
    }
  }
}

template <bool CAUSAL>
__global__ __launch_bounds__(256, 1) void attn_bwd_dkdv_kernel(
    const bf16* __restrict__ Qc, const bf16* __restrict__ Qct, const bf16* __restrict__ dOc,
    const bf16* __restrict__ dOct, const float* __restrict__ lse_c, const float* __restrict__ Dc,
    const bf16* __restrict__ Kp, const bf16* __restrict__ Vp, float* __restrict__ dK32,
    float* __restrict__ dV32, bf16* __restrict__ dk, bf16* __restrict__ dv, int64_t S, int64_t Sp,
    int U, int h0, int G, int Hkv) {
  __shared__ __attribute__((aligned(1024))) char smem[2 * KV_STAGE];
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  const int r32 = lane & 31, g = lane >> 5;
  const int kvh = h0 / G + blockIdx.y;
  const uint32_t kb0 = blockIdx.x * 128u;
  const uint32_t kw = kb0 + 32 * w;      // first key of this wave
  const uint32_t mykey = kw + r32;       // key column owned by this lane
  const int hlo = max(h0, kvh * G), hhi = min(h0 + U, (kvh + 1) * G);
  const bool first = kvh * G >= h0;           // no earlier chunk touched kvh
  const bool last = (kvh + 1) * G <= h0 + U;  // no later chunk will
  const uint32_t nqt = (uint32_t)(Sp / QT);
  const uint32_t qt_lo = CAUSAL ? kb0 / QT : 0;   // lowest query tile needed
  const uint32_t per_head = nqt - qt_lo;
  const int total = (int)(per_head * (hhi - hlo));

  auto ptrs = [&](int hh) {
    QTilePtrs p;
    const int64_t hoff = (int64_t)(hh - h0) * Sp * HEAD_DIM;
    p.q = reinterpret_cast<const char*>(Qc + hoff);
    p.dO = reinterpret_cast<const char*>(dOc + hoff);
    p.qt = reinterpret_cast<const char*>(Qct + hoff);
    p.dOt = reinterpret_cast<const char*>(dOct + hoff);
    p.lse = reinterpret_cast<const char*>(lse_c + (int64_t)(hh - h0) * Sp);
    p.D = reinterpret_cast<const char*>(Dc + (int64_t)(hh - h0) * Sp);
    p.col_bytes = (uint32_t)Sp * 2u;
    return p;
  };

  // First tile: head hlo, query tile nqt-1.
  QTilePtrs cur = ptrs(hlo);
  issue_qtile(cur, (nqt - 1) * QT, smem, w, lane);

  // K and V B-operand fragments (lane = key column, k = head dim).
  bf16x8 kf[8], vf[8];
  {
    const bf16* kp = Kp + ((int64_t)kvh * Sp + mykey) * HEAD_DIM + 8 * g;
    const bf16* vp = Vp + ((int64_t)kvh * Sp + mykey) * HEAD_DIM + 8 * g;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      kf[s] = *reinterpret_cast<const bf16x8*>(kp + 16 * s);
      vf[s] = *reinterpret_cast<const bf16x8*>(vp + 16 * s);
    }
  }

  // Accumulators: C layout with lane = head-dim column 32*dt + r32 and
  // element i = key row kw + 8*(i/4) + 4*g + (i%4).
  f32x16 dka[4], dva[4];
  float* dK32h = dK32 + (int64_t)kvh * Sp * HEAD_DIM;
  float* dV32h = dV32 + (int64_t)kvh * Sp * HEAD_DIM;
  if (first) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        dka[dt][i] = 0.f;
        dva[dt][i] = 0.f;
      }
  } else {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const uint32_t off = (kw + 8 * (i >> 2) + 4 * g + (i & 3)) * HEAD_DIM + 32 * dt + r32;
        dka[dt][i] = dK32h[off];
        dva[dt][i] = dV32h[off];
      }
  }

  int hh = hlo;
  uint32_t qt = nqt - 1;     // query tile of the current iteration
  for (int it = 0; it < total; ++it) {
    char* buf = smem + (it & 1) * KV_STAGE;
    const uint32_t qb = qt * QT;
    // next tile (descending query tiles, then the next head)
    uint32_t nq = qt - 1;
    int nh = hh;
    if (qt == qt_lo) {
      nq = nqt - 1;
      nh = hh + 1;
    }
    wait_vmem();
    __syncthreads();   // this tile landed for all waves; the other buffer is free
    if (it + 1 < total) {
      if (nh != hh) cur = ptrs(nh);
      issue_qtile(cur, nq * QT, smem + ((it + 1) & 1) * KV_STAGE, w, lane);
    }

    // Subtile 1 (rows qb+32..63) is needed whenever subtile 0 is.
    const bool need0 = !CAUSAL || qb + 31 >= kw;
    const bool need1 = !CAUSAL || qb + 63 >= kw;
    if (need1) {
      bf16x8 pf1[2], sf1[2];
      subtile_scores<CAUSAL>(buf, 32, qb + 32, mykey, qb + 32 < kw + 31, r32, g, kf, vf, pf1, sf1);
      if (need0) {
        bf16x8 pf0[2], sf0[2];
        subtile_scores<CAUSAL>(buf, 0, qb, mykey, qb < kw + 31, r32, g, kf, vf, pf0, sf0);
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) {
          const int drow = 32 * dt + r32;
#pragma unroll
          for (int kt = 0; kt < 2; ++kt) {
            dva[dt] = mfma32x32x16(pf0[kt], lds_read_b128(buf + OFF_DOT, swz128(drow, 2 * kt + g)), dva[dt]);
            dka[dt] = mfma32x32x16(sf0[kt], lds_read_b128(buf + OFF_QT, swz128(drow, 2 * kt + g)), dka[dt]);
          }
        }
      }
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const int drow = 32 * dt + r32;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
          dva[dt] = mfma32x32x16(pf1[kt], lds_read_b128(buf + OFF_DOT, swz128(drow, 4 + 2 * kt + g)), dva[dt]);
          dka[dt] = mfma32x32x16(sf1[kt], lds_read_b128(buf + OFF_QT, swz128(drow, 4 + 2 * kt + g)), dka[dt]);
        }
      }
    }
    qt = nq;
    hh = nh;
  }

  if (last) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const uint32_t key = kw + 8 * (i >> 2) + 4 * g + (i & 3);
        if (key < (uint64_t)S) {
          const int64_t off = ((int64_t)key * Hkv + kvh) * HEAD_DIM + 32 * dt + r32;
          dk[off] = (bf16)(dka[dt][i] * kScale);
          dv[off] = (bf16)dva[dt][i];
        }
      }
  } else {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const uint32_t off = (kw + 8 * (i >> 2) + 4 * g + (i & 3)) * HEAD_DIM + 32 * dt + r32;
        dK32h[off] = dka[dt][i];
        dV32h[off] = dva[dt][i];
      }
  }
}

// ---------------------------------------------------------------------- dQ
// LDS stage for one 32-key tile: K [32][128], V [32][128] (256-B rows) and
// K^T [128][32] in MFMA order (64-B rows).
constexpr int BKQ = 32;
constexpr int KT8 = BKQ * HEAD_DIM * 2;   // 8 KB
constexpr int DQ_OFF_K = 0, DQ_OFF_V = KT8, DQ_OFF_KT = 2 * KT8;
constexpr int DQ_STAGE = 3 * KT8;

__device__ __forceinline__ void issue_ktile(const char* Kh, const char* Vh, const char* Kth,
                                            uint32_t col_bytes, uint32_t kb, char* buf, int w,
                                            int lane) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int blk = 2 * w + i;
    const int row = 4 * blk + (lane >> 4);
    const uint32_t off = (kb + row) * 256u + (((lane & 15) ^ (row & 15)) << 4);
    dma_b128(Kh + off, buf + DQ_OFF_K + blk * 1024);
    dma_b128(Vh + off, buf + DQ_OFF_V + blk * 1024);
    const int crow = 16 * blk + (lane >> 2);
    dma_b128(Kth + crow * col_bytes + kb * 2u + (((lane & 3) ^ ((crow >> 2) & 3)) << 4),
             buf + DQ_OFF_KT + blk * 1024);
  }
}

template <bool CAUSAL>
__global__ __launch_bounds__(256, 2) void attn_bwd_dq_kernel(
    const bf16* __restrict__ Qc, const bf16* __restrict__ dOc, const float* __restrict__ lse_c,
    const float* __restrict__ Dc, const bf16* __restrict__ Kp, const bf16* __restrict__ Kt,
    const bf16* __restrict__ Vp, bf16* __restrict__ dQc, int64_t S, int64_t Sp, int U, int h0,
    int G, int nqb) {
  __shared__ __attribute__((aligned(1024))) char smem[2 * DQ_STAGE];
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  const int r32 = lane & 31, g = lane >> 5;
  const int L = blockIdx.x;
  const int qb = nqb - 1 - L / U;
  const int u = L % U;
  const int kvh = (h0 + u) / G;
  const uint32_t q0 = (uint32_t)qb * 128;
  const uint32_t qw = q0 + 32 * w;
  const uint32_t myq = qw + r32;
  const uint32_t Sv = (uint32_t)S;

  const char* Kh = reinterpret_cast<const char*>(Kp + (int64_t)kvh * Sp * HEAD_DIM);
  const char* Vh = reinterpret_cast<const char*>(Vp + (int64_t)kvh * Sp * HEAD_DIM);
  const char* Kth = reinterpret_cast<const char*>(Kt + (int64_t)kvh * HEAD_DIM * Sp);
  const uint32_t col_bytes = (uint32_t)Sp * 2u;
  const int ntiles = CAUSAL ? (int)((q0 + 128) / BKQ) : (int)(Sp / BKQ);
  issue_ktile(Kh, Vh, Kth, col_bytes, 0, smem, w, lane);

  bf16x8 qf[8], df[8];
  {
    const int64_t rowoff = ((int64_t)u * Sp + myq) * HEAD_DIM + 8 * g;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      qf[s] = *reinterpret_cast<const bf16x8*>(Qc + rowoff + 16 * s);
      df[s] = *reinterpret_cast<const bf16x8*>(dOc + rowoff + 16 * s);
    }
  }
  const float lse2 = lse_c[(int64_t)u * Sp + myq];   // already times log2(e)
  const float Dq = Dc[(int64_t)u * Sp + myq];

  f32x16 qacc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) qacc[dt][i] = 0.f;

  for (int j = 0; j < ntiles; ++j) {
    const uint32_t kb = (uint32_t)j * BKQ;
    char* buf = smem + (j & 1) * DQ_STAGE;
    wait_vmem();
    __syncthreads();
    if (j + 1 < ntiles)
      issue_ktile(Kh, Vh, Kth, col_bytes, kb + BKQ, smem + ((j + 1) & 1) * DQ_STAGE, w, lane);
    if (CAUSAL && kb > qw + 31) continue;

    f32x16 sacc, pacc;
#pragma unroll
    for (int i = 0; i < 16; ++i) { sacc[i] = 0.f; pacc[i] = 0.f; }
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      sacc = mfma32x32x16(lds_read_b128(buf + DQ_OFF_K, swz256(r32, 2 * s + g)), qf[s], sacc);
      pacc = mfma32x32x16(lds_read_b128(buf + DQ_OFF_V, swz256(r32, 2 * s + g)), df[s], pacc);
    }
    const bool diag = CAUSAL ? (kb + BKQ - 1 > qw) : (kb + BKQ > Sv);
    float p[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) p[i] = fast_exp2(fmaf(sacc[i], kSl2, -lse2));
    if (diag) {   // wave-uniform
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const uint32_t key = kb + 8 * (i >> 2) + 4 * g + (i & 3);
        const bool vis = CAUSAL ? (key <= myq) : (key < Sv);
        if (!vis) p[i] = 0.f;
      }
    }
    bf16x8 sf[2];
#pragma unroll
    for (int i = 0; i < 16; ++i) sf[i >> 3][i & 7] = (bf16)(p[i] * (pacc[i] - Dq));
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const int drow = 32 * dt + r32;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
        qacc[dt] = mfma32x32x16(lds_read_b128(buf + DQ_OFF_KT, swz64b(drow, 2 * kt + g)), sf[kt],
                                qacc[dt]);
    }
  }

  bf16* op = dQc + ((int64_t)u * Sp + myq) * HEAD_DIM + 4 * g;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      bf16x4 ov;
#pragma unroll
      for (int b = 0; b < 4; ++b) ov[b] = (bf16)(qacc[dt][4 * a + b] * kScale);
      *reinterpret_cast<bf16x4*>(op + 32 * dt + 8 * a) = ov;
    }
}

}  // namespace

hipError_t launch_attn_bwd_dkdv(const bf16* Qc, const bf16* Qct, const bf16* dOc,
                                const bf16* dOct, const float* lse_c, const float* D,
                                const bf16* Kp, const bf16* Vp, float* dK32, float* dV32, bf16* dk,
                                bf16* dv, int64_t S, int64_t Sp, int U, int h0, int G, int Hkv,
                                int causal, hipStream_t st) {
  const int kv_lo = h0 / G, kv_hi = (h0 + U - 1) / G;
  dim3 grid((unsigned)(Sp / 128), (unsigned)(kv_hi - kv_lo + 1));
  if (causal)
    hipLaunchKernelGGL(attn_bwd_dkdv_kernel<true>, grid, dim3(256), 0, st, Qc, Qct, dOc, dOct,
                       lse_c, D, Kp, Vp, dK32, dV32, dk, dv, S, Sp, U, h0, G, Hkv);
  else
    hipLaunchKernelGGL(attn_bwd_dkdv_kernel<false>, grid, dim3(256), 0, st, Qc, Qct, dOc, dOct,
                       lse_c, D, Kp, Vp, dK32, dV32, dk, dv, S, Sp, U, h0, G, Hkv);
  return hipGetLastError();
}

hipError_t launch_attn_bwd_dq(const bf16* Qc, const bf16* dOc, const float* lse_c, const float* D,
                              const bf16* Kp, const bf16* Kt, const bf16* Vp, bf16* dQc, int64_t S,
                              int64_t Sp, int U, int h0, int G, int causal, hipStream_t st) {
  const int nqb = (int)(Sp / 128);
  dim3 grid((unsigned)(nqb * U));
  if (causal)
    hipLaunchKernelGGL(attn_bwd_dq_kernel<true>, grid, dim3(256), 0, st, Qc, dOc, lse_c, D, Kp, Kt,
                       Vp, dQc, S, Sp, U, h0, G, nqb);
  else
    hipLaunchKernelGGL(attn_bwd_dq_kernel<false>, grid, dim3(256), 0, st, Qc, dOc, lse_c, D, Kp,
                       Kt, Vp, dQc, S, Sp, U, h0, G, nqb);
  return hipGetLastError();
}

}  // namespace upipe
