// Causal GQA flash-attention backward for gfx950 (one head chunk per launch).
//
// Analytic gradient of softmax attention (paper Section 2.1), with the
// probabilities rebuilt from the saved row log-sum-exp:
//   P_ij  = exp(q_i.k_j/sqrt d - lse_i),   D_i = dO_i . O_i
//   dS_ij = P_ij (dO_i . v_j - D_i)
//   dV_j += sum_i P_ij dO_i,   dK_j += sum_i dS_ij q_i / sqrt d,
//   dQ_i  = sum_j dS_ij k_j / sqrt d.
// Two kernels, no atomics, one fixed summation order:
//   dkdv: a workgroup owns 128 keys of one key/value head (4 waves x 32 keys)
//         and walks the chunk's query heads in ascending order, and within a
//         head the 32-row query tiles in ascending order.  Its fp32 dK/dV
//         accumulators start from the values the previous chunk left in the
//         workspace (UPipe keeps per-group dK/dV accumulators alive across
//         stages, Appendix A), so any chunk size U yields bit-identical sums.
//   dq:   a workgroup owns 128 query rows of one head and walks key tiles in
//         ascending order, recomputing P and dS.
// Transposed operands come from the MFMA-ordered [d][S] copies (common.h).
#include "common.h"
#include "kernels.h"

namespace upipe {

namespace {

constexpr float kSl2 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e)/sqrt(128)
constexpr float kScale = 0.08838834764831845f;                      // 1/sqrt(128)
constexpr float kLog2e = 1.4426950408889634f;

// ------------------------------------------------------------------ dK / dV
// LDS stage for one 32-row query tile: Q [32][128], dO [32][128] (rows of
// 256 B, chunk swizzle c ^ (r & 15)), Q^T and dO^T [128][32] in MFMA order
// (rows of 64 B, chunk swizzle c ^ ((r >> 1) & 3)), lse*log2e and D [32].
constexpr int QT = 32;
constexpr int ROWT_BYTES = QT * HEAD_DIM * 2;       // 8 KB
constexpr int OFF_Q = 0, OFF_DO = ROWT_BYTES, OFF_QT = 2 * ROWT_BYTES,
              OFF_DOT = 3 * ROWT_BYTES, OFF_LSE = 4 * ROWT_BYTES,
              OFF_D = OFF_LSE + QT * 4;
constexpr int KV_STAGE = OFF_D + QT * 4;

__device__ __forceinline__ uint32_t row_off(int row, int chunk) {
  return row * 256 + ((chunk ^ (row & 15)) << 4);
}
__device__ __forceinline__ uint32_t col_off(int drow, int chunk) {
  return drow * 64 + ((chunk ^ ((drow >> 1) & 3)) << 4);
}

struct QTileRegs {
  u32x4 q[2], dO[2], qt[2], dOt[2];
  float lse, D;
};

// Each tile is 512 pieces of 16 bytes: 256 threads move two pieces of each
// of the four tiles; threads 0..31 / 32..63 also move one float of lse / D.
__device__ __forceinline__ void load_qtile(QTileRegs& r, const bf16* Qh, const bf16* Qth,
                                           const bf16* dOh, const bf16* dOth,
                                           const float* lseh, const float* Dh,
                                           int64_t Sp, int64_t qb, int t) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int pi = t + 256 * i;
    const int row = pi >> 4, chunk = pi & 15;
    r.q[i] = *reinterpret_cast<const u32x4*>(Qh + (qb + row) * HEAD_DIM + chunk * 8);
    r.dO[i] = *reinterpret_cast<const u32x4*>(dOh + (qb + row) * HEAD_DIM + chunk * 8);
    const int drow = pi >> 2, c = pi & 3;
    r.qt[i] = *reinterpret_cast<const u32x4*>(Qth + (int64_t)drow * Sp + qb + c * 8);
    r.dOt[i] = *reinterpret_cast<const u32x4*>(dOth + (int64_t)drow * Sp + qb + c * 8);
  }
  if (t < 32) r.lse = lseh[qb + t] * kLog2e;
  else if (t < 64) r.D = Dh[qb + t - 32];
}

__device__ __forceinline__ void store_qtile(const QTileRegs& r, char* buf, int t) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int pi = t + 256 * i;
    const int row = pi >> 4, chunk = pi & 15;
    lds_write_b128(buf + OFF_Q, row_off(row, chunk), r.q[i]);
    lds_write_b128(buf + OFF_DO, row_off(row, chunk), r.dO[i]);
    const int drow = pi >> 2, c = pi & 3;
    lds_write_b128(buf + OFF_QT, col_off(drow, c), r.qt[i]);
    lds_write_b128(buf + OFF_DOT, col_off(drow, c), r.dOt[i]);
  }
  if (t < 32) reinterpret_cast<float*>(buf + OFF_LSE)[t] = r.lse;
  else if (t < 64) reinterpret_cast<float*>(buf + OFF_D)[t - 32] = r.D;
}

template <bool CAUSAL>
__global__ __launch_bounds__(256, 1) void attn_bwd_dkdv_kernel(
    const bf16* __restrict__ Qc, const bf16* __restrict__ Qct,
    const bf16* __restrict__ dOc, const bf16* __restrict__ dOct,
    const float* __restrict__ lse_c, const float* __restrict__ Dc,
    const bf16* __restrict__ Kp, const bf16* __restrict__ Vp,
    float* __restrict__ dK32, float* __restrict__ dV32,
    bf16* __restrict__ dk, bf16* __restrict__ dv,
    int64_t S, int64_t Sp, int U, int h0, int G, int Hkv) {
  __shared__ __attribute__((aligned(16))) char smem[2 * KV_STAGE];
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  const int r32 = lane & 31, g = lane >> 5;
  const int kvh = h0 / G + blockIdx.y;
  const int64_t kb0 = (int64_t)blockIdx.x * 128;
  const int64_t kw = kb0 + 32 * w;      // first key of this wave
  const int64_t mykey = kw + r32;       // key column owned by this lane
  const int hlo = max(h0, kvh * G), hhi = min(h0 + U, (kvh + 1) * G);
  const bool first = kvh * G >= h0;           // no earlier chunk touched kvh
  const bool last = (kvh + 1) * G <= h0 + U;  // no later chunk will

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
  const int64_t accbase = (int64_t)kvh * Sp * HEAD_DIM;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if (first) {
        dka[dt][i] = 0.f;
        dva[dt][i] = 0.f;
      } else {
        const int64_t key = kw + 8 * (i >> 2) + 4 * g + (i & 3);
        const int64_t off = accbase + key * HEAD_DIM + 32 * dt + r32;
        dka[dt][i] = dK32[off];
        dva[dt][i] = dV32[off];
      }
    }

  const int64_t qt_begin = CAUSAL ? kb0 / QT : 0;
  const int64_t qt_end = Sp / QT;
  const int64_t per_head = qt_end - qt_begin;
  const int64_t total = per_head * (hhi - hlo);

  QTileRegs regs;
  auto tile_ptrs_load = [&](int64_t it) {
    const int hh = hlo + (int)(it / per_head) - h0;
    const int64_t qb = (qt_begin + it % per_head) * QT;
    load_qtile(regs, Qc + (int64_t)hh * Sp * HEAD_DIM, Qct + (int64_t)hh * HEAD_DIM * Sp,
               dOc + (int64_t)hh * Sp * HEAD_DIM, dOct + (int64_t)hh * HEAD_DIM * Sp,
               lse_c + (int64_t)hh * Sp, Dc + (int64_t)hh * Sp, Sp, qb, t);
  };
  if (total > 0) {
    tile_ptrs_load(0);
    store_qtile(regs, smem, t);
  }
  __syncthreads();

  for (int64_t it = 0; it < total; ++it) {
    const int64_t qb = (qt_begin + it % per_head) * QT;
    char* buf = smem + (it & 1) * KV_STAGE;
    const bool more = it + 1 < total;
    if (more) tile_ptrs_load(it + 1);

    const bool needed = !CAUSAL || qb + QT - 1 >= kw;
    if (needed) {
      f32x16 sacc, pacc;
#pragma unroll
      for (int i = 0; i < 16; ++i) { sacc[i] = 0.f; pacc[i] = 0.f; }
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        sacc = mfma32x32x16(lds_read_b128(buf + OFF_Q, row_off(r32, 2 * s + g)), kf[s], sacc);
        pacc = mfma32x32x16(lds_read_b128(buf + OFF_DO, row_off(r32, 2 * s + g)), vf[s], pacc);
      }
      const float* lsel = reinterpret_cast<const float*>(buf + OFF_LSE);
      const float* Dl = reinterpret_cast<const float*>(buf + OFF_D);
      bf16x8 pf[2], sf[2];
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const f32x4 l4 = *reinterpret_cast<const f32x4*>(lsel + 8 * a + 4 * g);
        const f32x4 d4 = *reinterpret_cast<const f32x4*>(Dl + 8 * a + 4 * g);
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int i = 4 * a + b;
          float p = fast_exp2(fmaf(sacc[i], kSl2, -l4[b]));
          if (CAUSAL) {
            const int64_t q = qb + 8 * a + 4 * g + b;
            if (mykey > q) p = 0.f;
          }
          const float ds = p * (pacc[i] - d4[b]);
          pf[i >> 3][i & 7] = (bf16)p;
          sf[i >> 3][i & 7] = (bf16)ds;
        }
      }
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const int drow = 32 * dt + r32;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
          dva[dt] = mfma32x32x16(pf[kt], lds_read_b128(buf + OFF_DOT, col_off(drow, 2 * kt + g)), dva[dt]);
          dka[dt] = mfma32x32x16(sf[kt], lds_read_b128(buf + OFF_QT, col_off(drow, 2 * kt + g)), dka[dt]);
        }
      }
    }
    if (more) store_qtile(regs, smem + ((it + 1) & 1) * KV_STAGE, t);
    __syncthreads();
  }

#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int64_t key = kw + 8 * (i >> 2) + 4 * g + (i & 3);
      const int d = 32 * dt + r32;
      if (last) {
        if (key < S) {
          const int64_t off = (key * Hkv + kvh) * HEAD_DIM + d;
          dk[off] = (bf16)(dka[dt][i] * kScale);
          dv[off] = (bf16)dva[dt][i];
        }
      } else {
        const int64_t off = accbase + key * HEAD_DIM + d;
        dK32[off] = dka[dt][i];
        dV32[off] = dva[dt][i];
      }
    }
}

// ---------------------------------------------------------------------- dQ
// LDS stage for one 64-key tile: K [64][128], V [64][128] (256-B rows,
// swizzle c ^ (r & 15)) and K^T [128][64] in MFMA order (128-B rows,
// swizzle c ^ (r & 7)).
constexpr int BKQ = 64;
constexpr int KT_BYTES = BKQ * HEAD_DIM * 2;   // 16 KB
constexpr int DQ_OFF_K = 0, DQ_OFF_V = KT_BYTES, DQ_OFF_KT = 2 * KT_BYTES;
constexpr int DQ_STAGE = 3 * KT_BYTES;

__device__ __forceinline__ uint32_t kt_off(int drow, int chunk) {
  return drow * 128 + ((chunk ^ (drow & 7)) << 4);
}

struct KTileRegs {
  u32x4 k[4], v[4], kt[4];
};

__device__ __forceinline__ void load_ktile(KTileRegs& r, const bf16* Kh, const bf16* Vh,
                                           const bf16* Kth, int64_t Sp, int64_t kb, int t) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int pi = t + 256 * i;
    const int row = pi >> 4, chunk = pi & 15;
    r.k[i] = *reinterpret_cast<const u32x4*>(Kh + (kb + row) * HEAD_DIM + chunk * 8);
    r.v[i] = *reinterpret_cast<const u32x4*>(Vh + (kb + row) * HEAD_DIM + chunk * 8);
    const int drow = pi >> 3, c = pi & 7;
    r.kt[i] = *reinterpret_cast<const u32x4*>(Kth + (int64_t)drow * Sp + kb + c * 8);
  }
}

__device__ __forceinline__ void store_ktile(const KTileRegs& r, char* buf, int t) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int pi = t + 256 * i;
    lds_write_b128(buf + DQ_OFF_K, row_off(pi >> 4, pi & 15), r.k[i]);
    lds_write_b128(buf + DQ_OFF_V, row_off(pi >> 4, pi & 15), r.v[i]);
    lds_write_b128(buf + DQ_OFF_KT, kt_off(pi >> 3, pi & 7), r.kt[i]);
  }
}

template <bool CAUSAL>
__global__ __launch_bounds__(256, 1) void attn_bwd_dq_kernel(
    const bf16* __restrict__ Qc, const bf16* __restrict__ dOc,
    const float* __restrict__ lse_c, const float* __restrict__ Dc,
    const bf16* __restrict__ Kp, const bf16* __restrict__ Kt,
    const bf16* __restrict__ Vp, bf16* __restrict__ dQc,
    int64_t S, int64_t Sp, int U, int h0, int G, int nqb) {
  __shared__ __attribute__((aligned(16))) char smem[2 * DQ_STAGE];
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  const int r32 = lane & 31, g = lane >> 5;
  const int L = blockIdx.x;
  const int qb = nqb - 1 - L / U;
  const int u = L % U;
  const int kvh = (h0 + u) / G;
  const int64_t q0 = (int64_t)qb * 128;
  const int64_t qw = q0 + 32 * w;
  const int64_t myq = qw + r32;

  const bf16* Kh = Kp + (int64_t)kvh * Sp * HEAD_DIM;
  const bf16* Vh = Vp + (int64_t)kvh * Sp * HEAD_DIM;
  const bf16* Kth = Kt + (int64_t)kvh * HEAD_DIM * Sp;

  bf16x8 qf[8], df[8];
  {
    const int64_t rowoff = ((int64_t)u * Sp + myq) * HEAD_DIM + 8 * g;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      qf[s] = *reinterpret_cast<const bf16x8*>(Qc + rowoff + 16 * s);
      df[s] = *reinterpret_cast<const bf16x8*>(dOc + rowoff + 16 * s);
    }
  }
  const float lse2 = lse_c[(int64_t)u * Sp + myq] * kLog2e;
  const float Dq = Dc[(int64_t)u * Sp + myq];

  f32x16 qacc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) qacc[dt][i] = 0.f;

  const int ntiles = CAUSAL ? (int)((q0 + 128) / BKQ) : (int)(Sp / BKQ);
  KTileRegs regs;
  load_ktile(regs, Kh, Vh, Kth, Sp, 0, t);
  store_ktile(regs, smem, t);
  __syncthreads();

  for (int j = 0; j < ntiles; ++j) {
    const int64_t kb = (int64_t)j * BKQ;
    char* buf = smem + (j & 1) * DQ_STAGE;
    const bool more = j + 1 < ntiles;
    if (more) load_ktile(regs, Kh, Vh, Kth, Sp, kb + BKQ, t);

    const bool needed = !CAUSAL || kb <= qw + 31;
    if (needed) {
      bf16x8 sf[2][2];
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
        f32x16 sacc, pacc;
#pragma unroll
        for (int i = 0; i < 16; ++i) { sacc[i] = 0.f; pacc[i] = 0.f; }
        const int row = 32 * tt + r32;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          sacc = mfma32x32x16(lds_read_b128(buf + DQ_OFF_K, row_off(row, 2 * s + g)), qf[s], sacc);
          pacc = mfma32x32x16(lds_read_b128(buf + DQ_OFF_V, row_off(row, 2 * s + g)), df[s], pacc);
        }
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int64_t key = kb + 32 * tt + 8 * (i >> 2) + 4 * g + (i & 3);
          float p = fast_exp2(fmaf(sacc[i], kSl2, -lse2));
          const bool vis = CAUSAL ? (key <= myq) : (key < S);
          if (!vis) p = 0.f;
          sf[tt][i >> 3][i & 7] = (bf16)(p * (pacc[i] - Dq));
        }
      }
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const int drow = 32 * dt + r32;
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
          for (int kt = 0; kt < 2; ++kt)
            qacc[dt] = mfma32x32x16(lds_read_b128(buf + DQ_OFF_KT, kt_off(drow, 4 * tt + 2 * kt + g)),
                                    sf[tt][kt], qacc[dt]);
      }
    }
    if (more) store_ktile(regs, smem + ((j + 1) & 1) * DQ_STAGE, t);
    __syncthreads();
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

hipError_t launch_attn_bwd_dkdv(const bf16* Qc, const bf16* Qct,
                                const bf16* dOc, const bf16* dOct,
                                const float* lse_c, const float* D,
                                const bf16* Kp, const bf16* Vp, float* dK32,
                                float* dV32, bf16* dk, bf16* dv, int64_t S,
                                int64_t Sp, int U, int h0, int G, int Hkv,
                                int causal, hipStream_t st) {
  const int kv_lo = h0 / G, kv_hi = (h0 + U - 1) / G;
  dim3 grid((unsigned)(Sp / 128), (unsigned)(kv_hi - kv_lo + 1));
  if (causal)
    hipLaunchKernelGGL(attn_bwd_dkdv_kernel<true>, grid, dim3(256), 0, st, Qc,
                       Qct, dOc, dOct, lse_c, D, Kp, Vp, dK32, dV32, dk, dv, S,
                       Sp, U, h0, G, Hkv);
  else
    hipLaunchKernelGGL(attn_bwd_dkdv_kernel<false>, grid, dim3(256), 0, st, Qc,
                       Qct, dOc, dOct, lse_c, D, Kp, Vp, dK32, dV32, dk, dv, S,
                       Sp, U, h0, G, Hkv);
  return hipGetLastError();
}

hipError_t launch_attn_bwd_dq(const bf16* Qc, const bf16* dOc,
                              const float* lse_c, const float* D,
                              const bf16* Kp, const bf16* Kt, const bf16* Vp,
                              bf16* dQc, int64_t S, int64_t Sp, int U, int h0,
                              int G, int causal, hipStream_t st) {
  const int nqb = (int)(Sp / 128);
  dim3 grid((unsigned)(nqb * U));
  if (causal)
    hipLaunchKernelGGL(attn_bwd_dq_kernel<true>, grid, dim3(256), 0, st, Qc,
                       dOc, lse_c, D, Kp, Kt, Vp, dQc, S, Sp, U, h0, G, nqb);
  else
    hipLaunchKernelGGL(attn_bwd_dq_kernel<false>, grid, dim3(256), 0, st, Qc,
                       dOc, lse_c, D, Kp, Kt, Vp, dQc, S, Sp, U, h0, G, nqb);
  return hipGetLastError();
}

}  // namespace upipe
