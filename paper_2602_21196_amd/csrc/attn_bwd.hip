// Causal GQA flash-attention backward for gfx950 (one head chunk per launch).
//
// Analytic gradient of softmax attention (paper Section 2.1), with the
// probabilities rebuilt from the saved row log-sum-exp (staged as -sqrt(d) lse,
// the initial value of each row's score accumulator):
//   P_ij  = exp(q_i.k_j/sqrt d - lse_i),   D_i = dO_i . O_i
//   dS_ij = P_ij (dO_i . v_j - D_i)
//   dV_j += sum_i P_ij dO_i,   dK_j += sum_i dS_ij q_i / sqrt d,
//   dQ_i  = sum_j dS_ij k_j / sqrt d.
// Two kernels, no atomics, one fixed summation order:
//   dkdv: a workgroup owns 128 keys of one key/value head (4 waves x 32 keys,
//         K and V fragments in registers) and walks the chunk's query heads in
//         ascending order and, within a head, the 128-row query tiles from the
//         last one down to its diagonal (each tile as 64-row halves, upper
//         first, and each half as two 32-row subtiles, upper first), so that
//         all resident workgroups read the same query tiles at about the same
//         time (shared L2 lines).  Its
//         fp32 dK/dV accumulators start from the values the previous chunk
//         left in the workspace (UPipe keeps per-group dK/dV accumulators alive
//         across stages, Appendix A), so any chunk size U gives bit-identical
//         sums.
//   dq:   a workgroup owns 256 query rows of one head (8 waves) and walks
//         64-key stages in ascending order, recomputing P and dS.
// Tiles reach LDS through buffer->LDS copies issued one tile ahead.
// Transposed operands are read out of row-major tiles (common.h, tr_operand).
#include "common.h"
#include "kernels.h"

namespace upipe {

namespace {

constexpr float kSl2 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e)/sqrt(128)
constexpr float kScale = 0.08838834764831845f;                      // 1/sqrt(128)

// ------------------------------------------------------------------ dK / dV
// LDS stage for one tile of QT query rows of one head: Q and dO rows
// [QT][128] (256-B rows, transposing-read swizzle), then lse and D [QT].  The
// B operands of dV += P^T dO and dK += dS^T Q are read out of the rows with
// transposing LDS reads, so no [d][S] copies of Q and dO are needed.  A tile
// is consumed as pairs of 32-row subtiles, the upper 64 rows first.
constexpr int QT = 128;
constexpr int ROWT = QT * HEAD_DIM * 2;
constexpr int OFF_Q = 0, OFF_DO = ROWT, OFF_LSE = 2 * ROWT, OFF_D = OFF_LSE + QT * 4;
constexpr int KV_STAGE = 2 * ROWT + QT * 8;
constexpr int KV_BLK = ROWT / 1024 / 4;     // 1 KB blocks per wave per array

struct QStageSrc {
  buf_rsrc q, dO, lse, D;
};

// This wave's share of one tile's copies: KV_BLK blocks of 1 KB each of Q and
// dO rows; lanes of wave 0 copy the QT lse values, lanes of wave 1 the QT D
// values (16 bytes per lane).
__device__ __forceinline__ void issue_qstage(const QStageSrc& r, uint32_t qb, char* buf, int w,
                                             int lane) {
  // The source offsets are recomputed for every tile (a few VALU
  // instructions) instead of being held in registers across the tile loop,
  // where the register file is full; the empty asm keeps the compiler from
  // hoisting them back out of the loop.
  asm volatile("" : "+v"(lane));
#pragma unroll
  for (int i = 0; i < KV_BLK; ++i) {
    const int blk = KV_BLK * w + i;
    // this lane's 16 bytes: Q / dO row `row` of the tile (16 lanes per row),
    // chunk swizzled for the transposing reads
    const int row = 4 * blk + (lane >> 4);
    const uint32_t off = row * 256u + (((lane & 15) ^ tsw(row)) << 4);
    dma_buf_b128(r.q, off, qb * 256u, buf + OFF_Q + blk * 1024);
    dma_buf_b128(r.dO, off, qb * 256u, buf + OFF_DO + blk * 1024);
  }
  if (lane < QT / 4) {
    if (w == 0) dma_buf_b128(r.lse, lane * 16u, qb * 4u, buf + OFF_LSE);
    else if (w == 1) dma_buf_b128(r.D, lane * 16u, qb * 4u, buf + OFF_D);
  }
}

// Operand fragments of one block of 16 MFMAs.
struct Frags {
  bf16x8 f[16];
};

// S^T / dP^T block of one 32-row subtile (rows `sub`..+31 of the tile):
// fragment 2 s + 0 is Q, 2 s + 1 is dO, both for head-dim 16 s..
__device__ __forceinline__ void read_sdp(const char* buf, int sub, int r32, int g, Frags& fr) {
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    fr.f[2 * s] = lds_read_b128(buf + OFF_Q, swzt(sub + r32, 2 * s + g));
    fr.f[2 * s + 1] = lds_read_b128(buf + OFF_DO, swzt(sub + r32, 2 * s + g));
  }
}

// dV / dK block of one subtile: fragment 4 dt + 2 kt + 0 is dO, + 1 is Q, as
// B operands with head-dim columns 32 dt.. and the 16 query rows sub + 16 kt..
__device__ __forceinline__ void read_dvdk(const char* buf, int sub, int lane, Frags& fr) {
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      fr.f[4 * dt + 2 * kt] = tr_operand(buf + OFF_DO, sub + 16 * kt, 32 * dt, lane);
      fr.f[4 * dt + 2 * kt + 1] = tr_operand(buf + OFF_Q, sub + 16 * kt, 32 * dt, lane);
    }
}

// Accumulator seeds of the 32-row subtile at rows `sub`.. of the tile, in the
// MFMA C layout (element 4a + b is row sub + 8a + 4g + b), loaded from the
// staged rows straight into the accumulators: the score accumulator starts at
// -sqrt(d) lse of its row, so that it ends at q.k - sqrt(d) lse and
// P = exp2(acc log2(e) / sqrt(d)) needs no lse term; the dP accumulator
// starts at D, and the value fragments come negated, so that chain ends at
// D - dP and dS needs no subtraction: P (D - dP) = -dS.  A pair's seeds are
// read before its fragments: LDS reads complete in order, and a seed read
// behind a burst of fragment reads would wait for the whole burst.
__device__ __forceinline__ void subtile_seed(const char* buf, int sub, int g, f32x16& sacc,
                                             f32x16& pacc) {
  const float* Dl = reinterpret_cast<const float*>(buf + OFF_D) + sub;
  const float* Ll = reinterpret_cast<const float*>(buf + OFF_LSE) + sub;
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    const f32x4 d4 = *reinterpret_cast<const f32x4*>(Dl + 8 * a + 4 * g);
    const f32x4 l4 = *reinterpret_cast<const f32x4*>(Ll + 8 * a + 4 * g);
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      pacc[4 * a + b] = d4[b];
      sacc[4 * a + b] = l4[b];
    }
  }
}

// S^T and D - dP^T of one subtile from its fragments (16 MFMAs), on top of
// the seeds.
__device__ __forceinline__ void subtile_sdp(const Frags& fr, const bf16x8 (&kf)[8],
                                            const bf16x8 (&nvf)[8], f32x16& sacc, f32x16& pacc) {
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    sacc = mfma32x32x16(fr.f[2 * s], kf[s], sacc);
    pacc = mfma32x32x16(fr.f[2 * s + 1], nvf[s], pacc);
  }
}

// P and -dS of one subtile as bf16 A operands, from its lse-seeded scores
// and D - dP.  Negation is exact and commutes with rounding, so the dK
// accumulators carry exactly -dK (the final scale is -1/sqrt d).  No masking
// here (subtile_mask).
__device__ __forceinline__ void subtile_pds(const f32x16& sacc, const f32x16& pacc,
                                            bf16x8 (&pf)[2], bf16x8 (&sf)[2]) {
  float p[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) p[i] = fast_exp2(sacc[i] * kSl2);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    pf[i >> 3][i & 7] = (bf16)p[i];
    sf[i >> 3][i & 7] = (bf16)(p[i] * pacc[i]);
  }
}

// Subtiles across the diagonal (wave-uniform `diag`; first row qs): zero the
// P and dS entries of keys after the row, by selection (unmasked they may be
// inf or NaN).  This runs after the conversions and between two regions: a
// branch ends the compiler's scheduling block, and inside a region it would
// split the MFMA / VALU interleave in two.
template <bool CAUSAL>
__device__ __forceinline__ void subtile_mask(uint32_t qs, uint32_t mykey, bool diag, int g,
                                             bf16x8 (&pf)[2], bf16x8 (&sf)[2]) {
  if (CAUSAL && diag) {
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (mykey > qs + 8 * (i >> 2) + 4 * g + (i & 3)) {
        pf[i >> 3][i & 7] = (bf16)0.f;
        sf[i >> 3][i & 7] = (bf16)0.f;
      }
  }
}

__device__ __forceinline__ void dvdk_products(const Frags& fr, const bf16x8 (&pf)[2],
                                              const bf16x8 (&sf)[2], f32x16 (&dva)[4],
                                              f32x16 (&dka)[4]) {
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      dva[dt] = mfma32x32x16(pf[kt], fr.f[4 * dt + 2 * kt], dva[dt]);
      dka[dt] = mfma32x32x16(sf[kt], fr.f[4 * dt + 2 * kt + 1], dka[dt]);
    }
}

// Scheduling request for a region of 16 MFMAs and the VALU work of one
// subtile's P and dS: one MFMA after every few VALU instructions, so the
// matrix unit and the vector ALU of the one wave on the SIMD work side by
// side (the region's LDS reads are left to the scheduler: asking for them
// first bunched the first MFMAs behind them).
constexpr int KV_NV = 5;   // VALU instructions requested between two MFMAs
// Region A (no VALU): its 16 MFMAs with the 32 transposing reads of the
// next block's fragments, two per MFMA; region D with the next pair's
// fragment reads, one per MFMA.
template <int NDS>
__device__ __forceinline__ void interleave_mfma_lds() {
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, NDS, 0);
  }
}
__device__ __forceinline__ void interleave_mfma_valu() {
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, KV_NV, 0);
  }
}

// One pair of subtiles (rows base..base+63 of the tile), in four fenced
// regions so that each block of 16 MFMAs shares its region with VALU work it
// does not depend on:
//   A: S/dP products of the upper subtile
//   B: S/dP products of the lower subtile   | P, dS of the upper subtile
//   C: dV/dK products of the upper subtile  | P, dS of the lower subtile
//   D: dV/dK products of the lower subtile
// The LDS fragments of each block are read one region ahead; fa holds the
// upper subtile's S / dP fragments on entry, and with PF it is refilled
// during region D (which has no other LDS reads) with those of the next
// pair of the tile.  The lower subtile is computed even where only the upper
// one is needed: the diagonal mask then zeroes all of its P and dS.
template <bool CAUSAL, bool PF>
__device__ __forceinline__ void pair_step(const char* buf, int base, uint32_t qb, uint32_t kw,
                                          uint32_t mykey, int r32, int g, int lane,
                                          const bf16x8 (&kf)[8], const bf16x8 (&vf)[8],
                                          f32x16 (&dva)[4], f32x16 (&dka)[4], Frags& fa) {
  Frags fb;
  f32x16 s1, p1, s0, p0;
  bf16x8 pf1[2], sf1[2], pf0[2], sf0[2];
  const uint32_t q1 = qb + base + 32, q0 = qb + base;
  subtile_seed(buf, base + 32, g, s1, p1);
  subtile_seed(buf, base, g, s0, p0);
  __builtin_amdgcn_sched_barrier(0);
  read_sdp(buf, base, r32, g, fb);
  __builtin_amdgcn_sched_barrier(0);
  subtile_sdp(fa, kf, vf, s1, p1);                                            // A
  read_dvdk(buf, base + 32, lane, fa);
  interleave_mfma_lds<2>();
  __builtin_amdgcn_sched_barrier(0);
  subtile_sdp(fb, kf, vf, s0, p0);                                            // B
  subtile_pds(s1, p1, pf1, sf1);
  interleave_mfma_valu();
  __builtin_amdgcn_sched_barrier(0);
  subtile_mask<CAUSAL>(q1, mykey, q1 < kw + 31, g, pf1, sf1);
  dvdk_products(fa, pf1, sf1, dva, dka);                                      // C
  read_dvdk(buf, base, lane, fb);
  subtile_pds(s0, p0, pf0, sf0);
  interleave_mfma_valu();
  __builtin_amdgcn_sched_barrier(0);
  subtile_mask<CAUSAL>(q0, mykey, q0 < kw + 31, g, pf0, sf0);
  dvdk_products(fb, pf0, sf0, dva, dka);                                      // D
  if (PF) {   // the next pair's upper subtile
    read_sdp(buf, base - 32, r32, g, fa);
    interleave_mfma_lds<1>();
  }
}

template <bool CAUSAL>
__global__ __launch_bounds__(256, 1) void attn_bwd_dkdv_kernel(
    const bf16* __restrict__ Qc, const bf16* __restrict__ dOc, const float* __restrict__ lse_c,
    const float* __restrict__ Dc, const bf16* __restrict__ Kp, const bf16* __restrict__ Vp,
    float* __restrict__ dK32,
    float* __restrict__ dV32, bf16* __restrict__ dk, bf16* __restrict__ dv, int64_t S, int64_t Sp,
    int U, int h0, int G, int64_t kv_row, int64_t kv_head) {
  __shared__ __attribute__((aligned(1024))) char smem[2 * KV_STAGE];
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const int r32 = lane & 31, g = lane >> 5;
  const int kvh = h0 / G + blockIdx.y;
  const uint32_t kb0 = blockIdx.x * 128u;
  const uint32_t kw = kb0 + 32 * w;      // first key of this wave
  const uint32_t mykey = kw + r32;       // key column owned by this lane
  const uint32_t Spv = (uint32_t)Sp;
  const int hlo = max(h0, kvh * G), hhi = min(h0 + U, (kvh + 1) * G);
  const bool first = kvh * G >= h0;           // no earlier chunk touched kvh
  const bool last = (kvh + 1) * G <= h0 + U;  // no later chunk will
  const uint32_t nqt = (Spv + QT - 1) / QT;
  const uint32_t qt_lo = CAUSAL ? kb0 / QT : 0;   // lowest query tile needed
  const uint32_t per_head = nqt - qt_lo;
  const int total = (int)(per_head * (hhi - hlo));

  auto srcs = [&](int hh) {
    QStageSrc r;
    const int64_t hoff = (int64_t)(hh - h0) * Sp * HEAD_DIM;
    r.q = make_rsrc(Qc + hoff, Spv * 256u);
    r.dO = make_rsrc(dOc + hoff, Spv * 256u);
    r.lse = make_rsrc(lse_c + (int64_t)(hh - h0) * Sp, Spv * 4u);
    r.D = make_rsrc(Dc + (int64_t)(hh - h0) * Sp, Spv * 4u);
    return r;
  };

  // First tile: head hlo, query tile nqt-1.
  QStageSrc cur = srcs(hlo);
  issue_qstage(cur, (nqt - 1) * QT, smem, w, lane);

  // K and -V B-operand fragments (lane = key column, k = head dim); -V makes
  // the dP products count down from D.
  bf16x8 kf[8], vf[8];
  {
    const bf16* kp = Kp + ((int64_t)kvh * Sp + mykey) * HEAD_DIM + 8 * g;
    const bf16* vp = Vp + ((int64_t)kvh * Sp + mykey) * HEAD_DIM + 8 * g;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      kf[s] = *reinterpret_cast<const bf16x8*>(kp + 16 * s);
      vf[s] = -*reinterpret_cast<const bf16x8*>(vp + 16 * s);
    }
    // They are only ever MFMA operands, which may come from AGPRs: placing
    // them there leaves the VGPRs to the score accumulators and the P / dS
    // arithmetic (fewer AGPR -> VGPR moves, no spills).
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      asm volatile("" : "+a"(kf[s]));
      asm volatile("" : "+a"(vf[s]));
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
      if (nh != hh) cur = srcs(nh);
      issue_qstage(cur, nq * QT, smem + ((it + 1) & 1) * KV_STAGE, w, lane);
    }
    // Pairs of 32-row subtiles, upper rows first; a pair is needed when its
    // last row reaches this wave's first key (and lies inside the sequence).
    // The upper pair reads the lower pair's first fragments in its region D.
    Frags fa;
    const bool run1 = qb + 64 < Spv && (!CAUSAL || qb + 127 >= kw);
    const bool run0 = qb < Spv && (!CAUSAL || qb + 63 >= kw);
    if (run1) {
      read_sdp(buf, 96, r32, g, fa);
      pair_step<CAUSAL, true>(buf, 64, qb, kw, mykey, r32, g, lane, kf, vf, dva, dka, fa);
    }
    if (run0) {
      if (!run1) read_sdp(buf, 32, r32, g, fa);
      pair_step<CAUSAL, false>(buf, 0, qb, kw, mykey, r32, g, lane, kf, vf, dva, dka, fa);
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
          const int64_t off = (int64_t)key * kv_row + kvh * kv_head + 32 * dt + r32;
          dk[off] = (bf16)(dka[dt][i] * -kScale);
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
// Workgroup = 8 waves x 32 query rows (256 rows, two waves per SIMD).  LDS
// stage for one tile of DQ_BK keys: K and V rows [DQ_BK][128] (256-B rows).
// The A operand of dQ^T = K^T . dS^T is read out of the K rows with
// transposing LDS reads, so no [d][S] copy of K is needed.
constexpr int DQ_BQ = 256;
constexpr int DQ_BK = 64;
constexpr int DQ_T = DQ_BK * HEAD_DIM * 2;
constexpr int DQ_OFF_K = 0, DQ_OFF_V = DQ_T;
constexpr int DQ_STAGE = 2 * DQ_T;
constexpr int DQ_BLK = DQ_T / 1024 / 8;   // 1 KB blocks per wave per tile
constexpr int DQ_LA = 6;                   // K/V fragment reads kept in flight

// This wave's share of one tile's copies: DQ_BLK blocks of 1 KB each of K
// rows (transposing-read swizzle) and V rows (4 rows of 256 B per block).
__device__ __forceinline__ void issue_kstage(buf_rsrc rk, buf_rsrc rv, const uint32_t (&offk)[DQ_BLK],
                                             const uint32_t (&offv)[DQ_BLK], uint32_t kb, char* buf,
                                             int w) {
#pragma unroll
  for (int i = 0; i < DQ_BLK; ++i) {
    const int blk = DQ_BLK * w + i;
    dma_buf_b128(rk, offk[i], kb * 256u, buf + DQ_OFF_K + blk * 1024);
    dma_buf_b128(rv, offv[i], kb * 256u, buf + DQ_OFF_V + blk * 1024);
  }
}

template <bool CAUSAL, bool ROPE>
__global__ __launch_bounds__(512, 1) void attn_bwd_dq_kernel(
    const bf16* __restrict__ Qc, const bf16* __restrict__ dOc, const float* __restrict__ lse_c,
    const float* __restrict__ Dc, const bf16* __restrict__ Kp, const bf16* __restrict__ Vp,
    bf16* __restrict__ dQc, int64_t S, int64_t Sp, int U, int h0,
    int G, int nqb, RopeArgs rope) {
  __shared__ __attribute__((aligned(1024))) char smem[2 * DQ_STAGE];
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const int r32 = lane & 31, g = lane >> 5;
  const int L = blockIdx.x;
  const int qb = nqb - 1 - L / U;
  const int u = L % U;
  const int kvh = (h0 + u) / G;
  const uint32_t Spv = (uint32_t)Sp;
  const uint32_t q0 = (uint32_t)qb * DQ_BQ;
  const uint32_t qw = q0 + 32 * w;
  const uint32_t myq = qw + r32;
  const uint32_t Sv = (uint32_t)S;
  const bool rows_ok = qw < Spv;            // the last block may hold 128 rows only

  // One head's K and V rows [Sp][128], 32-bit addressed.
  const buf_rsrc rk = make_rsrc(Kp + (int64_t)kvh * Sp * HEAD_DIM, Spv * 256u);
  const buf_rsrc rv = make_rsrc(Vp + (int64_t)kvh * Sp * HEAD_DIM, Spv * 256u);
  uint32_t offk[DQ_BLK], offv[DQ_BLK];
#pragma unroll
  for (int i = 0; i < DQ_BLK; ++i) {
    const int blk = DQ_BLK * w + i;
    const int r = 4 * blk + (lane >> 4);      // row of the tile, 16 lanes per row
    offk[i] = r * 256u + (((lane & 15) ^ tsw(r)) << 4);
    offv[i] = r * 256u + (((lane & 15) ^ (r & 15)) << 4);
  }
  const int nst = CAUSAL ? (int)((min(q0 + DQ_BQ, Spv) + DQ_BK - 1) / DQ_BK) : (int)(Spv / DQ_BK);
  issue_kstage(rk, rv, offk, offv, 0, smem, w);

  bf16x8 qf[8], df[8];
  float nlse = 0.f, Dq = 0.f;
#pragma unroll
  for (int s = 0; s < 8; ++s)
#pragma unroll
    for (int e = 0; e < 8; ++e) { qf[s][e] = (bf16)0.f; df[s][e] = (bf16)0.f; }
  if (rows_ok) {
    const int64_t rowoff = ((int64_t)u * Sp + myq) * HEAD_DIM + 8 * g;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      qf[s] = *reinterpret_cast<const bf16x8*>(Qc + rowoff + 16 * s);
      df[s] = *reinterpret_cast<const bf16x8*>(dOc + rowoff + 16 * s);
    }
    nlse = lse_c[(int64_t)u * Sp + myq];   // -sqrt(d) lse: the score accumulator's seed
    Dq = Dc[(int64_t)u * Sp + myq];
  }

  f32x16 qacc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) qacc[dt][i] = 0.f;

  for (int j = 0; j < nst; ++j) {
    const uint32_t ks = (uint32_t)j * DQ_BK;
    char* buf = smem + (j & 1) * DQ_STAGE;
    wait_vmem();
    __syncthreads();   // tile j landed for all waves; tile j-1's buffer is free
    if (j + 1 < nst) issue_kstage(rk, rv, offk, offv, ks + DQ_BK, smem + ((j + 1) & 1) * DQ_STAGE, w);
    if (!rows_ok) continue;
#pragma unroll
    for (int h64 = 0; h64 < DQ_BK / 64; ++h64) {
      const uint32_t kb = ks + 64 * h64;
      if (CAUSAL && kb > qw + 31) break;     // rest of the tile masked for this wave
      const bool diag = CAUSAL ? (kb + 63 > qw) : (kb + 64 > Sv);
      // The 64 keys in two halves of 32: one score and one dP accumulator
      // live at a time, which leaves registers for DQ_LA fragment reads in
      // flight ahead of the S / dP MFMAs (with both halves' accumulators
      // live the compiler kept one, waiting before every MFMA).  The dQ
      // products still add the 16-key steps in ascending order.
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        f32x16 sacc, pacc;
#pragma unroll
        for (int i = 0; i < 16; ++i) { sacc[i] = nlse; pacc[i] = 0.f; }
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          const int row = 64 * h64 + 32 * hh + r32;
          sacc = mfma32x32x16(lds_read_b128(buf + DQ_OFF_K, swzt(row, 2 * s + g)), qf[s], sacc);
          pacc = mfma32x32x16(lds_read_b128(buf + DQ_OFF_V, swz256(row, 2 * s + g)), df[s], pacc);
        }
        __builtin_amdgcn_sched_group_barrier(0x100, DQ_LA, 0);
#pragma unroll
        for (int i = 0; i < 16 - DQ_LA; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, DQ_LA, 0);
        bf16x8 sf[2];
        float p[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) p[i] = fast_exp2(sacc[i] * kSl2);
        if (diag) {   // wave-uniform
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const uint32_t key = kb + 32 * hh + 8 * (i >> 2) + 4 * g + (i & 3);
            const bool vis = CAUSAL ? (key <= myq) : (key < Sv);
            if (!vis) p[i] = 0.f;
          }
        }
#pragma unroll
        for (int i = 0; i < 16; ++i) sf[i >> 3][i & 7] = (bf16)(p[i] * (pacc[i] - Dq));
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int dt = 0; dt < 4; ++dt)
            qacc[dt] = mfma32x32x16(
                tr_operand(buf + DQ_OFF_K, 64 * h64 + 32 * hh + 16 * c, 32 * dt, lane), sf[c],
                qacc[dt]);
      }
    }
  }

  if (!rows_ok) return;
  if (ROPE) {   // dQ was taken with respect to rotated queries: turn it back
#pragma unroll
    for (int dt = 0; dt < 2; ++dt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int e = 32 * dt + 8 * (i >> 2) + 4 * g + (i & 3);
        float c, s;
        cos_sin_turns(rope_turn(rope.pos0 + myq, rope_turns_per_pos(e, rope.log2_base)), c, s);
        rope_pair(qacc[dt], qacc[dt + 2], i, c, s, true);
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

hipError_t launch_attn_bwd_dkdv(const bf16* Qc, const bf16* dOc, const float* lse_c, const float* D,
                                const bf16* Kp, const bf16* Vp, float* dK32, float* dV32, bf16* dk,
                                bf16* dv, int64_t kv_row, int64_t kv_head, int64_t S, int64_t Sp,
                                int U, int h0, int G, int causal, hipStream_t st) {
  const int kv_lo = h0 / G, kv_hi = (h0 + U - 1) / G;
  dim3 grid((unsigned)(Sp / 128), (unsigned)(kv_hi - kv_lo + 1));
  if (causal)
    hipLaunchKernelGGL(attn_bwd_dkdv_kernel<true>, grid, dim3(256), 0, st, Qc, dOc, lse_c, D, Kp,
                       Vp, dK32, dV32, dk, dv, S, Sp, U, h0, G, kv_row, kv_head);
  else
    hipLaunchKernelGGL(attn_bwd_dkdv_kernel<false>, grid, dim3(256), 0, st, Qc, dOc, lse_c, D, Kp,
                       Vp, dK32, dV32, dk, dv, S, Sp, U, h0, G, kv_row, kv_head);
  return hipGetLastError();
}

hipError_t launch_attn_bwd_dq(const bf16* Qc, const bf16* dOc, const float* lse_c, const float* D,
                              const bf16* Kp, const bf16* Vp, bf16* dQc, int64_t S, int64_t Sp,
                              int U, int h0, int G, int causal, RopeArgs rope, hipStream_t st) {
  const int nqb = (int)((Sp + DQ_BQ - 1) / DQ_BQ);
  dim3 grid((unsigned)(nqb * U));
#define UPIPE_DQ(C, R)                                                                         \
  hipLaunchKernelGGL((attn_bwd_dq_kernel<C, R>), grid, dim3(512), 0, st, Qc, dOc, lse_c, D, Kp, \
                     Vp, dQc, S, Sp, U, h0, G, nqb, rope)
  if (causal) {
    if (rope.on) UPIPE_DQ(true, true);
    else UPIPE_DQ(true, false);
  } else {
    if (rope.on) UPIPE_DQ(false, true);
    else UPIPE_DQ(false, false);
  }
#undef UPIPE_DQ
  return hipGetLastError();
}

}  // namespace upipe
