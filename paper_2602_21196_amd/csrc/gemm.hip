// Projection GEMMs of the attention block on gfx950: C = A . B, bf16 inputs,
// fp32 accumulation on MFMA 32x32x16.
//
// The block needs nine differently laid-out products (QKV projection slice,
// output projection, their data and weight gradients; paper Section 3.3 and
// Appendix A).  No tensor is transposed in HBM.  Every operand tile is staged
// into LDS exactly as it lies in memory -- 128 rows of 256 bytes:
//   K-major operand  (k contiguous)    : rows = m (or n), 128 k per row;
//   MN-major operand (m/n contiguous)  : rows = k, 128 m (or n) per row --
// by buffer->LDS copies (no register staging), and the MFMA fragments are
// read in one common k order, k = 8g + 0..7 within each 16-k step:
//   a K-major operand          : plain 16-byte reads;
//   an MN-major operand        : transposing reads (tr_operand_k8).
// Operands may be split into 128-wide blocks with their own stride (the
// head-major chunk buffers [U][Sp][128]).
//
// Tile: 128 x 128 per workgroup, 4 waves as 2 x 2 of 64 x 32+32 (wave column
// half wn holds columns 32 wn + 64 nt + 0..31, nt = 0, 1: the coordinate pairs
// (e, e + 64) of a 128-wide head sit in one lane, which the rotary embedding
// of the head-major epilogue needs), BK = 128, one 64 KB LDS stage per
// workgroup and two workgroups per CU.  The k loop runs in ascending order with
// one fp32 accumulator chain per output element, so a product split over
// several calls (k ranges accumulated through an fp32 buffer) is bitwise equal
// to a single call over the whole k range.
#include "common.h"
#include "gemm.h"

namespace upipe {

namespace {

constexpr int BM = 128, BN = 128, BKG = 128;
constexpr int TILE_BYTES = 128 * 256;     // 32 KB per operand per stage

// Address of operand element (r, k).
// The block width is a power of two (128, or the unblocked 2^50), so the
// block index and the offset inside it are a shift and a mask.
__device__ __forceinline__ const bf16* elem_ptr(const GemmOperand& o, bool kmajor, int64_t r,
                                                int64_t k) {
  const int sh = __builtin_ctzll((unsigned long long)o.blk);
  const int64_t mask = o.blk - 1;
  if (kmajor) return o.p + (k >> sh) * o.blk_stride + r * o.ld + (k & mask);
  return o.p + (r >> sh) * o.blk_stride + k * o.ld + (r & mask);
}

// Buffer resource over the operand's tile at (r0, k0), bounded by the valid
// rows (K-major: rows r0.. < rows_valid) or valid k (MN-major: k0.. <
// k_valid), so that padding reads as zero.
__device__ __forceinline__ buf_rsrc tile_rsrc(const GemmOperand& o, bool kmajor, int64_t r0,
                                              int64_t k0) {
  const int64_t n_lines = kmajor ? o.rows_valid - r0 : o.k_valid - k0;   // 256-B lines in use
  int64_t bytes = n_lines <= 0 ? 0 : ((n_lines > 128 ? 127 : n_lines - 1) * o.ld + 128) * 2;
  return make_rsrc(elem_ptr(o, kmajor, r0, k0), (uint32_t)bytes);
}

// This wave's share of one operand tile: 8 blocks of 4 lines of 256 B.  The
// lane offsets `off` place line chunk c at LDS chunk c ^ tsw(line).
__device__ __forceinline__ void issue_tile(buf_rsrc r, const uint32_t (&off)[8], char* tile, int w) {
#pragma unroll
  for (int i = 0; i < 8; ++i) dma_buf_b128(r, off[i], 0, tile + (8 * w + i) * 1024);
}

__device__ __forceinline__ void lane_offsets(int64_t ld, int w, int lane, uint32_t (&off)[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int line = 4 * (8 * w + i) + (lane >> 4);
    off[i] = (uint32_t)(line * ld * 2) + (((lane & 15) ^ tsw(line)) << 4);
  }
}

// MN-major operand fragment: the 32 columns r0.. of a [k][128] tile at
// k-step ks, lane l getting column r0 + (l % 32) at k = 16 ks + 8g + 0..7
// (g = l / 32) -- eight consecutive k, so that a K-major partner reads the
// same k as one plain 16-byte chunk.  (The attention kernels' tr_operand
// takes k = 4g + 0..3, 8 + 4g + 0..3 instead, the row order of an MFMA
// result tile; here both operands come from LDS and only have to agree.)
// Two ds_read_b64_tr_b16 per lane: within each 16-lane group, loader lane t
// reads the 8 bytes at row 16 ks + 8g + t/4 (+ 4 for the second read),
// columns r0 + 16 ((l >> 4) & 1) + 4 (t % 4); with the swzt swizzle the
// 8 rows x 4 chunks of one read fill every bank exactly twice.
__device__ __forceinline__ bf16x8 tr_operand_k8(const char* tile, int ks, int r0, int lane) {
  typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
  const int t = lane & 15, hi = (lane >> 4) & 1, g = lane >> 5;
  const int col = r0 + 16 * hi + 4 * (t & 3);
  const int row = 16 * ks + 8 * g + (t >> 2);
  const uint32_t cb = (uint32_t)(col & 7) << 1;   // byte offset inside the 16-byte chunk
  const bf16x4 lo =
      __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(tile + swzt(row, col >> 3) + cb));
  const bf16x4 up =
      __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(tile + swzt(row + 4, col >> 3) + cb));
  bf16x8 v;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    v[e] = lo[e];
    v[4 + e] = up[e];
  }
  return v;
}

// Fragment of the 32 rows (m or n) r0.. at k-step ks (16 k) of one tile, in
// the k order k = 16 ks + 8g + 0..7 shared by both modes:
//   KM: K-major tile, one plain 16-byte read (chunk 2 ks + g of the row)
//   MN: MN-major tile, transposing reads (tr_operand_k8)
// The plain reads of 32 rows x 2 chunks touch each bank once per 16 lanes.
enum { KM = 0, MN = 1 };
template <int MODE>
__device__ __forceinline__ bf16x8 frag(const char* tile, int r0, int ks, int lane) {
  const int r32 = lane & 31, g = lane >> 5;
  if (MODE == KM) return lds_read_b128(tile, swzt(r0 + r32, 2 * ks + g));
  return tr_operand_k8(tile, ks, r0, lane);
}

// One stage of LDS (64 KB) per workgroup, so that two workgroups share a CU:
// the copies of one overlap the products of the other.  Measured on the
// Llama layer share against a double-buffered single workgroup per CU: the
// projection products 14.4 -> 10.9 ms, the weight gradients 5.7 -> 3.0 ms per
// step (one stage in flight per workgroup left the copy latency exposed).
template <int EPI>
struct GemmStages {
  static constexpr int N = 1;
};

template <bool A_K, bool B_K, int EPI>
__global__ __launch_bounds__(256, 3 - GemmStages<EPI>::N) void gemm_kernel(
    GemmOperand A, GemmOperand B, GemmEpilogue E, int64_t M, int64_t N, int64_t k_begin,
    int64_t k_len) {
  constexpr int AM = A_K ? KM : MN;
  constexpr int BMODE = B_K ? KM : MN;
  constexpr int NST = GemmStages<EPI>::N;
  __shared__ __attribute__((aligned(1024))) char smem[NST * 2 * TILE_BYTES];
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const int r32 = lane & 31, g = lane >> 5;
  const int wm = w >> 1, wn = w & 1;
  const int64_t tiles_n = N / BN;
  // Workgroups are dispatched round-robin over the 8 XCDs, each with its own
  // L2; which tile a workgroup computes is a permutation chosen per product
  // (the results do not depend on it):
  //   HEADS   (long k, a few weight columns): every XCD takes a contiguous
  //           run of tiles, m-major, so the activation rows are fetched once;
  //   PARTIAL (split-K weight gradients): every XCD takes whole splits, and
  //           walks a split along its shorter side first (the tiles that
  //           share the wider operand's block run together);
  //   ACC32   (short k, many weight columns): round-robin, so each XCD keeps
  //           an eighth of the weight columns in its L2.
  int64_t tile = blockIdx.x, split = blockIdx.y;
  if (EPI != GEMM_EPI_ACC32) {
    const int64_t nx = gridDim.x;
    const int64_t d = (int64_t)blockIdx.y * nx + blockIdx.x;   // dispatch order
    const int64_t nwg = nx * gridDim.y, xcd = d % 8, slot = d / 8;
    const int64_t per = nwg / 8, rem = nwg % 8;
    const int64_t L = xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
    tile = L % nx;
    split = L / nx;
    const int64_t tiles_m = M / BM;
    if (EPI == GEMM_EPI_PARTIAL && tiles_m < tiles_n)   // m fastest
      tile = (tile % tiles_m) * tiles_n + tile / tiles_m;
  }
  const int64_t m0 = (tile / tiles_n) * BM, n0 = (tile % tiles_n) * BN;
  const int64_t kb0 = k_begin + split * k_len;
  int64_t kend = kb0 + k_len;
  if (kend > k_begin + E.k_total) kend = k_begin + E.k_total;
  const int nk = kend > kb0 ? (int)((kend - kb0 + BKG - 1) / BKG) : 0;

  f32x16 acc[2][2];
  if (EPI == GEMM_EPI_ACC32 && !E.first) {
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        const int64_t n = n0 + 32 * wn + 64 * nt + r32;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int64_t m = m0 + 64 * wm + 32 * mt + 8 * (i >> 2) + 4 * g + (i & 3);
          acc[mt][nt][i] = m < E.m_store ? E.c32[m * E.ldc + n] : 0.f;
        }
      }
  } else {
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[mt][nt][i] = 0.f;
  }

  uint32_t offa[8], offb[8];
  lane_offsets(A.ld, w, lane, offa);
  lane_offsets(B.ld, w, lane, offb);
  auto issue = [&](int kk) {
    const int64_t k0 = kb0 + (int64_t)kk * BKG;
    char* buf = smem + (kk % NST) * 2 * TILE_BYTES;
    issue_tile(tile_rsrc(A, A_K, m0, k0), offa, buf, w);
    issue_tile(tile_rsrc(B, B_K, n0, k0), offb, buf + TILE_BYTES, w);
  };
  if (nk > 0) issue(0);
  for (int kk = 0; kk < nk; ++kk) {
    const char* bufA = smem + (kk % NST) * 2 * TILE_BYTES;
    const char* bufB = bufA + TILE_BYTES;
    if (NST == 1 && kk > 0) {
      __syncthreads();   // every wave is done with stage kk-1
      issue(kk);
    }
    wait_vmem();
    __syncthreads();   // stage kk landed for all waves; stage kk-1's buffer is free
    if (NST == 2 && kk + 1 < nk) issue(kk + 1);
#pragma unroll
    for (int ks = 0; ks < BKG / 16; ++ks) {
      bf16x8 af[2], bfr[2];
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) af[mt] = frag<AM>(bufA, 64 * wm + 32 * mt, ks, lane);
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) bfr[nt] = frag<BMODE>(bufB, 32 * wn + 64 * nt, ks, lane);
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) acc[mt][nt] = mfma32x32x16(af[mt], bfr[nt], acc[mt][nt]);
    }
  }

  // ---- epilogues.  Lane holds column n = n0 + 32wn + 64nt + r32 and rows
  //      m = m0 + 64wm + 32mt + 8a + 4g + b for element i = 4a + b.
  if (EPI == GEMM_EPI_HEADS && E.rope.on &&
      ((E.rope_groups >> (n0 / 128 < E.n_split ? 0 : 1)) & 1)) {
    // Pair (e, e + 64), e = 32wn + r32, of rows m: acc[mt][0][i], acc[mt][1][i].
    // The turn of the first row of each 32-row block is reduced in fp64; the
    // offsets 8a + b (< 28) add at most 28 theta_e / 2 pi turns in fp32.
    const double f = rope_turns_per_pos(32 * wn + r32, E.rope.log2_base);
    const float ff = (float)f;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      const float t0 = rope_turn(E.rope.pos0 + m0 + 64 * wm + 32 * mt + 4 * g, f);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        float c, s;
        cos_sin_turns(fmaf((float)(8 * (i >> 2) + (i & 3)), ff, t0), c, s);
        rope_pair(acc[mt][0], acc[mt][1], i, c, s, false);
      }
    }
  }
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      const int64_t n = n0 + 32 * wn + 64 * nt + r32;
      const int64_t mb = m0 + 64 * wm + 32 * mt;
      if (EPI == GEMM_EPI_HEADS) {
        const int64_t nb = n / 128, e = n % 128;
        const int grp = nb < E.n_split ? 0 : 1;
        const int64_t head = nb - (grp ? E.n_split : 0);
        bf16* dn = E.dst_norm[grp];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int64_t m = mb + 8 * (i >> 2) + 4 * g + (i & 3);
          dn[(head * E.Sp + m) * 128 + e] = (bf16)acc[mt][nt][i];
        }
      } else if (EPI == GEMM_EPI_ACC32) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int64_t m = mb + 8 * (i >> 2) + 4 * g + (i & 3);
          if (m < E.m_store) {
            if (E.last) E.out[m * E.ldo + n] = (bf16)acc[mt][nt][i];
            else E.c32[m * E.ldc + n] = acc[mt][nt][i];
          }
        }
      } else {  // GEMM_EPI_PARTIAL
        float* P = E.partial + split * M * N;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int64_t m = mb + 8 * (i >> 2) + 4 * g + (i & 3);
          P[m * N + n] = acc[mt][nt][i];
        }
      }
    }
}

// t = sum over splits s = 0.. of partial[s][m][n], summed in ascending s,
// then added to acc32[m][n] unless `first`; the total goes to acc32 unless
// `last`, else to out[m * ldo + col0 + n] as bf16.
__global__ __launch_bounds__(256) void reduce_splitk_kernel(const float* __restrict__ partial,
                                                            int splits, int64_t M, int64_t N,
                                                            bf16* __restrict__ out, int64_t ldo,
                                                            int64_t col0, float* __restrict__ acc32,
                                                            int first, int last) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= M * N) return;
  float s = 0.f;
  for (int k = 0; k < splits; ++k) s += partial[(int64_t)k * M * N + idx];
  if (!first) s = acc32[idx] + s;
  if (last) {
    const int64_t m = idx / N, n = idx % N;
    out[m * ldo + col0 + n] = (bf16)s;
  } else {
    acc32[idx] = s;
  }
}

template <bool A_K, bool B_K, int EPI>
hipError_t launch_t(const GemmOperand& A, const GemmOperand& B, const GemmEpilogue& E, int64_t M,
                    int64_t N, int64_t k_begin, int64_t k_len, int splits, hipStream_t st) {
  dim3 grid((unsigned)((M / BM) * (N / BN)), (unsigned)splits);
  hipLaunchKernelGGL((gemm_kernel<A_K, B_K, EPI>), grid, dim3(256), 0, st, A, B, E, M, N,
                     k_begin, k_len);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(const GemmOperand& A, bool a_kmajor, const GemmOperand& B, bool b_kmajor,
                       const GemmEpilogue& E, int epi, int64_t M, int64_t N, int64_t k_begin,
                       int64_t k_len, int splits, hipStream_t st) {
  // A K-major tile reads 128 consecutive k of each row: the k range must be
  // made of whole tiles (an MN-major operand is bounded by its buffer
  // resource instead); pieces must start on tile boundaries.
  if ((M % BM) || (N % BN) || (k_len % BKG) || (k_begin % BKG)) return hipErrorInvalidValue;
  if ((a_kmajor || b_kmajor) && (E.k_total % BKG)) return hipErrorInvalidValue;
#define UPIPE_GEMM_CASE(AK, BK_, EP)                                               \
  if (a_kmajor == AK && b_kmajor == BK_ && epi == EP)                              \
    return launch_t<AK, BK_, EP>(A, B, E, M, N, k_begin, k_len, splits, st);
  UPIPE_GEMM_CASE(true, false, GEMM_EPI_HEADS)     // X . W slice
  UPIPE_GEMM_CASE(true, false, GEMM_EPI_ACC32)     // O_c . Wo_c
  UPIPE_GEMM_CASE(true, true, GEMM_EPI_HEADS)      // dY . Wo_c^T
  UPIPE_GEMM_CASE(true, true, GEMM_EPI_ACC32)      // dQ_c . Wq_c^T, dK . Wk^T
  UPIPE_GEMM_CASE(false, false, GEMM_EPI_PARTIAL)  // X^T . dQ_c, O^T . dY
#undef UPIPE_GEMM_CASE
  return hipErrorInvalidValue;
}

hipError_t launch_reduce_splitk(const float* partial, int splits, int64_t M, int64_t N, bf16* out,
                                int64_t ldo, int64_t col0, float* acc32, int first, int last,
                                hipStream_t st) {
  const int64_t n = M * N;
  hipLaunchKernelGGL(reduce_splitk_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                     partial, splits, M, N, out, ldo, col0, acc32, first, last);
  return hipGetLastError();
}

}  // namespace upipe
