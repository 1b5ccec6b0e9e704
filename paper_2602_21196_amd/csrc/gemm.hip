// Projection GEMMs of the attention block on gfx950: C = A . B, bf16 inputs,
// fp32 accumulation on MFMA 32x32x16.
//
// The block needs nine differently laid-out products (QKV projection slice,
// output projection, their data and weight gradients; paper Section 3.3 and
// Appendix A).  Instead of transposing tensors in HBM, each operand is
// described by a small descriptor and staged into LDS as [row][k] tiles:
//   K-major operand   (k contiguous in memory)  : 16-byte rows copied as is;
//   MN-major operand  (m or n contiguous)       : 8x8 bf16 blocks loaded as
//     eight 16-byte rows and transposed in registers (v_perm_b32) on the way.
// Operands may be split into 128-wide blocks with their own stride (the
// head-major chunk buffers [U][Sp][128]).
//
// Tile: 128 x 128 per workgroup, 4 waves as 2 x 2 of 64 x 64, BK = 32,
// double-buffered LDS.  The k loop runs in ascending order with one fp32
// accumulator chain per output element, so a product split over several
// calls (k ranges accumulated through an fp32 buffer) is bitwise equal to a
// single call over the whole k range.
#include "common.h"
#include "gemm.h"

namespace upipe {

namespace {

constexpr int BM = 128, BN = 128, BKG = 32;
constexpr int TILE_BYTES = BM * BKG * 2;  // 8 KB per operand per stage

__device__ __forceinline__ uint32_t t_off(int row, int chunk) {
  return row * 64 + ((chunk ^ ((row >> 1) & 3)) << 4);
}

__device__ __forceinline__ const bf16* kmajor_ptr(const GemmOperand& o, int64_t r, int64_t k) {
  return o.p + (k / o.blk) * o.blk_stride + r * o.ld + (k % o.blk);
}
__device__ __forceinline__ const bf16* mnmajor_ptr(const GemmOperand& o, int64_t r, int64_t k) {
  return o.p + (r / o.blk) * o.blk_stride + k * o.ld + (r % o.blk);
}

struct OpRegs {
  u32x4 v[8];
};

// K-major: 512 pieces (128 rows x 4 chunks) per tile, two per thread.
__device__ __forceinline__ void load_kmajor(OpRegs& r, const GemmOperand& o, int64_t r0,
                                            int64_t k0, int t) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int pi = t + 256 * i;
    const int row = pi >> 2, c = pi & 3;
    const int64_t gr = r0 + row, gk = k0 + 8 * c;
    u32x4 val = {0u, 0u, 0u, 0u};
    if (gr < o.rows_valid && gk < o.k_valid)
      val = *reinterpret_cast<const u32x4*>(kmajor_ptr(o, gr, gk));
    r.v[i] = val;
  }
}
__device__ __forceinline__ void store_kmajor(const OpRegs& r, char* buf, int t) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int pi = t + 256 * i;
    lds_write_b128(buf, t_off(pi >> 2, pi & 3), r.v[i]);
  }
}

// MN-major: 64 blocks of 8 (k) x 8 (rows) per tile; threads [base, base+64).
__device__ __forceinline__ void load_mnmajor(OpRegs& r, const GemmOperand& o, int64_t r0,
                                             int64_t k0, int tl) {
  const int kb = tl >> 4, rb = tl & 15;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int64_t gk = k0 + 8 * kb + i, gr = r0 + 8 * rb;
    u32x4 val = {0u, 0u, 0u, 0u};
    if (gk < o.k_valid && gr < o.rows_valid)
      val = *reinterpret_cast<const u32x4*>(mnmajor_ptr(o, gr, gk));
    r.v[i] = val;
  }
}
// In: v[i] = row-block (8 rows) at k = 8kb+i.  Out: LDS row 8rb+m gets the
// 8 k-values of that row as one 16-byte chunk.
__device__ __forceinline__ void store_mnmajor(const OpRegs& r, char* buf, int tl) {
  const int kb = tl >> 4, rb = tl & 15;
#pragma unroll
  for (int m = 0; m < 8; ++m) {
    const int p = m >> 1;
    const uint32_t sel = (m & 1) ? 0x07060302u : 0x05040100u;
    u32x4 out;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      out[j] = __builtin_amdgcn_perm(r.v[2 * j + 1][p], r.v[2 * j][p], sel);
    lds_write_b128(buf, t_off(8 * rb + m, kb), out);
  }
}

template <bool A_K, bool B_K>
struct Loader {
  OpRegs a, b;
  __device__ __forceinline__ void load(const GemmOperand& A, const GemmOperand& B, int64_t m0,
                                       int64_t n0, int64_t k0, int t) {
    if (A_K) load_kmajor(a, A, m0, k0, t);
    else if (t < 64) load_mnmajor(a, A, m0, k0, t);
    if (B_K) load_kmajor(b, B, n0, k0, t);
    else if (t >= 64 && t < 128) load_mnmajor(b, B, n0, k0, t - 64);
  }
  __device__ __forceinline__ void store(char* bufA, char* bufB, int t) {
    if (A_K) store_kmajor(a, bufA, t);
    else if (t < 64) store_mnmajor(a, bufA, t);
    if (B_K) store_kmajor(b, bufB, t);
    else if (t >= 64 && t < 128) store_mnmajor(b, bufB, t - 64);
  }
};

template <bool A_K, bool B_K, int EPI>
__global__ __launch_bounds__(256, 2) void gemm_kernel(GemmOperand A, GemmOperand B, GemmEpilogue E,
                                                      int64_t M, int64_t N, int64_t k_begin,
                                                      int64_t k_len) {
  __shared__ __attribute__((aligned(16))) char smem[4 * TILE_BYTES];
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  const int r32 = lane & 31, g = lane >> 5;
  const int wm = w >> 1, wn = w & 1;
  const int64_t tiles_n = N / BN;
  const int64_t tile = blockIdx.x;
  const int64_t m0 = (tile / tiles_n) * BM, n0 = (tile % tiles_n) * BN;
  const int64_t split = blockIdx.y;
  const int64_t kb0 = k_begin + split * k_len;
  int64_t kend = kb0 + k_len;
  if (kend > k_begin + E.k_total) kend = k_begin + E.k_total;
  const int nk = (int)((kend - kb0 + BKG - 1) / BKG);

  f32x16 acc[2][2];
  if (EPI == GEMM_EPI_ACC32 && !E.first) {
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        const int64_t n = n0 + 64 * wn + 32 * nt + r32;
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

  Loader<A_K, B_K> ld;
  if (nk > 0) {
    ld.load(A, B, m0, n0, kb0, t);
    ld.store(smem, smem + TILE_BYTES, t);
  }
  __syncthreads();
  for (int kk = 0; kk < nk; ++kk) {
    char* bufA = smem + (kk & 1) * 2 * TILE_BYTES;
    char* bufB = bufA + TILE_BYTES;
    const bool more = kk + 1 < nk;
    if (more) ld.load(A, B, m0, n0, kb0 + (int64_t)(kk + 1) * BKG, t);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 af[2], bfr[2];
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
        af[mt] = lds_read_b128(bufA, t_off(64 * wm + 32 * mt + r32, 2 * ks + g));
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
        bfr[nt] = lds_read_b128(bufB, t_off(64 * wn + 32 * nt + r32, 2 * ks + g));
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) acc[mt][nt] = mfma32x32x16(af[mt], bfr[nt], acc[mt][nt]);
    }
    if (more) {
      char* nA = smem + ((kk + 1) & 1) * 2 * TILE_BYTES;
      ld.store(nA, nA + TILE_BYTES, t);
    }
    __syncthreads();
  }

  // ---- epilogues.  Lane holds column n = n0 + 64wn + 32nt + r32 and rows
  //      m = m0 + 64wm + 32mt + 8a + 4g + b for element i = 4a + b.
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      const int64_t n = n0 + 64 * wn + 32 * nt + r32;
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

// out[m * ldo + col0 + n] = bf16(sum over splits s = 0.. of partial[s][m][n]),
// summed in ascending s.
__global__ __launch_bounds__(256) void reduce_splitk_kernel(const float* __restrict__ partial,
                                                            int splits, int64_t M, int64_t N,
                                                            bf16* __restrict__ out, int64_t ldo,
                                                            int64_t col0) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= M * N) return;
  float s = 0.f;
  for (int k = 0; k < splits; ++k) s += partial[(int64_t)k * M * N + idx];
  const int64_t m = idx / N, n = idx % N;
  out[m * ldo + col0 + n] = (bf16)s;
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
                                int64_t ldo, int64_t col0, hipStream_t st) {
  const int64_t n = M * N;
  hipLaunchKernelGGL(reduce_splitk_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                     partial, splits, M, N, out, ldo, col0);
  return hipGetLastError();
}

}  // namespace upipe
