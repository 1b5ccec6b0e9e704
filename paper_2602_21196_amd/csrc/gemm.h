// Descriptors and launchers of the projection GEMMs (gemm.hip).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <stdexcept>

#include "common.h"

namespace upipe {

// One operand of C[m][n] = sum_k A[m][k] B[k][n], seen as [row][k] where row
// is m for A and n for B.  Element (r, k) lives at
//   K-major : p + (k / blk) * blk_stride + r * ld + (k % blk)
//   MN-major: p + (r / blk) * blk_stride + k * ld + (r % blk)
// Rows >= rows_valid and k >= k_valid read as zero.  blk = 128 describes the
// head-major chunk buffers [U][Sp][128]; an unblocked operand uses a block
// larger than any index and blk_stride = 0.  blk must be a power of two (the
// kernel splits an index with a shift and a mask).
struct GemmOperand {
  const bf16* p;
  int64_t ld;
  int64_t blk;
  int64_t blk_stride;
  int64_t rows_valid;
  int64_t k_valid;
};

constexpr int64_t kNoBlock = int64_t(1) << 50;

inline GemmOperand operand(const bf16* p, int64_t ld, int64_t rows_valid, int64_t k_valid,
                           int64_t blk = kNoBlock, int64_t blk_stride = 0) {
  static_assert((kNoBlock & (kNoBlock - 1)) == 0, "kNoBlock must be a power of two");
  if (blk <= 0 || (blk & (blk - 1)) != 0) throw std::invalid_argument("GEMM block width");
  return GemmOperand{p, ld, blk, blk_stride, rows_valid, k_valid};
}

enum { GEMM_EPI_HEADS = 0, GEMM_EPI_ACC32 = 1, GEMM_EPI_PARTIAL = 2 };

struct GemmEpilogue {
  // GEMM_EPI_HEADS: output column block nb (128 wide) is head nb of group 0
  // if nb < n_split, else head nb - n_split of group 1; dst_norm[g] is
  // [heads][Sp][128].  Every row m < M is written.
  bf16* dst_norm[2];
  int64_t n_split;
  int64_t Sp;
  // Rotary embedding of the heads of the groups whose bit is set in
  // rope_groups (bit g: group g), row m at position rope.pos0 + m, applied
  // to the fp32 accumulators before rounding.
  RopeArgs rope;
  int rope_groups;
  // GEMM_EPI_ACC32: accumulators start at c32[m][n] (ldc) unless `first`;
  // the result goes to c32 unless `last`, else to out[m][n] (ldo) as bf16.
  // Rows >= m_store are neither read nor written.
  float* c32;
  int64_t ldc;
  bf16* out;
  int64_t ldo;
  int64_t m_store;
  int first;
  int last;
  // GEMM_EPI_PARTIAL: split s of the k range writes partial[s][M][N] fp32.
  float* partial;
  // k extent, counted from k_begin (splits beyond it are clamped).
  int64_t k_total;
};

// M and N must be multiples of 128.  The k range [k_begin, k_begin + k_total)
// is cut into `splits` pieces of k_len; k_begin and k_len are multiples of
// 128, and so is k_total when an operand is K-major (hipErrorInvalidValue
// otherwise).  Supported
// combinations: (A K-major, B MN-major, HEADS | ACC32), (A K-major, B K-major,
// HEADS | ACC32), (A MN-major, B MN-major, PARTIAL).
hipError_t launch_gemm(const GemmOperand& A, bool a_kmajor, const GemmOperand& B, bool b_kmajor,
                       const GemmEpilogue& E, int epi, int64_t M, int64_t N, int64_t k_begin,
                       int64_t k_len, int splits, hipStream_t st);

// t = sum_s partial[s][m][n] in ascending s, plus acc32[m][n] unless first;
// t goes to acc32[m][n] unless last, else out[m * ldo + col0 + n] = bf16(t).
// (first = last = 1 never touches acc32.)
hipError_t launch_reduce_splitk(const float* partial, int splits, int64_t M, int64_t N, bf16* out,
                                int64_t ldo, int64_t col0, float* acc32, int first, int last,
                                hipStream_t st);

}  // namespace upipe
