// Layout kernels: the one-GPU stand-ins for UPipe's all-to-all buffers.
//
// In the paper (Section 3.3, Appendix A) each stage's query/key/value heads
// arrive through inp_all_to_all into head-distributed buffers [S, U/C, d],
// and the stage output leaves through out_all_to_all into its slot of the
// preallocated `final_out`.  On one GPU these become:
//   pack   token-major [S, H, d] (chosen heads)  ->  head-major [n, Sp, d]
//   unpack head-major [n, Sp, d]                 ->  token-major [S, H, d]
// Rows S..Sp-1 of packed buffers are zero, so the attention kernels never
// test sequence bounds on loads.  All kernels are HBM-bound copies.
#include "common.h"
#include "kernels.h"

namespace upipe {

// One workgroup packs a 64-row slab of one head; 256 threads, each moving
// four 16-byte pieces.
__global__ __launch_bounds__(256) void pack_rows_kernel(
    const bf16* __restrict__ src, int64_t S, int H, int h0, int64_t Sp, bf16* __restrict__ dst) {
  const int t = threadIdx.x;
  const int hh = blockIdx.y;
  const int64_t s0 = (int64_t)blockIdx.x * 64;
  const int h = h0 + hh;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int pi = t + 256 * r;
    const int row = pi >> 4, chunk = pi & 15;
    const int64_t s = s0 + row;
    u32x4 val = {0u, 0u, 0u, 0u};
    if (s < S)
      val = *reinterpret_cast<const u32x4*>(src + (s * H + h) * HEAD_DIM + chunk * 8);
    *reinterpret_cast<u32x4*>(dst + ((int64_t)hh * Sp + s) * HEAD_DIM + chunk * 8) = val;
  }
}

// Copies rows [0, S) of head-major [n, Sp, d] into heads h0.. of [S, H, d].
__global__ __launch_bounds__(256) void unpack_rows_kernel(
    const bf16* __restrict__ src, int64_t S, int H, int h0, int n, int64_t Sp,
    bf16* __restrict__ dst) {
  const int64_t pieces = S * n * 16;
  for (int64_t pi = (int64_t)blockIdx.x * 256 + threadIdx.x; pi < pieces;
       pi += (int64_t)gridDim.x * 256) {
    const int chunk = pi & 15;
    const int64_t rest = pi >> 4;
    const int hh = rest % n;
    const int64_t s = rest / n;
    const u32x4 val = *reinterpret_cast<const u32x4*>(
        src + ((int64_t)hh * Sp + s) * HEAD_DIM + chunk * 8);
    *reinterpret_cast<u32x4*>(dst + (s * H + h0 + hh) * HEAD_DIM + chunk * 8) = val;
  }
}

// D[hh][s] = sum_e dO(s, hh, e) * O(s, hh, e) in fp32 (the backward's row
// term) and the chunk's log-sum-exp rows times -sqrt(d) (the initial value
// of the backward kernels' score accumulators: they end at
// q.k - sqrt(d) lse, so P = exp2(acc log2(e) / sqrt(d))), copied to a padded
// buffer.  Element
// (s, hh, e) of an operand X lives at X + s * x_row + hh * x_head + e.  One
// wave per (row, head); lanes hold two elements each and reduce by shuffles.
__global__ __launch_bounds__(256) void rowdot_lse_kernel(
    const bf16* __restrict__ a, int64_t a_row, int64_t a_head,
    const bf16* __restrict__ b, int64_t b_row, int64_t b_head,
    const float* __restrict__ lse, int64_t S, int h0, int n, int64_t Sp,
    float* __restrict__ D, float* __restrict__ lse_c) {
  const int lane = threadIdx.x & 63;
  const int64_t task = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (task >= (int64_t)n * Sp) return;
  const int hh = task / Sp;
  const int64_t s = task % Sp;
  float acc = 0.f, l = 0.f;
  if (s < S) {
    const bf16* pa = a + s * a_row + hh * a_head + 2 * lane;
    const bf16* pb = b + s * b_row + hh * b_head + 2 * lane;
    acc = (float)pa[0] * (float)pb[0] + (float)pa[1] * (float)pb[1];
    l = lse[(int64_t)(h0 + hh) * S + s] * -11.313708498984761f;   // -sqrt(128) lse
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
  if (lane == 0) {
    D[(int64_t)hh * Sp + s] = acc;
    lse_c[(int64_t)hh * Sp + s] = l;
  }
}

// Fold a partial softmax result over a disjoint key set (one ring step) into
// the running one, per row (s, h) of o [S, H, d] and lse [H, S]:
//   lse' = log(e^lse + e^lse_p),  o' = e^(lse - lse') o + e^(lse_p - lse') o_p,
// with -inf marking an empty key set.  Sixteen lanes (16 bytes each) hold one
// row; all of a row's lanes sit in one wave, and the new lse is computed from
// the loaded values, so every lane has read the row's lse before any writes it.
__global__ __launch_bounds__(256) void lse_merge_kernel(bf16* __restrict__ o, float* __restrict__ lse,
                                                        const bf16* __restrict__ o_p,
                                                        const float* __restrict__ lse_p, int64_t S,
                                                        int H) {
  const int64_t rows = S * H;
  const int c = threadIdx.x & 15;
  for (int64_t r = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 4; r < rows;
       r += (int64_t)gridDim.x * 16) {
    const int64_t s = r / H;
    const int h = (int)(r % H);
    const int64_t li = (int64_t)h * S + s;
    const float la = lse[li], lb = lse_p[li];
    const float m = fmaxf(la, lb);
    float wa = 0.f, wb = 0.f, lnew = -INFINITY;
    if (m != -INFINITY) {
      wa = la == -INFINITY ? 0.f : __expf(la - m);
      wb = lb == -INFINITY ? 0.f : __expf(lb - m);
      const float tot = wa + wb;
      lnew = m + __logf(tot);
      wa /= tot;
      wb /= tot;
    }
    const int64_t off = r * HEAD_DIM + 8 * c;
    const bf16x8 a = *reinterpret_cast<const bf16x8*>(o + off);
    const bf16x8 b = *reinterpret_cast<const bf16x8*>(o_p + off);
    bf16x8 out;
#pragma unroll
    for (int e = 0; e < 8; ++e) out[e] = (bf16)(wa * (float)a[e] + wb * (float)b[e]);
    *reinterpret_cast<bf16x8*>(o + off) = out;
    if (c == 0) lse[li] = lnew;
  }
}

hipError_t launch_lse_merge(bf16* o, float* lse, const bf16* o_p, const float* lse_p, int64_t S,
                            int H, hipStream_t st) {
  const int64_t blocks = (S * H + 15) / 16;
  hipLaunchKernelGGL(lse_merge_kernel, dim3((unsigned)(blocks < (1 << 20) ? blocks : (1 << 20))),
                     dim3(256), 0, st, o, lse, o_p, lse_p, S, H);
  return hipGetLastError();
}

// In-place rotary embedding of H heads of S rows (the standalone form for
// callers that project Q and K themselves, and the dK pass of the layer
// backward; the layer's forward fuses it into the projection).
// Thread = (row s, slice j of 8 pairs e = 8j..8j+7): the slice's frequencies
// are formed once per thread, its 8 angles once per row, and every head of
// the row is turned with them.  HBM-bound: one read and one write of x.
__global__ __launch_bounds__(256) void rope_kernel(bf16* __restrict__ x, int64_t S, int H,
                                                   int64_t row_stride, int64_t head_stride,
                                                   RopeArgs rope, int inverse) {
  const int j = threadIdx.x & 7;
  double f[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) f[e] = rope_turns_per_pos(8 * j + e, rope.log2_base);
  const int64_t step = (int64_t)gridDim.x * 32;
  for (int64_t s = (int64_t)blockIdx.x * 32 + (threadIdx.x >> 3); s < S; s += step) {
    float c[8], sn[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) cos_sin_turns(rope_turn(rope.pos0 + s, f[e]), c[e], sn[e]);
    bf16* row = x + s * row_stride + 8 * j;
    for (int h = 0; h < H; ++h) {
      bf16x8* pa = reinterpret_cast<bf16x8*>(row + h * head_stride);
      bf16x8* pb = reinterpret_cast<bf16x8*>(row + h * head_stride + 64);
      bf16x8 a = *pa, b = *pb;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float xa = (float)a[e], xb = (float)b[e];
        rope_pair(xa, xb, c[e], sn[e], inverse != 0);
        a[e] = (bf16)xa;
        b[e] = (bf16)xb;
      }
      *pa = a;
      *pb = b;
    }
  }
}

hipError_t launch_rope(bf16* x, int64_t S, int H, int64_t row, int64_t head, RopeArgs rope,
                       int inverse, hipStream_t st) {
  const int64_t blocks = (S + 31) / 32;
  hipLaunchKernelGGL(rope_kernel, dim3((unsigned)(blocks < 8192 ? blocks : 8192)), dim3(256), 0,
                     st, x, S, H, row, head, rope, inverse);
  return hipGetLastError();
}

hipError_t launch_pack_rows(const bf16* src, int64_t S, int H, int h0, int n,
                            int64_t Sp, bf16* dst, hipStream_t st) {
  dim3 grid((unsigned)(Sp / 64), (unsigned)n);
  hipLaunchKernelGGL(pack_rows_kernel, grid, dim3(256), 0, st, src, S, H, h0, Sp, dst);
  return hipGetLastError();
}

hipError_t launch_unpack_rows(const bf16* src, int64_t S, int H, int h0, int n,
                              int64_t Sp, bf16* dst, hipStream_t st) {
  const int64_t pieces = S * n * 16;
  int64_t blocks = (pieces + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(unpack_rows_kernel, dim3((unsigned)blocks), dim3(256), 0,
                     st, src, S, H, h0, n, Sp, dst);
  return hipGetLastError();
}

hipError_t launch_rowdot_lse(const bf16* a, int64_t a_row, int64_t a_head,
                             const bf16* b, int64_t b_row, int64_t b_head,
                             const float* lse, int64_t S, int h0, int n,
                             int64_t Sp, float* D, float* lse_c,
                             hipStream_t st) {
  const int64_t tasks = (int64_t)n * Sp;
  hipLaunchKernelGGL(rowdot_lse_kernel, dim3((unsigned)((tasks + 3) / 4)),
                     dim3(256), 0, st, a, a_row, a_head, b, b_row, b_head, lse,
                     S, h0, n, Sp, D, lse_c);
  return hipGetLastError();
}

}  // namespace upipe
