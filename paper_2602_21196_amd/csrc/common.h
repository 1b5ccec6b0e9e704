// Shared device-side helpers for the gfx950 kernels.
//
// MFMA fragment conventions used throughout (v_mfma_f32_32x32x16_bf16, wave64):
//   A operand: lane l supplies row (l % 32) of the 32x16 A tile and the 8
//              k-values of k-group g = l / 32.
//   B operand: lane l supplies column (l % 32) of the 16x32 B tile and the 8
//              k-values of k-group g.
//   The k-values a lane supplies may be any fixed permutation of the 16 k's
//   as long as A and B use the same one; contractions only need agreement.
//   C/D:       lane l holds column (l % 32); element i of its 16 floats is
//              row 8*(i/4) + 4*g + (i%4).
//
// Transposed operands (V^T, K^T, Q^T, dO^T) are never stored: they are read
// out of the row-major [S][128] tiles in LDS with ds_read_b64_tr_b16 (see
// tr_operand), which hands each lane one column of a 4-row block.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace upipe {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int HEAD_DIM = 128;   // the only supported head width
constexpr int SEQ_PAD = 128;    // sequence padding granule of packed buffers

__host__ __device__ inline int64_t round_up(int64_t x, int64_t m) {
  return (x + m - 1) / m * m;
}

__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) {
  return __builtin_amdgcn_exp2f(x);
}

__device__ __forceinline__ bf16x8 lds_read_b128(const char* base, uint32_t off) {
  return *reinterpret_cast<const bf16x8*>(base + off);
}

__device__ __forceinline__ void lds_write_b128(char* base, uint32_t off, u32x4 v) {
  *reinterpret_cast<u32x4*>(base + off) = v;
}

// Direct global -> LDS copy of 16 bytes per lane (global_load_lds_dwordx4):
// lane L's bytes land at lds_wave_base + 16 * L, where lds_wave_base must be
// the same for the whole wave.  Completion is tracked by vmcnt.
typedef __attribute__((address_space(3))) void lds_void;
__device__ __forceinline__ void dma_b128(const void* g, char* lds_wave_base) {
  __builtin_amdgcn_global_load_lds(g, (lds_void*)lds_wave_base, 16, 0, 0);
}

// Raw buffer resource over `bytes` bytes at `base` (stride 0, gfx9 data
// format word); loads at offsets past `bytes` return zeros instead of faulting.
typedef __amdgpu_buffer_rsrc_t buf_rsrc;
__device__ __forceinline__ buf_rsrc make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// Buffer -> LDS copy of 16 bytes per lane (buffer_load_dwordx4 ... lds): the
// bytes at voff + soff (lane offset + uniform offset) of lane L land at
// lds_wave_base + 16 * L.  No vector ALU work for the address; tracked by vmcnt.
__device__ __forceinline__ void dma_buf_b128(buf_rsrc r, uint32_t voff, uint32_t soff,
                                             char* lds_wave_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)lds_wave_base, 16, voff, soff, 0, 0);
}

// Wait until every outstanding global load of this wave has completed.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x3F70); }

// 16-byte chunk swizzles of 256-B rows (16 chunks).  swz256: chunk c of row
// r at c ^ (r & 15).  swzt: chunk c of row r at c ^ tsw(r), where tsw swaps
// the two 2-bit halves of r mod 16.  Both put the sixteen consecutive rows of
// a plain MFMA operand read (same logical chunk) in sixteen distinct slots;
// swzt also spreads the 8 rows x 4 chunks of a transposing read (tr_operand)
// over every slot exactly twice, the minimum for its 512 bytes.
__device__ __forceinline__ uint32_t swz256(int r, int c) { return r * 256 + ((c ^ (r & 15)) << 4); }
__device__ __forceinline__ uint32_t tsw(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }
__device__ __forceinline__ uint32_t swzt(int r, int c) { return r * 256 + ((c ^ tsw(r)) << 4); }

// MFMA operand whose k index runs down the rows of a row-major [k][n] tile of
// 256-B rows stored with swzt (A and B operands have the same lane layout):
// lane l gets column n0 + (l % 32) at rows k0 + 4g + {0..3} (elements 0..3)
// and k0 + 8 + 4g + {0..3} (elements 4..7), g = l / 32 -- the k order in
// which a lane holds the rows of a C tile (rows 8a + 4g + b), so P and dS
// fragments taken from C tiles pair with it directly.  ds_read_b64_tr_b16:
// within each 16-lane group, loader lane t reads the 8 bytes at row
// k0 + 4g + t/4, columns n0 + 16 * ((l >> 4) & 1) + 4 (t % 4), and receiver
// lane t gets column t of the group's 16 columns for those four rows.
__device__ __forceinline__ bf16x8 tr_operand(const char* tile, int k0, int n0, int lane) {
  typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
  const int t = lane & 15, hi = (lane >> 4) & 1, g = lane >> 5;
  const int col = n0 + 16 * hi + 4 * (t & 3);
  const int r0 = k0 + 4 * g + (t >> 2);
  const uint32_t cb = (uint32_t)(col & 7) << 1;   // byte offset inside the 16-byte chunk
  const bf16x4 lo =
      __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(tile + swzt(r0, col >> 3) + cb));
  const bf16x4 up =
      __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(tile + swzt(r0 + 8, col >> 3) + cb));
  bf16x8 v;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    v[e] = lo[e];
    v[4 + e] = up[e];
  }
  return v;
}

// ---- rotary position embedding (RoFormer), head coordinate pairs (e, e + 64)
// for e < 64: at sequence position p the pair turns by p * theta_e with
// theta_e = base^(-e/64); the inverse (transpose) turns by the opposite angle.
struct RopeArgs {
  double log2_base;   // log2 of the frequency base
  int64_t pos0;       // position of sequence row 0
  int on;             // 0: no rotation
};

// theta_e / (2 pi): turns per position of pair e, in fp64.  Positions reach
// 2^24, so the whole turns of p * theta_e are removed in fp64 before anything
// is rounded to fp32.
__device__ __forceinline__ double rope_turns_per_pos(int e, double log2_base) {
  return exp2(-(double)e * log2_base * (1.0 / 64.0)) * 0.15915494309189535;
}

// Fractional part, in [-1/2, 1/2], of p * f turns.
__device__ __forceinline__ float rope_turn(int64_t p, double f) {
  const double r = (double)p * f;
  return (float)(r - rint(r));
}

// cos(2 pi t), sin(2 pi t): v_cos_f32 / v_sin_f32 take their argument in
// turns; t is first brought into [-1/2, 1/2].
__device__ __forceinline__ void cos_sin_turns(float t, float& c, float& s) {
  t -= rintf(t);
  c = __builtin_amdgcn_cosf(t);
  s = __builtin_amdgcn_sinf(t);
}

// Rotate the pair (a, b) by the angle whose cos / sin are (c, s); `inverse`
// turns the other way.
__device__ __forceinline__ void rope_pair(float& a, float& b, float c, float s, bool inverse) {
  if (inverse) s = -s;
  const float ra = a * c - b * s;
  const float rb = b * c + a * s;
  a = ra;
  b = rb;
}

// The same on element i of two accumulator tiles.
__device__ __forceinline__ void rope_pair(f32x16& a, f32x16& b, int i, float c, float s,
                                          bool inverse) {
  float x = a[i], y = b[i];
  rope_pair(x, y, c, s, inverse);
  a[i] = x;
  b[i] = y;
}

}  // namespace upipe
