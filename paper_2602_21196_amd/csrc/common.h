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
// "MFMA order" of a transposed copy: a buffer stored [d][S] (sequence index
// contiguous) keeps, inside every aligned block of 16 positions, the element
// of sequence index perm16(p) at position p, where perm16 swaps bits 2 and 3.
// Then the 16 floats one lane holds in a C tile (rows 8a+4g+b) become, after
// conversion to bf16, exactly the B/A-operand vectors that read 8 consecutive
// positions 16*kt + 8*g + j of such a buffer.  perm16 is an involution.
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

__host__ __device__ inline int64_t perm16(int64_t p) {
  return (p & ~int64_t(12)) | ((p & 4) << 1) | ((p & 8) >> 1);
}

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

// 16-byte chunk swizzles.  Rows of 256 B (16 chunks): chunk c of row r is
// stored at c ^ (r & 15).  Rows of 128 B (8 chunks): c ^ (r & 7) ^ ((r>>3) & 1).
// Rows of 64 B (4 chunks): c ^ ((r >> 1) & 3).  For the MFMA operand reads
// (consecutive lanes = consecutive rows, same logical chunk) these are free of
// bank conflicts for both 32- and 64-bank LDS.
__device__ __forceinline__ uint32_t swz256(int r, int c) { return r * 256 + ((c ^ (r & 15)) << 4); }
__device__ __forceinline__ uint32_t swz128(int r, int c) {
  return r * 128 + ((c ^ (r & 7) ^ ((r >> 3) & 1)) << 4);
}
__device__ __forceinline__ uint32_t swz64(int r, int c) { return r * 64 + ((c ^ ((r >> 1) & 3)) << 4); }
// Rows of 64 B for 64-bank LDS (measured on gfx950): c ^ ((r >> 2) & 3) puts
// the 16 rows read together in 16 distinct 16-byte bank groups.
__device__ __forceinline__ uint32_t swz64b(int r, int c) { return r * 64 + ((c ^ ((r >> 2) & 3)) << 4); }

}  // namespace upipe
