// Host-side launchers of the gfx950 kernels.  Every launcher enqueues on the
// given stream and returns the launch status; shapes are validated by the
// caller (api.cpp) before any of these run.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace upipe {

// ---- layout (layout.hip) -------------------------------------------------
// src [S, H, d] heads h0..h0+n-1  ->  dst [n, Sp, d]; rows >= S are zero.
hipError_t launch_pack_rows(const bf16* src, int64_t S, int H, int h0, int n,
                            int64_t Sp, bf16* dst, hipStream_t st);
// src [n, Sp, d] rows < S  ->  dst [S, H, d] heads h0..h0+n-1.
hipError_t launch_unpack_rows(const bf16* src, int64_t S, int H, int h0, int n,
                              int64_t Sp, bf16* dst, hipStream_t st);
// D[n, Sp] = rowsum(a * b) over the head width and lse_c[n, Sp] = -sqrt(d)
// times the lse rows h0.. of the caller's [Hq, S] array (zero for rows >= S).  Element
// (s, hh, e) of a is a[s * a_row + hh * a_head + e], likewise for b.
hipError_t launch_rowdot_lse(const bf16* a, int64_t a_row, int64_t a_head,
                             const bf16* b, int64_t b_row, int64_t b_head,
                             const float* lse, int64_t S, int h0, int n,
                             int64_t Sp, float* D, float* lse_c,
                             hipStream_t st);

// ---- attention forward (attn_fwd.hip) ------------------------------------
// Qc [U, Sqp, d], Kp and Vp [Hkv, Skvp, d] -> Oc [U, Sqp, d] and lse rows
// h0..h0+U-1 of the caller's [Hq, Sq] array.  Query row i sees key j iff
// j < Skv and (not causal or j <= i + delta); rows that see no key get O = 0,
// lse = -inf.  Self-attention: Sq = Skv = S, delta = 0.
hipError_t launch_attn_fwd(const bf16* Qc, const bf16* Kp, const bf16* Vp,
                           bf16* Oc, float* lse, int64_t Sq, int64_t Sqp,
                           int64_t Skv, int64_t Skvp, int64_t delta, int U,
                           int h0, int G, int causal, hipStream_t st);
// The same with the key range of every query block cut into `ns` splits of
// equal stage counts, split s writing O to Oc + s U Sqp d ([ns][U][Sqp][d])
// and lse row (lse_h0 + s U + u) of leading dimension lse_ld, rows i <
// lse_rows (the plain call: ns = 1, lse_h0 = h0, lse_ld = lse_rows = Sq).
hipError_t launch_attn_fwd_split(const bf16* Qc, const bf16* Kp, const bf16* Vp, bf16* Oc,
                                 float* lse, int64_t Sq, int64_t Sqp, int64_t Skv, int64_t Skvp,
                                 int64_t delta, int U, int h0, int G, int causal, int ns,
                                 int lse_h0, int64_t lse_ld, int64_t lse_rows, hipStream_t st);
// Number of key splits the forward uses for these padded lengths (1 or 2).
int attn_fwd_key_splits(int64_t Sqp, int64_t Skvp);
// In place, per row (s, h) of o [S, H, d] and lse [H, S]: fold the partial
// result (o_p, lse_p) over a disjoint key set into (o, lse).
hipError_t launch_lse_merge(bf16* o, float* lse, const bf16* o_p,
                            const float* lse_p, int64_t S, int H,
                            hipStream_t st);

// ---- attention backward (attn_bwd.hip) -----------------------------------
// lse_c below holds -sqrt(d) lse, the initial value of a row's score
// accumulator (the kernels evaluate P = exp2(acc log2(e) / sqrt(d))).
// Key/value gradients of the chunk's heads, accumulated in fp32 on top of
// dK32/dV32 [Hkv, Sp, d] (read unless the chunk holds a group's first head;
// dK32 carries the unscaled sum with its sign flipped, -sum dS^T Q), written
// back there, or -- when the chunk holds the group's last head --
// scaled and rounded into dk/dv bf16: row s of key/value head g at element
// s * kv_row + g * kv_head (token-major [S, Hkv, d]: kv_row = Hkv * d,
// kv_head = d; head-major [Hkv, Sp, d]: kv_row = d, kv_head = Sp * d).
hipError_t launch_attn_bwd_dkdv(const bf16* Qc, const bf16* dOc,
                                const float* lse_c, const float* D,
                                const bf16* Kp, const bf16* Vp, float* dK32,
                                float* dV32, bf16* dk, bf16* dv, int64_t kv_row,
                                int64_t kv_head, int64_t S, int64_t Sp, int U,
                                int h0, int G, int causal, hipStream_t st);
// dQc [U, Sp, d] of the chunk's heads.  With rope.on, Q and K are the rotated
// ones and dQ is turned back by the inverse rotation of its row before it is
// rounded.
hipError_t launch_attn_bwd_dq(const bf16* Qc, const bf16* dOc,
                              const float* lse_c, const float* D,
                              const bf16* Kp, const bf16* Vp, bf16* dQc, int64_t S, int64_t Sp, int U, int h0,
                              int G, int causal, RopeArgs rope, hipStream_t st);
// In place: rotate every head h < H of row s < S, the 128 values at element
// s * row + h * head of x, at position pos0 + s (inverse: by the opposite
// angle).  Token-major [S, H, d]: row = H * d, head = d.
hipError_t launch_rope(bf16* x, int64_t S, int H, int64_t row, int64_t head,
                       RopeArgs rope, int inverse, hipStream_t st);

}  // namespace upipe
