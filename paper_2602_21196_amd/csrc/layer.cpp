// Attention-block entry points: projections around the chunked attention.
//
// Forward (paper Section 3.3, Appendix A "Untied Ulysses (forward)"):
//   K, V = x Wk, x Wv                      once (kept for every chunk)
//   per chunk c of U heads:
//     Q_c  = x Wq_c                          QKV projection slice
//     O_c  = attention(Q_c, K, V)           flash forward, lse saved
//     final_out[:, chunk] = O_c              (o_saved)
//     Y32 += O_c Wo_c                        output-projection accumulation
//   y = bf16(Y32)
// Backward (Appendix A "Untied Ulysses (backward)"), with K, V and Q_c
// recomputed from x (activation checkpointing keeps x, final_out, lse):
//   per chunk c:
//     dO_c  = dY Wo_c^T,   D = rowsum(dO_c * O_c)
//     dWo_c = O_c^T dY                       split-K over S, ordered sum
//     Q_c   = x Wq_c                         recompute
//     dK, dV += ...,  dQ_c                   attention backward
//     dX32 += dQ_c Wq_c^T                    full-size fp32 accumulator
//     dWq_c = x^T dQ_c                       split-K over S
//   dX32 += dK Wk^T;  dX32 += dV Wv^T;  dx = bf16(dX32)
//   dWk = x^T dK,  dWv = x^T dV
// Every fp32 accumulator is carried across chunks in one fixed order, so all
// outputs are bitwise identical for every chunk size U.
// Rotary embedding (optional, Section 4 "Implementation"): Q_c and K are
// rotated in the projection epilogue, on the fp32 accumulators, before they
// are rounded and stored -- in place, with no extra pass or fp32 copy.  The
// backward recomputes them the same way and turns dQ_c back by the inverse
// rotation in the dQ kernel's final write, and dK in one in-place pass after
// the last chunk.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/upipe.h"
#include "api_internal.h"
#include "gemm.h"
#include "kernels.h"

namespace upipe {

namespace {

constexpr int64_t kSplitTarget = 32;   // weight-gradient split count target

int check_layer_shape(int64_t S, int d_model, int Hq, int Hkv, int d, int U) {
  int rc = check_attn_shape(S, Hq, Hkv, d, U);
  if (rc != UPIPE_OK) return rc;
  if (d_model < 1) return UPIPE_ERR_INVALID_ARG;
  if (d_model % 128 != 0) return UPIPE_ERR_UNSUPPORTED;
  if (d_model > 65536) return UPIPE_ERR_UNSUPPORTED;
  if (round_up(S, SEQ_PAD) * (int64_t)d_model >= (int64_t(1) << 40)) return UPIPE_ERR_UNSUPPORTED;
  return UPIPE_OK;
}

// Split length of the sequence for weight gradients: a function of S only
// (never of U), a multiple of the GEMM k-step.
int64_t wgrad_split_len(int64_t S) {
  int64_t len = round_up((S + kSplitTarget - 1) / kSplitTarget, 256);
  return len < 256 ? 256 : len;
}

struct LayerFwdPlan {
  int64_t Sp = 0;
  size_t Kp = 0, Vp = 0, Qc = 0, Oc = 0, Y32 = 0, total = 0;
  bool y32 = false;
};

struct LayerBwdPlan {
  int64_t Sp = 0, split_len = 0;
  int splits = 0;
  AttnBwdPlan attn;            // offsets relative to `attn_base`
  size_t attn_base = 0, dX32 = 0, dKb = 0, dVb = 0, partial = 0, total = 0;
};

LayerFwdPlan plan_layer_fwd(int64_t S, int d_model, int Hq, int Hkv, int U) {
  LayerFwdPlan p;
  p.Sp = round_up(S, SEQ_PAD);
  const size_t head = (size_t)p.Sp * HEAD_DIM * 2;
  Carver c;
  p.Kp = c.take(Hkv * head);
  p.Vp = c.take(Hkv * head);
  p.Qc = c.take(U * head);
  p.Oc = c.take(U * head);
  p.y32 = Hq / U > 1;
  if (p.y32) p.Y32 = c.take((size_t)S * d_model * 4);
  p.total = c.used;
  return p;
}

LayerBwdPlan plan_layer_bwd(int64_t S, int d_model, int Hq, int Hkv, int U) {
  LayerBwdPlan p;
  p.Sp = round_up(S, SEQ_PAD);
  p.split_len = wgrad_split_len(S);
  p.splits = (int)((S + p.split_len - 1) / p.split_len);
  p.attn = plan_attn_bwd(S, Hq, Hkv, U);
  Carver c;
  p.attn_base = c.take(p.attn.total);
  p.dX32 = c.take((size_t)S * d_model * 4);
  p.dKb = c.take((size_t)S * Hkv * HEAD_DIM * 2);
  p.dVb = c.take((size_t)S * Hkv * HEAD_DIM * 2);
  const int64_t widest = (U > Hkv ? U : Hkv) * (int64_t)HEAD_DIM;
  p.partial = c.take((size_t)p.splits * d_model * widest * 4);
  p.total = c.used;
  return p;
}

// Head-major outputs; `rope` rotates the heads of group 0 (Q, or K of K|V).
GemmEpilogue heads_epi(bf16* n0, bf16* n1, int64_t n_split, int64_t Sp,
                       RopeArgs rope = RopeArgs{}) {
  GemmEpilogue e{};
  e.dst_norm[0] = n0;
  e.dst_norm[1] = n1;
  e.n_split = n_split;
  e.Sp = Sp;
  e.rope = rope;
  e.rope_groups = rope.on ? 1 : 0;
  return e;
}

GemmEpilogue acc_epi(float* c32, int64_t ldc, bf16* out, int64_t ldo, int64_t m_store, bool first,
                     bool last) {
  GemmEpilogue e{};
  e.c32 = c32;
  e.ldc = ldc;
  e.out = out;
  e.ldo = ldo;
  e.m_store = m_store;
  e.first = first;
  e.last = last;
  return e;
}

// C = A . B over the whole k range in one piece.
hipError_t gemm1(const GemmOperand& A, bool ak, const GemmOperand& B, bool bk, GemmEpilogue E,
                 int epi, int64_t M, int64_t N, int64_t K, hipStream_t st) {
  E.k_total = K;
  return launch_gemm(A, ak, B, bk, E, epi, M, N, 0, round_up(K, 128), 1, st);
}

}  // namespace

int run_layer_fwd(const bf16* x, const bf16* wqkv, const bf16* wo, bf16* y, bf16* o_saved,
                  float* lse, int64_t S, int dm, int Hq, int Hkv, int U, RopeArgs rope,
                  char* ws, hipStream_t st) {
  const LayerFwdPlan p = plan_layer_fwd(S, dm, Hq, Hkv, U);
  const int64_t Sp = p.Sp, ldw = (int64_t)(Hq + 2 * Hkv) * HEAD_DIM;
  bf16* Kp = (bf16*)(ws + p.Kp);
  bf16* Vp = (bf16*)(ws + p.Vp);
  bf16* Qc = (bf16*)(ws + p.Qc);
  bf16* Oc = (bf16*)(ws + p.Oc);
  float* Y32 = p.y32 ? (float*)(ws + p.Y32) : nullptr;
  const int G = Hq / Hkv;
  const GemmOperand X = operand(x, dm, S, dm);
  // K | V = x [Wk | Wv], both head-major.
  UPIPE_LAUNCH(kGemm, st,
               gemm1(X, true, operand(wqkv + (int64_t)Hq * HEAD_DIM, ldw, 2 * Hkv * HEAD_DIM, dm),
                     false, heads_epi(Kp, Vp, Hkv, Sp, rope), GEMM_EPI_HEADS, Sp,
                     2 * Hkv * HEAD_DIM, dm, st));
  const int nu = Hq / U;
  for (int c = 0; c < nu; ++c) {
    const int h0 = c * U;
    UPIPE_LAUNCH(kGemm, st,
                 gemm1(X, true, operand(wqkv + (int64_t)h0 * HEAD_DIM, ldw, U * HEAD_DIM, dm),
                       false, heads_epi(Qc, nullptr, U, Sp, rope), GEMM_EPI_HEADS, Sp,
                       U * HEAD_DIM, dm, st));
    UPIPE_LAUNCH(kAttnFwd, st, launch_attn_fwd(Qc, Kp, Vp, Oc, lse, S, Sp, S, Sp, 0, U, h0, G, 1, st));
    UPIPE_LAUNCH(kUnpackRows, st, launch_unpack_rows(Oc, S, Hq, h0, U, Sp, o_saved, st));
    // Y32 (+)= O_c Wo_c; O_c read head-major, Wo rows [h0*d, (h0+U)*d).
    UPIPE_LAUNCH(kGemm, st,
                 gemm1(operand(Oc, HEAD_DIM, S, U * HEAD_DIM, HEAD_DIM, Sp * HEAD_DIM), true,
                       operand(wo + (int64_t)h0 * HEAD_DIM * dm, dm, dm, U * HEAD_DIM), false,
                       acc_epi(Y32, dm, y, dm, S, c == 0, c == nu - 1), GEMM_EPI_ACC32, Sp, dm,
                       U * HEAD_DIM, st));
  }
  return UPIPE_OK;
}

int run_layer_bwd(const bf16* x, const bf16* wqkv, const bf16* wo, const bf16* o_saved,
                  const float* lse, const bf16* dy, bf16* dx, bf16* dwqkv, bf16* dwo, int64_t S,
                  int dm, int Hq, int Hkv, int U, RopeArgs rope, char* ws, hipStream_t st) {
  const LayerBwdPlan p = plan_layer_bwd(S, dm, Hq, Hkv, U);
  const AttnBwdPlan& a = p.attn;
  char* ab = ws + p.attn_base;
  const int64_t Sp = p.Sp, ldw = (int64_t)(Hq + 2 * Hkv) * HEAD_DIM;
  bf16* Kp = (bf16*)(ab + a.Kp);
  bf16* Vp = (bf16*)(ab + a.Vp);
  float* dK32 = a.carry ? (float*)(ab + a.dK32) : nullptr;
  float* dV32 = a.carry ? (float*)(ab + a.dV32) : nullptr;
  bf16* Qc = (bf16*)(ab + a.Qc);
  bf16* dOc = (bf16*)(ab + a.dOc);
  bf16* dQc = (bf16*)(ab + a.dQc);
  float* D = (float*)(ab + a.D);
  float* lse_c = (float*)(ab + a.lse_c);
  float* dX32 = (float*)(ws + p.dX32);
  bf16* dKb = (bf16*)(ws + p.dKb);
  bf16* dVb = (bf16*)(ws + p.dVb);
  float* partial = (float*)(ws + p.partial);
  const int G = Hq / Hkv;
  const int64_t kvw = (int64_t)Hkv * HEAD_DIM;
  const GemmOperand X = operand(x, dm, S, dm);
  const GemmOperand XT = operand(x, dm, dm, S);        // MN-major view: (m = col, k = s)
  const GemmOperand dY = operand(dy, dm, S, dm);
  const GemmOperand dYn = operand(dy, dm, dm, S);      // MN-major view: (n = col, k = s)

  // Weight gradient C[M][N] = A^T-ish product over the sequence, split into
  // fixed pieces and summed in order into out[m * ldo + col0 + n].
  auto wgrad = [&](const GemmOperand& A, const GemmOperand& B, int64_t M, int64_t N, bf16* out,
                   int64_t ldo, int64_t col0) -> int {
    GemmEpilogue e{};
    e.partial = partial;
    e.k_total = S;
    UPIPE_LAUNCH(kGemmWgrad, st,
                 launch_gemm(A, false, B, false, e, GEMM_EPI_PARTIAL, M, N, 0, p.split_len,
                             p.splits, st));
    UPIPE_LAUNCH(kReduceSplitk, st,
                 launch_reduce_splitk(partial, p.splits, M, N, out, ldo, col0, st));
    return UPIPE_OK;
  };

  // Recompute K and V (head-major).
  UPIPE_LAUNCH(kGemm, st,
               gemm1(X, true, operand(wqkv + (int64_t)Hq * HEAD_DIM, ldw, 2 * kvw, dm), false,
                     heads_epi(Kp, Vp, Hkv, Sp, rope), GEMM_EPI_HEADS, Sp, 2 * kvw, dm,
                     st));
  const int nu = Hq / U;
  for (int c = 0; c < nu; ++c) {
    const int h0 = c * U;
    const int64_t w = (int64_t)U * HEAD_DIM;
    // dO_c = dY Wo_c^T (Wo rows of the chunk are k-contiguous).
    UPIPE_LAUNCH(kGemm, st,
                 gemm1(dY, true, operand(wo + (int64_t)h0 * HEAD_DIM * dm, dm, w, dm), true,
                       heads_epi(dOc, nullptr, U, Sp), GEMM_EPI_HEADS, Sp, w, dm,
                       st));
    UPIPE_LAUNCH(kRowdotLse, st,
                 launch_rowdot_lse(dOc, HEAD_DIM, Sp * HEAD_DIM, o_saved + (int64_t)h0 * HEAD_DIM,
                                   (int64_t)Hq * HEAD_DIM, HEAD_DIM, lse, S, h0, U, Sp, D, lse_c,
                                   st));
    // dWo_c = O_c^T dY: rows (u, e) of the chunk, columns d_model.
    int rc = wgrad(operand(o_saved + (int64_t)h0 * HEAD_DIM, (int64_t)Hq * HEAD_DIM, w, S), dYn,
                   w, dm, dwo + (int64_t)h0 * HEAD_DIM * dm, dm, 0);
    if (rc != UPIPE_OK) return rc;
    // Q_c recomputed, head-major.
    UPIPE_LAUNCH(kGemm, st,
                 gemm1(X, true, operand(wqkv + (int64_t)h0 * HEAD_DIM, ldw, w, dm), false,
                       heads_epi(Qc, nullptr, U, Sp, rope), GEMM_EPI_HEADS, Sp, w, dm,
                       st));
    UPIPE_LAUNCH(kAttnBwdDkdv, st,
                 launch_attn_bwd_dkdv(Qc, dOc, lse_c, D, Kp, Vp, dK32, dV32, dKb, dVb, S, Sp, U,
                                      h0, G, Hkv, 1, st));
    UPIPE_LAUNCH(kAttnBwdDq, st,
                 launch_attn_bwd_dq(Qc, dOc, lse_c, D, Kp, Vp, dQc, S, Sp, U, h0, G, 1, rope, st));
    // dX32 (+)= dQ_c Wq_c^T (Wqkv rows are k-contiguous in the chunk's columns).
    UPIPE_LAUNCH(kGemm, st,
                 gemm1(operand(dQc, HEAD_DIM, S, w, HEAD_DIM, Sp * HEAD_DIM), true,
                       operand(wqkv + (int64_t)h0 * HEAD_DIM, ldw, dm, w), true,
                       acc_epi(dX32, dm, dx, dm, S, c == 0, false), GEMM_EPI_ACC32, Sp, dm, w,
                       st));
    // dWq_c = x^T dQ_c.
    rc = wgrad(XT, operand(dQc, HEAD_DIM, w, S, HEAD_DIM, Sp * HEAD_DIM), dm, w, dwqkv, ldw,
               (int64_t)h0 * HEAD_DIM);
    if (rc != UPIPE_OK) return rc;
  }
  // dK is the gradient with respect to the rotated keys: turn it back, in
  // place (one bf16 pass over [S, Hkv, d]; kept out of the dK/dV kernel,
  // whose register allocation is at its limit).
  if (rope.on) UPIPE_LAUNCH(kRope, st, launch_rope(dKb, S, Hkv, rope, 1, st));
  // dX32 += dK Wk^T, then dX32 += dV Wv^T and round to dx.
  UPIPE_LAUNCH(kGemm, st,
               gemm1(operand(dKb, kvw, S, kvw), true,
                     operand(wqkv + (int64_t)Hq * HEAD_DIM, ldw, dm, kvw), true,
                     acc_epi(dX32, dm, dx, dm, S, false, false), GEMM_EPI_ACC32, Sp, dm, kvw, st));
  UPIPE_LAUNCH(kGemm, st,
               gemm1(operand(dVb, kvw, S, kvw), true,
                     operand(wqkv + (int64_t)(Hq + Hkv) * HEAD_DIM, ldw, dm, kvw), true,
                     acc_epi(dX32, dm, dx, dm, S, false, true), GEMM_EPI_ACC32, Sp, dm, kvw, st));
  // dWk = x^T dK, dWv = x^T dV.
  int rc = wgrad(XT, operand(dKb, kvw, kvw, S), dm, kvw, dwqkv, ldw, (int64_t)Hq * HEAD_DIM);
  if (rc != UPIPE_OK) return rc;
  rc = wgrad(XT, operand(dVb, kvw, kvw, S), dm, kvw, dwqkv, ldw, (int64_t)(Hq + Hkv) * HEAD_DIM);
  return rc;
}

}  // namespace upipe

using namespace upipe;

extern "C" {

size_t upipe_layer_fwd_workspace_size(int64_t S, int d_model, int Hq, int Hkv, int d, int U) {
  if (check_layer_shape(S, d_model, Hq, Hkv, d, U) != UPIPE_OK) return 0;
  return plan_layer_fwd(S, d_model, Hq, Hkv, U).total;
}

size_t upipe_layer_bwd_workspace_size(int64_t S, int d_model, int Hq, int Hkv, int d, int U) {
  if (check_layer_shape(S, d_model, Hq, Hkv, d, U) != UPIPE_OK) return 0;
  return plan_layer_bwd(S, d_model, Hq, Hkv, U).total;
}

int upipe_layer_fwd(const void* x, const void* wqkv, const void* wo, void* y, void* o_saved,
                    float* lse_saved, int64_t S, int d_model, int Hq, int Hkv, int d, int U,
                    double rope_base, int64_t pos0, void* ws, size_t ws_bytes,
                    hipStream_t stream) {
  try {
    int rc = check_layer_shape(S, d_model, Hq, Hkv, d, U);
    if (rc != UPIPE_OK) return rc;
    RopeArgs rope;
    rc = make_rope(rope_base, pos0, S, &rope);
    if (rc != UPIPE_OK) return rc;
    if (!aligned16(x) || !aligned16(wqkv) || !aligned16(wo) || !aligned16(y) ||
        !aligned16(o_saved) || !aligned16(lse_saved) || !aligned16(ws))
      return UPIPE_ERR_INVALID_ARG;
    if (ws_bytes < plan_layer_fwd(S, d_model, Hq, Hkv, U).total) return UPIPE_ERR_WORKSPACE;
    return run_layer_fwd((const bf16*)x, (const bf16*)wqkv, (const bf16*)wo, (bf16*)y,
                         (bf16*)o_saved, lse_saved, S, d_model, Hq, Hkv, U, rope, (char*)ws,
                         stream);
  } catch (...) {
    return UPIPE_ERR_HIP;
  }
}

int upipe_layer_bwd(const void* x, const void* wqkv, const void* wo, const void* o_saved,
                    const float* lse_saved, const void* dy, void* dx, void* dwqkv, void* dwo,
                    int64_t S, int d_model, int Hq, int Hkv, int d, int U, double rope_base,
                    int64_t pos0, void* ws, size_t ws_bytes, hipStream_t stream) {
  try {
    int rc = check_layer_shape(S, d_model, Hq, Hkv, d, U);
    if (rc != UPIPE_OK) return rc;
    RopeArgs rope;
    rc = make_rope(rope_base, pos0, S, &rope);
    if (rc != UPIPE_OK) return rc;
    if (!aligned16(x) || !aligned16(wqkv) || !aligned16(wo) || !aligned16(o_saved) ||
        !aligned16(lse_saved) || !aligned16(dy) || !aligned16(dx) || !aligned16(dwqkv) ||
        !aligned16(dwo) || !aligned16(ws))
      return UPIPE_ERR_INVALID_ARG;
    if (ws_bytes < plan_layer_bwd(S, d_model, Hq, Hkv, U).total) return UPIPE_ERR_WORKSPACE;
    return run_layer_bwd((const bf16*)x, (const bf16*)wqkv, (const bf16*)wo,
                         (const bf16*)o_saved, lse_saved, (const bf16*)dy, (bf16*)dx,
                         (bf16*)dwqkv, (bf16*)dwo, S, d_model, Hq, Hkv, U, rope, (char*)ws,
                         stream);
  } catch (...) {
    return UPIPE_ERR_HIP;
  }
}

}  // extern "C"
