// Attention-block entry points: projections around the chunked attention.
//
// Forward (paper Section 3.3, Appendix A "Untied Ulysses (forward)"):
//   K, V = x Wk, x Wv                      once (kept for every chunk)
//   per chunk c of U heads:
//     Q_c  = x Wq_c                          QKV projection slice
//     O_c  = attention(Q_c, K, V)           flash forward, lse saved
//     final_out[:, chunk] = O_c              (o_saved)
//   y = final_out Wo                         output projection, once
// Backward (Appendix A "Untied Ulysses (backward)"), with K, V and Q_c
// recomputed from x (activation checkpointing keeps x, final_out, lse):
//   dFO   = dY Wo^T                          gradient of final_out, once,
//                                            head-major, kept for the loop
//   dWo   = final_out^T dY                   split-K over S, ordered sum
//   per chunk c:
//     Q_c   = x Wq_c                         recompute
//     (O_c, lse_c = attention(Q_c, K, V)     full checkpointing only: the
//      dWo_c = O_c^T dY)                     attention output was not kept
//     D     = rowsum(dFO_c * O_c)
//     dK, dV += ...,  dQ_c                   attention backward; dQ_c lands
//                                            in its heads' slots of dQKV
//   dx    = [dQ | dK | dV] Wqkv^T            one product, bf16 out
//   dWqkv = x^T [dQ | dK | dV]               split-K over S
// The per-head results (dQ_c, the fp32 dK/dV carries taken in one fixed head
// order) do not depend on U, and every product over heads runs once, so all
// outputs are bitwise identical for every chunk size U.  On one GPU the
// paper's per-stage accumulation of dX (a d_model-wide buffer updated by
// every stage) becomes one product over the bf16 dQ of all heads, which is
// smaller than that accumulator and reads nothing twice.
// Rotary embedding (optional, Section 4 "Implementation"): Q_c and K are
// rotated in the projection epilogue, on the fp32 accumulators, before they
// are rounded and stored -- in place, with no extra pass or fp32 copy.  The
// backward recomputes them the same way and turns dQ_c back by the inverse
// rotation in the dQ kernel's final write, and dK in one in-place pass after
// the last chunk.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

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
  size_t Kp = 0, Vp = 0, Qc = 0, Oc = 0, total = 0;
};

struct LayerBwdPlan {
  int64_t Sp = 0, split_len = 0;
  int splits = 0;
  bool carry = false;          // a key/value group spans several chunks
  size_t Kp = 0, Vp = 0, dK32 = 0, dV32 = 0, Qc = 0, D = 0, lse_c = 0;
  size_t Oc = 0, lse_r = 0;    // recomputed attention output (full checkpointing)
  size_t dFO = 0, dQKV = 0, partial = 0;
  size_t dWqkv32 = 0, dWo32 = 0;   // weight-gradient sums over a batch of sequences
  size_t total = 0;
};

LayerFwdPlan plan_layer_fwd(int64_t S, int d_model, int Hq, int Hkv, int U) {
  (void)d_model;
  (void)Hq;
  LayerFwdPlan p;
  p.Sp = round_up(S, SEQ_PAD);
  const size_t head = (size_t)p.Sp * HEAD_DIM * 2;
  Carver c;
  p.Kp = c.take(Hkv * head);
  p.Vp = c.take(Hkv * head);
  p.Qc = c.take(U * head);
  p.Oc = c.take(U * head);
  p.total = c.used;
  return p;
}

LayerBwdPlan plan_layer_bwd(int64_t S, int d_model, int Hq, int Hkv, int U) {
  LayerBwdPlan p;
  p.Sp = round_up(S, SEQ_PAD);
  p.split_len = wgrad_split_len(S);
  p.splits = (int)((S + p.split_len - 1) / p.split_len);
  const size_t head = (size_t)p.Sp * HEAD_DIM * 2;
  const size_t row32 = (size_t)p.Sp * 4;
  Carver c;
  p.Kp = c.take(Hkv * head);
  p.Vp = c.take(Hkv * head);
  p.carry = group_split(Hq, Hkv, U);
  if (p.carry) {
    p.dK32 = c.take(Hkv * head * 2);
    p.dV32 = c.take(Hkv * head * 2);
  }
  p.Qc = c.take(U * head);
  p.D = c.take(U * row32);
  p.lse_c = c.take(U * row32);
  p.Oc = c.take(U * head);
  p.lse_r = c.take((size_t)Hq * S * 4);
  p.dFO = c.take(Hq * head);
  p.dQKV = c.take((Hq + 2 * Hkv) * head);
  // Split-K partials of the larger weight gradient: dWqkv [d_model, (Hq +
  // 2Hkv) d] or dWo [Hq d, d_model].
  const int64_t widest = (int64_t)(Hq + 2 * Hkv) * HEAD_DIM;
  p.partial = c.take((size_t)p.splits * d_model * widest * 4);
  p.dWqkv32 = c.take((size_t)d_model * widest * 4);
  p.dWo32 = c.take((size_t)Hq * HEAD_DIM * d_model * 4);
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

// bf16 result rows m < m_store into out[m * ldo + n], no fp32 carry.
GemmEpilogue store_epi(bf16* out, int64_t ldo, int64_t m_store) {
  GemmEpilogue e{};
  e.out = out;
  e.ldo = ldo;
  e.m_store = m_store;
  e.first = 1;
  e.last = 1;
  return e;
}

// C = A . B over the whole k range in one piece.
hipError_t gemm1(const GemmOperand& A, bool ak, const GemmOperand& B, bool bk, GemmEpilogue E,
                 int epi, int64_t M, int64_t N, int64_t K, hipStream_t st) {
  E.k_total = K;
  return launch_gemm(A, ak, B, bk, E, epi, M, N, 0, round_up(K, 128), 1, st);
}

}  // namespace

// One sequence of the batch.
int run_layer_fwd_seq(const bf16* x, const bf16* wqkv, const bf16* wo, bf16* y, bf16* o_saved,
                      float* lse, int64_t S, int dm, int Hq, int Hkv, int U, RopeArgs rope,
                      char* ws, hipStream_t st) {
  const LayerFwdPlan p = plan_layer_fwd(S, dm, Hq, Hkv, U);
  const int64_t Sp = p.Sp, ldw = (int64_t)(Hq + 2 * Hkv) * HEAD_DIM;
  const int64_t qw = (int64_t)Hq * HEAD_DIM;
  bf16* Kp = (bf16*)(ws + p.Kp);
  bf16* Vp = (bf16*)(ws + p.Vp);
  bf16* Qc = (bf16*)(ws + p.Qc);
  bf16* Oc = (bf16*)(ws + p.Oc);
  const int G = Hq / Hkv;
  const GemmOperand X = operand(x, dm, S, dm);
  // K | V = x [Wk | Wv], both head-major.
  UPIPE_LAUNCH(kGemm, st,
               gemm1(X, true, operand(wqkv + qw, ldw, 2 * Hkv * HEAD_DIM, dm),
                     false, heads_epi(Kp, Vp, Hkv, Sp, rope), GEMM_EPI_HEADS, Sp,
                     2 * Hkv * HEAD_DIM, dm, st));
  for (int h0 = 0; h0 < Hq; h0 += U) {
    UPIPE_LAUNCH(kGemm, st,
                 gemm1(X, true, operand(wqkv + (int64_t)h0 * HEAD_DIM, ldw, U * HEAD_DIM, dm),
                       false, heads_epi(Qc, nullptr, U, Sp, rope), GEMM_EPI_HEADS, Sp,
                       U * HEAD_DIM, dm, st));
    UPIPE_LAUNCH(kAttnFwd, st, launch_attn_fwd(Qc, Kp, Vp, Oc, lse, S, Sp, S, Sp, 0, U, h0, G, 1, st));
    UPIPE_LAUNCH(kUnpackRows, st, launch_unpack_rows(Oc, S, Hq, h0, U, Sp, o_saved, st));
  }
  // y = final_out Wo.
  UPIPE_LAUNCH(kGemm, st,
               gemm1(operand(o_saved, qw, S, qw), true, operand(wo, dm, dm, qw), false,
                     store_epi(y, dm, S), GEMM_EPI_ACC32, Sp, dm, qw, st));
  return UPIPE_OK;
}

// One sequence of the batch: dx of the sequence; the weight gradients of
// the sequence are added to the fp32 sums unless `first` and rounded into
// dwqkv, dwo when `last`.
int run_layer_bwd_seq(const bf16* x, const bf16* wqkv, const bf16* wo, const bf16* o_saved,
                      const float* lse, const bf16* dy, bf16* dx, bf16* dwqkv, bf16* dwo,
                      int64_t S, int dm, int Hq, int Hkv, int U, RopeArgs rope, int first,
                      int last, char* ws, hipStream_t st) {
  const LayerBwdPlan p = plan_layer_bwd(S, dm, Hq, Hkv, U);
  const int64_t Sp = p.Sp, ldw = (int64_t)(Hq + 2 * Hkv) * HEAD_DIM;
  const int64_t qw = (int64_t)Hq * HEAD_DIM, kvw = (int64_t)Hkv * HEAD_DIM;
  const int64_t head = Sp * HEAD_DIM;   // elements of one head-major head
  bf16* Kp = (bf16*)(ws + p.Kp);
  bf16* Vp = (bf16*)(ws + p.Vp);
  float* dK32 = p.carry ? (float*)(ws + p.dK32) : nullptr;
  float* dV32 = p.carry ? (float*)(ws + p.dV32) : nullptr;
  bf16* Qc = (bf16*)(ws + p.Qc);
  float* D = (float*)(ws + p.D);
  float* lse_c = (float*)(ws + p.lse_c);
  bf16* Oc = (bf16*)(ws + p.Oc);
  float* lse_r = (float*)(ws + p.lse_r);
  const bool recompute = o_saved == nullptr;   // full checkpointing: no saved output
  bf16* dFO = (bf16*)(ws + p.dFO);
  bf16* dQKV = (bf16*)(ws + p.dQKV);     // heads: dQ 0..Hq-1, dK Hq.., dV Hq+Hkv..
  bf16* dKh = dQKV + (int64_t)Hq * head;
  bf16* dVh = dKh + (int64_t)Hkv * head;
  float* partial = (float*)(ws + p.partial);
  float* dWqkv32 = (float*)(ws + p.dWqkv32);
  float* dWo32 = (float*)(ws + p.dWo32);
  const int G = Hq / Hkv;
  const int64_t nqkv = (int64_t)(Hq + 2 * Hkv) * HEAD_DIM;
  const GemmOperand X = operand(x, dm, S, dm);
  const GemmOperand XT = operand(x, dm, dm, S);        // MN-major view: (m = col, k = s)
  const GemmOperand dY = operand(dy, dm, S, dm);
  const GemmOperand dYn = operand(dy, dm, dm, S);      // MN-major view: (n = col, k = s)

  // Weight gradient C[M][N] = sum over s of A(m, s) B(n, s), split into fixed
  // pieces of the sequence and summed in order (then onto the batch sum
  // acc32 [M][N]) into out[m * ldo + n].
  auto wgrad = [&](const GemmOperand& A, const GemmOperand& B, int64_t M, int64_t N, bf16* out,
                   int64_t ldo, float* acc32) -> int {
    GemmEpilogue e{};
    e.partial = partial;
    e.k_total = S;
    UPIPE_LAUNCH(kGemmWgrad, st,
                 launch_gemm(A, false, B, false, e, GEMM_EPI_PARTIAL, M, N, 0, p.split_len,
                             p.splits, st));
    UPIPE_LAUNCH(kReduceSplitk, st,
                 launch_reduce_splitk(partial, p.splits, M, N, out, ldo, 0, acc32, first, last,
                                      st));
    return UPIPE_OK;
  };

  // Recompute K and V (head-major, K rotated).
  UPIPE_LAUNCH(kGemm, st,
               gemm1(X, true, operand(wqkv + qw, ldw, 2 * kvw, dm), false,
                     heads_epi(Kp, Vp, Hkv, Sp, rope), GEMM_EPI_HEADS, Sp, 2 * kvw, dm, st));
  // dFO = dY Wo^T for every head, head-major (Wo rows are k-contiguous).
  UPIPE_LAUNCH(kGemm, st,
               gemm1(dY, true, operand(wo, dm, qw, dm), true, heads_epi(dFO, nullptr, Hq, Sp),
                     GEMM_EPI_HEADS, Sp, qw, dm, st));
  int rc;
  if (!recompute) {   // dWo = final_out^T dY from the kept final_out
    rc = wgrad(operand(o_saved, qw, qw, S), dYn, qw, dm, dwo, dm, dWo32);
    if (rc != UPIPE_OK) return rc;
  }
  for (int h0 = 0; h0 < Hq; h0 += U) {
    const int64_t w = (int64_t)U * HEAD_DIM;
    bf16* dOc = dFO + (int64_t)h0 * head;
    bf16* dQc = dQKV + (int64_t)h0 * head;
    // Q_c recomputed, head-major, rotated.
    UPIPE_LAUNCH(kGemm, st,
                 gemm1(X, true, operand(wqkv + (int64_t)h0 * HEAD_DIM, ldw, w, dm), false,
                       heads_epi(Qc, nullptr, U, Sp, rope), GEMM_EPI_HEADS, Sp, w, dm, st));
    if (recompute) {
      // The chunk's attention output and lse again (the same kernel on the
      // same operands: bitwise what the forward produced), and its rows of
      // dWo = O_c^T dY.
      UPIPE_LAUNCH(kAttnFwd, st,
                   launch_attn_fwd(Qc, Kp, Vp, Oc, lse_r, S, Sp, S, Sp, 0, U, h0, G, 1, st));
      UPIPE_LAUNCH(kRowdotLse, st,
                   launch_rowdot_lse(dOc, HEAD_DIM, head, Oc, HEAD_DIM, head, lse_r, S, h0, U,
                                     Sp, D, lse_c, st));
      rc = wgrad(operand(Oc, HEAD_DIM, w, S, HEAD_DIM, head), dYn, w, dm,
                 dwo + (int64_t)h0 * HEAD_DIM * dm, dm, dWo32 + (int64_t)h0 * HEAD_DIM * dm);
      if (rc != UPIPE_OK) return rc;
    } else {
      UPIPE_LAUNCH(kRowdotLse, st,
                   launch_rowdot_lse(dOc, HEAD_DIM, head, o_saved + (int64_t)h0 * HEAD_DIM, qw,
                                     HEAD_DIM, lse, S, h0, U, Sp, D, lse_c, st));
    }
    rc = run_dkdv_chunk(Qc, dOc, lse_c, D, Kp, Vp, dK32, dV32, dKh, dVh, HEAD_DIM, head, S, Sp,
                        U, h0, G, 1, st);
    if (rc != UPIPE_OK) return rc;
    UPIPE_LAUNCH(kAttnBwdDq, st,
                 launch_attn_bwd_dq(Qc, dOc, lse_c, D, Kp, Vp, dQc, S, Sp, U, h0, G, 1, rope, st));
  }
  // dK is the gradient with respect to the rotated keys: turn it back, in
  // place (one bf16 pass over [Hkv, S, d]; kept out of the dK/dV kernel,
  // whose register allocation is at its limit).
  if (rope.on)
    UPIPE_LAUNCH(kRope, st, launch_rope(dKh, S, Hkv, HEAD_DIM, head, rope, 1, st));
  // dx = [dQ | dK | dV] Wqkv^T (head-major A; Wqkv rows are k-contiguous).
  UPIPE_LAUNCH(kGemm, st,
               gemm1(operand(dQKV, HEAD_DIM, S, nqkv, HEAD_DIM, head), true,
                     operand(wqkv, ldw, dm, nqkv), true, store_epi(dx, dm, S), GEMM_EPI_ACC32,
                     Sp, dm, nqkv, st));
  // dWqkv = x^T [dQ | dK | dV].
  return wgrad(XT, operand(dQKV, HEAD_DIM, nqkv, S, HEAD_DIM, head), dm, nqkv, dwqkv, ldw,
               dWqkv32);
}

// Batches: the B sequences run one after another through the same
// workspace; only the caller's tensors grow with B.
int run_layer_fwd(const bf16* x, const bf16* wqkv, const bf16* wo, bf16* y, bf16* o_saved,
                  float* lse, int64_t B, int64_t S, int dm, int Hq, int Hkv, int U, RopeArgs rope,
                  char* ws, hipStream_t st) {
  const int64_t xs = S * dm, os = S * Hq * HEAD_DIM, ls = (int64_t)Hq * S;
  for (int64_t b = 0; b < B; ++b) {
    const int rc = run_layer_fwd_seq(x + b * xs, wqkv, wo, y + b * xs, o_saved + b * os,
                                     lse + b * ls, S, dm, Hq, Hkv, U, rope, ws, st);
    if (rc != UPIPE_OK) return rc;
  }
  return UPIPE_OK;
}

int run_layer_bwd(const bf16* x, const bf16* wqkv, const bf16* wo, const bf16* o_saved,
                  const float* lse, const bf16* dy, bf16* dx, bf16* dwqkv, bf16* dwo, int64_t B,
                  int64_t S, int dm, int Hq, int Hkv, int U, RopeArgs rope, char* ws,
                  hipStream_t st) {
  const int64_t xs = S * dm, os = S * Hq * HEAD_DIM, ls = (int64_t)Hq * S;
  const bool kept = o_saved != nullptr;
  for (int64_t b = 0; b < B; ++b) {
    const int rc = run_layer_bwd_seq(x + b * xs, wqkv, wo, kept ? o_saved + b * os : nullptr,
                                     kept ? lse + b * ls : nullptr, dy + b * xs, dx + b * xs,
                                     dwqkv, dwo, S, dm, Hq, Hkv, U, rope, b == 0, b == B - 1, ws,
                                     st);
    if (rc != UPIPE_OK) return rc;
  }
  return UPIPE_OK;
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

int upipe_layer_fwd_ex(const void* x, const void* wqkv, const void* wo, void* y, void* o_saved,
                       float* lse_saved, int64_t B, int64_t S, int d_model, int Hq, int Hkv,
                       int d, int U, double rope_base, int64_t pos0, void* ws,
                       size_t ws_bytes, hipStream_t stream) {
  try {
    int rc = check_layer_shape(S, d_model, Hq, Hkv, d, U);
    if (rc != UPIPE_OK) return rc;
    if (!batch_ok(B, S * std::max<int64_t>(d_model, (int64_t)Hq * HEAD_DIM)))
      return UPIPE_ERR_INVALID_ARG;
    RopeArgs rope;
    rc = make_rope(rope_base, pos0, S, &rope);
    if (rc != UPIPE_OK) return rc;
    if (!aligned16(x) || !aligned16(wqkv) || !aligned16(wo) || !aligned16(y) ||
        !aligned16(o_saved) || !aligned16(lse_saved) || !aligned16(ws))
      return UPIPE_ERR_INVALID_ARG;
    if (ws_bytes < plan_layer_fwd(S, d_model, Hq, Hkv, U).total) return UPIPE_ERR_WORKSPACE;
    return run_layer_fwd((const bf16*)x, (const bf16*)wqkv, (const bf16*)wo, (bf16*)y,
                         (bf16*)o_saved, lse_saved, B, S, d_model, Hq, Hkv, U, rope, (char*)ws,
                         stream);
  } catch (...) {
    return UPIPE_ERR_HIP;
  }
}

int upipe_layer_bwd_ex(const void* x, const void* wqkv, const void* wo, const void* o_saved,
                       const float* lse_saved, const void* dy, void* dx, void* dwqkv,
                       void* dwo, int64_t B, int64_t S, int d_model, int Hq, int Hkv, int d,
                       int U, double rope_base, int64_t pos0, void* ws, size_t ws_bytes,
                       hipStream_t stream) {
  try {
    int rc = check_layer_shape(S, d_model, Hq, Hkv, d, U);
    if (rc != UPIPE_OK) return rc;
    if (!batch_ok(B, S * std::max<int64_t>(d_model, (int64_t)Hq * HEAD_DIM)))
      return UPIPE_ERR_INVALID_ARG;
    RopeArgs rope;
    rc = make_rope(rope_base, pos0, S, &rope);
    if (rc != UPIPE_OK) return rc;
    // o_saved and lse_saved: both given (kept attention output), or both NULL
    // (full checkpointing: recomputed).
    if ((o_saved == nullptr) != (lse_saved == nullptr)) return UPIPE_ERR_INVALID_ARG;
    const bool kept = o_saved != nullptr;
    if (!aligned16(x) || !aligned16(wqkv) || !aligned16(wo) || (kept && !aligned16(o_saved)) ||
        (kept && !aligned16(lse_saved)) || !aligned16(dy) || !aligned16(dx) ||
        !aligned16(dwqkv) || !aligned16(dwo) || !aligned16(ws))
      return UPIPE_ERR_INVALID_ARG;
    if (ws_bytes < plan_layer_bwd(S, d_model, Hq, Hkv, U).total) return UPIPE_ERR_WORKSPACE;
    return run_layer_bwd((const bf16*)x, (const bf16*)wqkv, (const bf16*)wo,
                         (const bf16*)o_saved, lse_saved, (const bf16*)dy, (bf16*)dx,
                         (bf16*)dwqkv, (bf16*)dwo, B, S, d_model, Hq, Hkv, U, rope, (char*)ws,
                         stream);
  } catch (...) {
    return UPIPE_ERR_HIP;
  }
}

int upipe_gemm_bf16(const void* a, const void* b, void* c, int64_t M, int64_t N, int64_t K,
                    hipStream_t stream) {
  try {
    if (M < 1 || N < 1 || K < 1) return UPIPE_ERR_INVALID_ARG;
    if (M % 128 || N % 128 || K % 128) return UPIPE_ERR_UNSUPPORTED;
    if (M > 65536 || N > 65536 || K > 65536) return UPIPE_ERR_UNSUPPORTED;
    if (!aligned16(a) || !aligned16(b) || !aligned16(c)) return UPIPE_ERR_INVALID_ARG;
    // A [M, K] row-major is K-major; B [K, N] row-major is N-major.
    UPIPE_LAUNCH(kGemm, stream,
                 gemm1(operand((const bf16*)a, K, M, K), true, operand((const bf16*)b, N, N, K),
                       false, store_epi((bf16*)c, N, M), GEMM_EPI_ACC32, M, N, K, stream));
    return UPIPE_OK;
  } catch (...) {
    return UPIPE_ERR_HIP;
  }
}

int upipe_layer_fwd(const void* x, const void* wqkv, const void* wo, void* y, void* o_saved,
                    float* lse_saved, int64_t S, int d_model, int Hq, int Hkv, int d, int U,
                    void* ws, size_t ws_bytes, hipStream_t stream) {
  return upipe_layer_fwd_ex(x, wqkv, wo, y, o_saved, lse_saved, 1, S, d_model, Hq, Hkv, d, U,
                            0.0, 0, ws, ws_bytes, stream);
}

int upipe_layer_bwd(const void* x, const void* wqkv, const void* wo, const void* o_saved,
                    const float* lse_saved, const void* dy, void* dx, void* dwqkv, void* dwo,
                    int64_t S, int d_model, int Hq, int Hkv, int d, int U, void* ws,
                    size_t ws_bytes, hipStream_t stream) {
  return upipe_layer_bwd_ex(x, wqkv, wo, o_saved, lse_saved, dy, dx, dwqkv, dwo, 1, S, d_model,
                            Hq, Hkv, d, U, 0.0, 0, ws, ws_bytes, stream);
}

}  // extern "C"
