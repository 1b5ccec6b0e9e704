/*
 * upipe.h -- C ABI of the MI355X (gfx950) head-chunked causal GQA attention
 * library: the per-GPU hot path of UPipe ("Untied Ulysses", arXiv 2602.21196).
 *
 * After the Ulysses re-layout (paper Section 3.1) one GPU holds the full
 * sequence S for its share of heads: Hq query heads and Hkv key/value heads,
 * head width d.  UPipe (Section 3.3) runs the attention block over those heads
 * in nu = Hq/U chunks of U heads, reusing one chunk-sized set of buffers for
 * every chunk, so activation scratch grows with U rather than with Hq.  Query
 * head h reads key/value head h / (Hq/Hkv) (grouped-query attention, Section
 * 2.1; chunks follow the GQA schedule of Section 4.1, which on one device is
 * ascending local head order).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Element types: bf16 tensors are raw IEEE bfloat16 (2 bytes), fp32 is
 *    IEEE binary32.  All tensors are dense, contiguous, row-major, with the
 *    shapes stated per call, and 16-byte aligned.
 *  - Pointers: all tensor and workspace pointers are DEVICE pointers owned by
 *    the caller.  The library never allocates, frees or synchronises device
 *    memory in the compute entry points; every kernel is enqueued on the
 *    caller's `stream`, and the calls return as soon as the work is queued.
 *  - Workspace: each compute call takes a caller-allocated device workspace of
 *    at least the size returned by its *_workspace_size query.  It holds the
 *    chunk-sized buffers that are reused for every chunk plus the buffers
 *    that live for the whole call; its contents on entry are ignored.
 *  - Outputs are overwritten, never accumulated into.
 *  - Scale: scores are q.k / sqrt(d) (Section 2.1); there is no scale knob.
 *  - Causal: key j is visible to query i iff j <= i.  causal = 0 gives full
 *    (bidirectional) attention over all S keys.
 *  - Determinism: for fixed shapes every output is bitwise identical across
 *    calls and across every valid U (one fixed reduction order: query heads
 *    ascending, then query tiles descending; fp32 partial sums are carried
 *    between chunks through the workspace; whether the forward splits a
 *    query block's key range in two depends on the lengths only).
 *  - Errors: arguments are validated on the host before anything is
 *    enqueued; a failing call enqueues nothing and returns a negative
 *    upipe_status.  A launch failure returns UPIPE_ERR_HIP (work queued
 *    before it stays queued).  Faults inside kernels surface at the caller's
 *    next synchronisation.  No C++ exception crosses this interface.
 *  - Supported shapes: d == 128; S >= 1 (any length: rows past the last tile
 *    are padded inside the workspace); 1 <= Hkv <= Hq, Hkv | Hq; 1 <= U,
 *    U | Hq; Hq <= 64; S * max(Hq, d_model/128) * d < 2^40.  The batched
 *    calls need B >= 1 and B times one sequence's largest tensor below
 *    2^61 elements (UPIPE_ERR_INVALID_ARG otherwise).
 *  - Thread safety: calls are reentrant across host threads and streams as
 *    long as each concurrent call has its own workspace and outputs.  The
 *    profiling switch below is process-global and not thread-safe.
 */
#ifndef UPIPE_H
#define UPIPE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  UPIPE_OK = 0,
  UPIPE_ERR_INVALID_ARG = -1, /* bad size, null/misaligned pointer, U or Hkv
                                 not dividing Hq, workspace too small      */
  UPIPE_ERR_UNSUPPORTED = -2, /* valid in principle, not built: d != 128,
                                 d_model % 128 != 0, Hq > 64, S rounded up
                                 to a multiple of 128 above 2^24 - 128      */
  UPIPE_ERR_WORKSPACE = -3,   /* ws_bytes below the size query's result     */
  UPIPE_ERR_HIP = -4          /* a HIP runtime call or launch failed        */
} upipe_status;

/* Human-readable name of a status code (static storage, never NULL). */
const char* upipe_status_string(int status);

/* Library ABI version: major*10000 + minor*100 + patch. */
int upipe_version(void);

/* ------------------------------------------------------------------------
 * Head schedule (paper Section 4.1 "Grouped-Query Attention Scheduling",
 * Section 3.3 stage count nu = H/U).  Pure host computation.
 *
 * Global view with H query heads, Hkv key/value heads, C devices and U heads
 * per stage (U a multiple of C, C | H, C | Hkv, U | H).  Device p owns query
 * heads [p H/C, (p+1) H/C) and key/value heads [p Hkv/C, (p+1) Hkv/C).
 * Stage s processes, on every device, the next U/C of its heads in ascending
 * order, so a key/value head is sent only at the first stage that reads it.
 *
 *   stage_heads: host array of H ints; on return stage_heads[s*U + j] is the
 *                j-th global query head of stage s, listed device by device.
 *   kv_stage:    host array of Hkv ints; kv_stage[g] is the stage at which
 *                key/value head g is first sent.
 * Returns UPIPE_OK or UPIPE_ERR_INVALID_ARG (nothing written then).
 * ---------------------------------------------------------------------- */
int upipe_gqa_schedule(int H, int Hkv, int C, int U, int* stage_heads,
                       int* kv_stage);

/* ------------------------------------------------------------------------
 * Workspace size queries.  Return the byte count the matching compute call
 * needs for these shapes, or 0 if the shapes are invalid or unsupported.
 * The size is  fixed(S, Hkv[, d_model]) + U * per_head(S)  (chunk buffers).
 * It does not depend on the batch size B: the calls that take a batch of B
 * sequences run them one after another through the same workspace.  The
 * attention calls keep no key/value copy when Hkv == 1 and S % 128 == 0.
 * ---------------------------------------------------------------------- */
size_t upipe_attn_fwd_workspace_size(int64_t S, int Hq, int Hkv, int d, int U);
size_t upipe_attn_bwd_workspace_size(int64_t S, int Hq, int Hkv, int d, int U);
size_t upipe_layer_fwd_workspace_size(int64_t S, int d_model, int Hq, int Hkv,
                                      int d, int U);
size_t upipe_layer_bwd_workspace_size(int64_t S, int d_model, int Hq, int Hkv,
                                      int d, int U);

/* ------------------------------------------------------------------------
 * Attention forward, head chunk by head chunk (Section 2.1 definition,
 * Section 3.3 chunking, Appendix A "Untied Ulysses (forward)").
 *
 *   q   bf16 [S, Hq, d]    queries, token-major (the Ulysses layout)
 *   k   bf16 [S, Hkv, d]   keys
 *   v   bf16 [S, Hkv, d]   values
 *   o   bf16 [S, Hq, d]    out: softmax(q k^T / sqrt d) v per head
 *   lse fp32 [Hq, S]       out: natural-log log-sum-exp of each row's scaled
 *                          scores (saved for the backward)
 * For each chunk c the U heads [cU, (c+1)U) are packed to a head-major chunk
 * buffer (the stand-in for the input all-to-all's destination), attended, and
 * unpacked into o (the output all-to-all's target, `final_out`).  With one
 * key/value head and S a multiple of 128, k and v already have the
 * head-major layout and are read in place (no copy in the workspace).
 * ---------------------------------------------------------------------- */
int upipe_attn_fwd(const void* q, const void* k, const void* v, void* o,
                   float* lse, int64_t S, int Hq, int Hkv, int d, int causal,
                   int U, void* ws, size_t ws_bytes, hipStream_t stream);

/* The same for a batch of B >= 1 independent sequences of length S (the
 * paper's batch-size ablation, Appendix "Batch Size Ablation", spends the
 * memory UPipe saves on B > 1): q, o [B, S, Hq, d], k, v [B, S, Hkv, d],
 * lse [B, Hq, S].  The sequences run one after another through the same
 * workspace, whose size does not depend on B.  B = 1 is upipe_attn_fwd. */
int upipe_attn_fwd_batch(const void* q, const void* k, const void* v, void* o,
                         float* lse, int64_t B, int64_t S, int Hq, int Hkv, int d,
                         int causal, int U, void* ws, size_t ws_bytes,
                         hipStream_t stream);

/* ------------------------------------------------------------------------
 * upipe_attn_fwd for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments, layouts, results and errors as upipe_attn_fwd, without
 * the workspace: the library uses a scratch array of its own, a static
 * device array of upipe_attn_fwd_noalloc_scratch_bytes() bytes (64 MiB) that
 * each GPU the library runs on holds until the process ends.  Shapes whose
 * upipe_attn_fwd_workspace_size exceeds it return UPIPE_ERR_WORKSPACE (with
 * one key/value head and U = 1: S up to 131072 when S % 128 == 0, about
 * 65500 otherwise).  The call
 * allocates nothing; its first call on a device looks up that device's
 * copy of the array.  The stream must belong to the current device
 * (UPIPE_ERR_INVALID_ARG otherwise).  Every
 * call on one GPU shares that GPU's array: calls that overlap on one GPU
 * (concurrent streams or host threads) race and must be serialised by the
 * caller.  Nothing in the array needs clearing between calls.
 * ---------------------------------------------------------------------- */
size_t upipe_attn_fwd_noalloc_scratch_bytes(void);
int upipe_attn_fwd_noalloc(const void* q, const void* k, const void* v, void* o,
                           float* lse, int64_t S, int Hq, int Hkv, int d, int causal,
                           int U, hipStream_t stream);

/* ------------------------------------------------------------------------
 * One ring step of context-parallel attention (Section 2.2, Ring Attention
 * with online softmax; Section 4, the Ulysses + Ring hybrid of USP that
 * UPipe extends): attention of a query block against one key/value block
 * that sits elsewhere in the sequence, returning the partial result that
 * upipe_lse_merge folds into the running one.
 *
 *   q   bf16 [Sq, Hq, d]    queries at global positions q_offset + i
 *   k   bf16 [Skv, Hkv, d]  keys at global positions kv_offset + j
 *   v   bf16 [Skv, Hkv, d]  values
 *   o   bf16 [Sq, Hq, d]    out: softmax-weighted values over the visible keys
 *   lse fp32 [Hq, Sq]       out: natural-log log-sum-exp of the visible scaled
 *                           scores
 * With causal = 1, key j is visible to query i iff kv_offset + j <=
 * q_offset + i; with causal = 0 every key is.  A row that sees no key gets
 * o = 0 and lse = -inf (the empty set, neutral for the merge).  Head chunking
 * by U as for upipe_attn_fwd; with Sq = Skv and q_offset = kv_offset this is
 * upipe_attn_fwd.  |offsets| <= 2^62 and q_offset - kv_offset < 2^63
 * (UPIPE_ERR_INVALID_ARG otherwise); workspace from
 * upipe_attn_fwd_ring_workspace_size (0 for invalid shapes).
 * ---------------------------------------------------------------------- */
size_t upipe_attn_fwd_ring_workspace_size(int64_t Sq, int64_t Skv, int Hq, int Hkv,
                                          int d, int U);
int upipe_attn_fwd_ring(const void* q, const void* k, const void* v, void* o,
                        float* lse, int64_t Sq, int64_t Skv, int64_t q_offset,
                        int64_t kv_offset, int Hq, int Hkv, int d, int causal,
                        int U, void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Merge of two partial attention results over disjoint key sets (the
 * online-softmax combination of successive ring steps, Section 2.2), in
 * place on the running result:
 *   lse' = log(exp(lse) + exp(lse_part))
 *   o'   = exp(lse - lse') o + exp(lse_part - lse') o_part
 * per row (s, h).  o, o_part bf16 [S, H, d]; lse, lse_part fp32 [H, S];
 * lse = -inf marks an empty set.  Needs no workspace; d = 128.  Callers must
 * not overlap o with o_part (or lse with lse_part).
 * ---------------------------------------------------------------------- */
int upipe_lse_merge(void* o, float* lse, const void* o_part, const float* lse_part,
                    int64_t S, int H, int d, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Attention backward (analytic gradient of the Section 2.1 definition,
 * Appendix A "Untied Ulysses (backward)": per-stage dQ, per-group dK/dV
 * accumulators that persist across stages).
 *
 *   q, k, v, o, lse  as produced/consumed by upipe_attn_fwd (same S)
 *   dout bf16 [S, Hq, d]   upstream gradient of o
 *   dq   bf16 [S, Hq, d]   out
 *   dk   bf16 [S, Hkv, d]  out: summed over each group's query heads
 *   dv   bf16 [S, Hkv, d]  out
 * `lse` must come from upipe_attn_fwd on the same q, k, v (it is used to
 * rebuild the probabilities without a second softmax pass).
 * ---------------------------------------------------------------------- */
int upipe_attn_bwd(const void* q, const void* k, const void* v, const void* o,
                   const float* lse, const void* dout, void* dq, void* dk,
                   void* dv, int64_t S, int Hq, int Hkv, int d, int causal,
                   int U, void* ws, size_t ws_bytes, hipStream_t stream);

/* The same for a batch of B >= 1 sequences (Appendix "Batch Size
 * Ablation"), layouts as for upipe_attn_fwd_batch with dout, dq like q and
 * dk, dv like k.  B = 1 is upipe_attn_bwd. */
int upipe_attn_bwd_batch(const void* q, const void* k, const void* v, const void* o,
                         const float* lse, const void* dout, void* dq, void* dk,
                         void* dv, int64_t B, int64_t S, int Hq, int Hkv, int d,
                         int causal, int U, void* ws, size_t ws_bytes,
                         hipStream_t stream);

/* ------------------------------------------------------------------------
 * Rotary position embedding (RoFormer), in place (Section 4 "Implementation":
 * RoPE applied to queries and keys without an fp32 copy of them).
 *
 *   x   bf16 [S, H, d], rotated in place (fp32 arithmetic, one rounding)
 *   pos0     position of row 0: row s sits at position pos0 + s
 *   base     frequency base (e.g. 500000 for Llama 3, 1000000 for Qwen 3)
 *   inverse  0: rotate; 1: rotate back (the transpose, for gradients)
 * Head coordinates e and e + d/2 form pair e (0 <= e < d/2), turned by the
 * angle (pos0 + s) * base^(-2e/d).  d = 128.  Angles are reduced in fp64, so
 * positions up to 2^32 keep full accuracy: 0 <= pos0 and pos0 + S <= 2^32
 * (UPIPE_ERR_UNSUPPORTED otherwise); base must be finite and > 0
 * (UPIPE_ERR_INVALID_ARG).  S = 0 is a no-op.  Needs no workspace.
 * ---------------------------------------------------------------------- */
int upipe_rope(void* x, int64_t S, int H, int d, int64_t pos0, double base, int inverse,
               hipStream_t stream);

/* ------------------------------------------------------------------------
 * Attention block forward (Section 3.3, Appendix A "Untied Ulysses
 * (forward)": per stage, QKV projection of the stage's heads, attention,
 * output written into its slot of `final_out`; after the last stage the
 * output projection y = final_out wo).  Always causal.
 *
 *   x         bf16 [S, d_model]                  hidden states
 *   wqkv      bf16 [d_model, (Hq + 2 Hkv) d]     columns [Q heads|K|V]
 *   wo        bf16 [Hq d, d_model]               output projection
 *   y         bf16 [S, d_model]                  out: final_out @ wo
 *   o_saved   bf16 [S, Hq, d]                    out: final_out (attention
 *                                                output, saved for backward)
 *   lse_saved fp32 [Hq, S]                       out: row log-sum-exp
 * d_model must be a multiple of 128.
 * ---------------------------------------------------------------------- */
int upipe_layer_fwd(const void* x, const void* wqkv, const void* wo, void* y,
                    void* o_saved, float* lse_saved, int64_t S, int d_model,
                    int Hq, int Hkv, int d, int U, void* ws, size_t ws_bytes,
                    hipStream_t stream);

/* ------------------------------------------------------------------------
 * Attention block backward (Appendix A "Untied Ulysses (backward)"): the
 * gradient of final_out, dY wo^T, is formed once and kept for the stage
 * loop, and dWo = final_out^T dY; per chunk, Q_c is recomputed from x and the
 * attention backward yields dQ_c and the running dK, dV sums; after the last
 * chunk dX = [dQ | dK | dV] wqkv^T and dWqkv = x^T [dQ | dK | dV], each in
 * one product.  K and V are recomputed from x (activation checkpointing
 * keeps only x, final_out, lse).
 *
 *   x, wqkv, wo        as for upipe_layer_fwd
 *   o_saved, lse_saved the forward's outputs for the same x and weights
 *                      (selective checkpointing: the attention output is
 *                      kept), or both NULL (full checkpointing: each
 *                      chunk's attention forward is recomputed, bitwise
 *                      equal to the forward's, at the cost of one more
 *                      attention forward; the results are identical)
 *   dy    bf16 [S, d_model]                 upstream gradient of y
 *   dx    bf16 [S, d_model]                 out
 *   dwqkv bf16 [d_model, (Hq + 2 Hkv) d]    out
 *   dwo   bf16 [Hq d, d_model]              out
 * Weight gradients reduce over S with a fixed split of the sequence and a
 * fixed-order sum of the partial products in fp32, rounded once
 * (deterministic, no atomics).
 * ---------------------------------------------------------------------- */
int upipe_layer_bwd(const void* x, const void* wqkv, const void* wo,
                    const void* o_saved, const float* lse_saved,
                    const void* dy, void* dx, void* dwqkv, void* dwo,
                    int64_t S, int d_model, int Hq, int Hkv, int d, int U,
                    void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * The block with a batch of B >= 1 sequences (Appendix "Batch Size
 * Ablation") and rotary position embedding of Q and K (Section 4
 * "Implementation": RoPE applied in place inside the projection, with no
 * fp32 copy and no extra pass).  x, y, dy, dx [B, S, d_model], o_saved
 * [B, S, Hq, d], lse_saved [B, Hq, S]; every sequence starts at position
 * pos0.  dwqkv and dwo are summed over the batch in sequence order in fp32
 * and rounded once.
 *   rope_base  0: no rotary embedding; > 0: Q and K heads are rotated as by
 *              upipe_rope(base = rope_base, pos0) on the fp32 projection
 *              accumulators before their single rounding to bf16; the
 *              backward recomputes them rotated and turns the gradients of
 *              the rotated Q and K back by the inverse rotation
 *   pos0       position of row 0 (same limits as upipe_rope)
 * The backward must get the same B, rope_base and pos0 as the forward.
 * With B = 1, rope_base = 0 these are upipe_layer_fwd / upipe_layer_bwd.
 * ---------------------------------------------------------------------- */
int upipe_layer_fwd_ex(const void* x, const void* wqkv, const void* wo, void* y,
                       void* o_saved, float* lse_saved, int64_t B, int64_t S,
                       int d_model, int Hq, int Hkv, int d, int U, double rope_base,
                       int64_t pos0, void* ws, size_t ws_bytes, hipStream_t stream);
int upipe_layer_bwd_ex(const void* x, const void* wqkv, const void* wo,
                       const void* o_saved, const float* lse_saved,
                       const void* dy, void* dx, void* dwqkv, void* dwo,
                       int64_t B, int64_t S, int d_model, int Hq, int Hkv, int d,
                       int U, double rope_base, int64_t pos0, void* ws,
                       size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * The block's projection product on its own (Appendix A: the QKV projection
 * and y = final_out wo are products of this form): c = a b with a bf16
 * [M, K] and b bf16 [K, N] row-major, c bf16 [M, N] row-major, fp32
 * accumulation in ascending k, one rounding.  M, N, K multiples of 128 and at
 * most 65536 (UPIPE_ERR_UNSUPPORTED otherwise).  For callers that project
 * outside the block, and to measure the GEMM kernel alone.  No workspace.
 * ---------------------------------------------------------------------- */
int upipe_gemm_bf16(const void* a, const void* b, void* c, int64_t M, int64_t N,
                    int64_t K, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Kernel timing (measurement aid).  While enabled, every kernel the library
 * launches is bracketed by two HIP events recorded on the launch stream.
 * upipe_profile_query() waits for the recorded events and reports, for the
 * kernel family `name` (see upipe_profile_name), the number of launches and
 * their summed duration in milliseconds since the last reset.  Enabling
 * creates events with hipEventCreate; the switch is process-global.
 * ---------------------------------------------------------------------- */
int upipe_profile_enable(int on);
int upipe_profile_reset(void);
int upipe_profile_query(const char* name, int* launches, double* total_ms);
/* Name of kernel family i (0 <= i < count), or NULL past the end. */
const char* upipe_profile_name(int i);

#ifdef __cplusplus
}
#endif

#endif /* UPIPE_H */
