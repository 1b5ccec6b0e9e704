// C ABI of the head-chunked attention library (declared in include/upipe.h).
//
// Host-side responsibilities: argument validation before anything is
// enqueued, the workspace plan (one chunk-sized set of buffers reused for
// every chunk, plus the buffers that live for the whole call), the chunk loop
// of UPipe (paper Section 3.3: nu = Hq/U stages of U heads), and optional
// per-kernel event timing.  All kernels run on the caller's stream.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <cmath>

#include <mutex>
#include <new>
#include <vector>

#include "../../include/upipe.h"
#include "api_internal.h"
#include "kernels.h"

namespace upipe {

// ------------------------------------------------------------ profiling
namespace {

struct ProfRecord {
  int family;
  hipEvent_t start, stop;
};

struct Profiler {
  bool on = false;
  std::vector<ProfRecord> recs;
  std::vector<hipEvent_t> pool;
  hipEvent_t get() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
};

Profiler& prof() {
  static Profiler p;
  return p;
}

}  // namespace

const char* const kFamilyNames[] = {
    "pack_rows",      "unpack_rows",   "rowdot_lse",     "attn_fwd",
    "attn_bwd_dkdv",  "attn_bwd_dq",   "gemm",           "gemm_wgrad",
    "reduce_splitk",  "lse_merge",     "rope",           "split_merge",
};
const int kNumFamilies = sizeof(kFamilyNames) / sizeof(kFamilyNames[0]);

ProfScope::ProfScope(int family, hipStream_t st) : st_(st) {
  Profiler& p = prof();
  if (!p.on) return;
  start_ = p.get();
  stop_ = p.get();
  family_ = family;
  if (start_ && stop_) (void)hipEventRecord(start_, st_);
}

ProfScope::~ProfScope() {
  Profiler& p = prof();
  if (!p.on || !start_ || !stop_) return;
  (void)hipEventRecord(stop_, st_);
  try {
    p.recs.push_back({family_, start_, stop_});
  } catch (...) {
  }
}

// --------------------------------------------------------------- checks
bool aligned16(const void* p) { return p && ((uintptr_t)p & 15u) == 0; }

int check_attn_shape(int64_t S, int Hq, int Hkv, int d, int U) {
  if (S < 1 || Hq < 1 || Hkv < 1 || U < 1) return UPIPE_ERR_INVALID_ARG;
  if (Hq % Hkv != 0 || Hq % U != 0) return UPIPE_ERR_INVALID_ARG;
  if (d != HEAD_DIM) return UPIPE_ERR_UNSUPPORTED;
  if (Hq > kMaxHeads) return UPIPE_ERR_UNSUPPORTED;
  const int64_t Sp = round_up(S, SEQ_PAD);
  if (Sp > kMaxSeq) return UPIPE_ERR_UNSUPPORTED;
  if (Sp * (int64_t)Hq * d >= (int64_t(1) << 40)) return UPIPE_ERR_UNSUPPORTED;
  return UPIPE_OK;
}

bool group_split(int Hq, int Hkv, int U) {
  const int G = Hq / Hkv;
  for (int g = 0; g < Hkv; ++g)
    if ((g * G) / U != ((g + 1) * G - 1) / U) return true;
  return false;
}

// ----------------------------------------------------------- ws planning
size_t Carver::take(size_t bytes) {
  const size_t off = (used + 255) & ~size_t(255);
  used = off + bytes;
  return off;
}

AttnFwdPlan plan_attn_fwd_ring(int64_t Sq, int64_t Skv, int Hq, int Hkv, int U) {
  AttnFwdPlan p;
  p.Sp = round_up(Sq, SEQ_PAD);
  p.Skvp = round_up(Skv, SEQ_PAD);
  const size_t qhead = (size_t)p.Sp * HEAD_DIM * 2, kvhead = (size_t)p.Skvp * HEAD_DIM * 2;
  Carver c;
  p.kv_direct = kv_in_place(Skv, Hkv);
  if (!p.kv_direct) {
    p.Kp = c.take(Hkv * kvhead);
    p.Vp = c.take(Hkv * kvhead);
  }
  p.Qc = c.take(U * qhead);
  p.ns = attn_fwd_key_splits(p.Sp, p.Skvp);
  p.Oc = c.take(p.ns * U * qhead);
  if (p.ns > 1) p.lse_part = c.take((size_t)p.ns * U * p.Sp * 4);
  p.total = c.used;
  return p;
}

AttnFwdPlan plan_attn_fwd(int64_t S, int Hq, int Hkv, int U) {
  return plan_attn_fwd_ring(S, S, Hq, Hkv, U);
}

AttnBwdPlan plan_attn_bwd(int64_t S, int Hq, int Hkv, int U) {
  AttnBwdPlan p;
  p.Sp = round_up(S, SEQ_PAD);
  const size_t head = (size_t)p.Sp * HEAD_DIM * 2;
  const size_t row32 = (size_t)p.Sp * 4;
  Carver c;
  p.kv_direct = kv_in_place(S, Hkv);
  if (!p.kv_direct) {
    p.Kp = c.take(Hkv * head);
    p.Vp = c.take(Hkv * head);
  }
  p.carry = group_split(Hq, Hkv, U);
  if (p.carry) {
    p.dK32 = c.take(Hkv * head * 2);
    p.dV32 = c.take(Hkv * head * 2);
  }
  p.Qc = c.take(U * head);
  p.dOc = c.take(U * head);
  p.dQc = c.take(U * head);
  p.D = c.take(U * row32);
  p.lse_c = c.take(U * row32);
  p.total = c.used;
  return p;
}

// ------------------------------------------------------- attention paths
int run_dkdv_chunk(const bf16* Qc, const bf16* dOc, const float* lse_c, const float* D,
                   const bf16* Kp, const bf16* Vp, float* dK32, float* dV32, bf16* dk, bf16* dv,
                   int64_t kv_row, int64_t kv_head, int64_t S, int64_t Sp, int U, int h0, int G,
                   int causal, hipStream_t st) {
  const bool per_head = U > 1 && (dK32 != nullptr || G == 1);
  if (!per_head) {
    UPIPE_LAUNCH(kAttnBwdDkdv, st,
                 launch_attn_bwd_dkdv(Qc, dOc, lse_c, D, Kp, Vp, dK32, dV32, dk, dv, kv_row,
                                      kv_head, S, Sp, U, h0, G, causal, st));
    return UPIPE_OK;
  }
  const int64_t head = Sp * HEAD_DIM;
  for (int u = 0; u < U; ++u)
    UPIPE_LAUNCH(kAttnBwdDkdv, st,
                 launch_attn_bwd_dkdv(Qc + u * head, dOc + u * head, lse_c + u * Sp, D + u * Sp,
                                      Kp, Vp, dK32, dV32, dk, dv, kv_row, kv_head, S, Sp, 1,
                                      h0 + u, G, causal, st));
  return UPIPE_OK;
}

int run_attn_fwd_ring(const bf16* q, const bf16* k, const bf16* v, bf16* o, float* lse,
                      int64_t Sq, int64_t Skv, int64_t delta, int Hq, int Hkv, int causal,
                      int U, char* ws, hipStream_t st) {
  const AttnFwdPlan p = plan_attn_fwd_ring(Sq, Skv, Hq, Hkv, U);
  const bf16* Kp = p.kv_direct ? k : (const bf16*)(ws + p.Kp);
  const bf16* Vp = p.kv_direct ? v : (const bf16*)(ws + p.Vp);
  bf16* Qc = (bf16*)(ws + p.Qc);
  bf16* Oc = (bf16*)(ws + p.Oc);
  const int G = Hq / Hkv;
  // Key/value heads: packed once (unless already head-major), resident for
  // every chunk (on one device the GQA schedule needs each key/value head
  // from its group's first stage on, Section 4.1).
  if (!p.kv_direct) {
    UPIPE_LAUNCH(kPackRows, st,
                 launch_pack_rows(k, Skv, Hkv, 0, Hkv, p.Skvp, (bf16*)(ws + p.Kp), st));
    UPIPE_LAUNCH(kPackRows, st,
                 launch_pack_rows(v, Skv, Hkv, 0, Hkv, p.Skvp, (bf16*)(ws + p.Vp), st));
  }
  for (int h0 = 0; h0 < Hq; h0 += U) {
    UPIPE_LAUNCH(kPackRows, st, launch_pack_rows(q, Sq, Hq, h0, U, p.Sp, Qc, st));
    if (p.ns == 1) {
      UPIPE_LAUNCH(kAttnFwd, st, launch_attn_fwd(Qc, Kp, Vp, Oc, lse, Sq, p.Sp, Skv, p.Skvp, delta,
                                                 U, h0, G, causal, st));
    } else {
      // Two key halves per query block (the grid would otherwise leave CUs
      // idle), merged like two ring steps: rows [U][Sp] as one head.
      float* lp = (float*)(ws + p.lse_part);
      const int64_t rows = (int64_t)U * p.Sp;
      UPIPE_LAUNCH(kAttnFwd, st,
                   launch_attn_fwd_split(Qc, Kp, Vp, Oc, lp, Sq, p.Sp, Skv, p.Skvp, delta, U, h0,
                                         G, causal, p.ns, 0, p.Sp, p.Sp, st));
      UPIPE_LAUNCH(kSplitMerge, st,
                   launch_lse_merge(Oc, lp, Oc + rows * HEAD_DIM, lp + rows, rows, 1, st));
      UPIPE_LAUNCH(kUnpackRows, st,
                   hipMemcpy2DAsync(lse + (int64_t)h0 * Sq, Sq * 4, lp, p.Sp * 4, Sq * 4, U,
                                    hipMemcpyDeviceToDevice, st));
    }
    UPIPE_LAUNCH(kUnpackRows, st, launch_unpack_rows(Oc, Sq, Hq, h0, U, p.Sp, o, st));
  }
  return UPIPE_OK;
}

int make_rope(double base, int64_t pos0, int64_t S, RopeArgs* out) {
  *out = RopeArgs{0.0, 0, 0};
  if (base == 0.0) return UPIPE_OK;
  if (!(base > 0.0) || !std::isfinite(base)) return UPIPE_ERR_INVALID_ARG;
  if (pos0 < 0 || pos0 > kMaxRopePos || S > kMaxRopePos - pos0) return UPIPE_ERR_UNSUPPORTED;
  *out = RopeArgs{std::log2(base), pos0, 1};
  return UPIPE_OK;
}

int run_attn_fwd(const bf16* q, const bf16* k, const bf16* v, bf16* o,
                 float* lse, int64_t S, int Hq, int Hkv, int causal, int U,
                 char* ws, hipStream_t st) {
  return run_attn_fwd_ring(q, k, v, o, lse, S, S, 0, Hq, Hkv, causal, U, ws, st);
}

int run_attn_bwd(const bf16* q, const bf16* k, const bf16* v, const bf16* o,
                 const float* lse, const bf16* dout, bf16* dq, bf16* dk,
                 bf16* dv, int64_t S, int Hq, int Hkv, int causal, int U,
                 char* ws, hipStream_t st) {
  const AttnBwdPlan p = plan_attn_bwd(S, Hq, Hkv, U);
  const bf16* Kp = p.kv_direct ? k : (const bf16*)(ws + p.Kp);
  const bf16* Vp = p.kv_direct ? v : (const bf16*)(ws + p.Vp);
  float* dK32 = p.carry ? (float*)(ws + p.dK32) : nullptr;
  float* dV32 = p.carry ? (float*)(ws + p.dV32) : nullptr;
  bf16* Qc = (bf16*)(ws + p.Qc);
  bf16* dOc = (bf16*)(ws + p.dOc);
  bf16* dQc = (bf16*)(ws + p.dQc);
  float* D = (float*)(ws + p.D);
  float* lse_c = (float*)(ws + p.lse_c);
  const int G = Hq / Hkv;
  if (!p.kv_direct) {
    UPIPE_LAUNCH(kPackRows, st,
                 launch_pack_rows(k, S, Hkv, 0, Hkv, p.Sp, (bf16*)(ws + p.Kp), st));
    UPIPE_LAUNCH(kPackRows, st,
                 launch_pack_rows(v, S, Hkv, 0, Hkv, p.Sp, (bf16*)(ws + p.Vp), st));
  }
  for (int h0 = 0; h0 < Hq; h0 += U) {
    UPIPE_LAUNCH(kPackRows, st, launch_pack_rows(q, S, Hq, h0, U, p.Sp, Qc, st));
    UPIPE_LAUNCH(kPackRows, st, launch_pack_rows(dout, S, Hq, h0, U, p.Sp, dOc, st));
    UPIPE_LAUNCH(kRowdotLse, st,
                 launch_rowdot_lse(dout + h0 * HEAD_DIM, (int64_t)Hq * HEAD_DIM, HEAD_DIM,
                                   o + h0 * HEAD_DIM, (int64_t)Hq * HEAD_DIM, HEAD_DIM, lse, S,
                                   h0, U, p.Sp, D, lse_c, st));
    const int rc = run_dkdv_chunk(Qc, dOc, lse_c, D, Kp, Vp, dK32, dV32, dk, dv,
                                  (int64_t)Hkv * HEAD_DIM, HEAD_DIM, S, p.Sp, U, h0, G, causal,
                                  st);
    if (rc != UPIPE_OK) return rc;
    UPIPE_LAUNCH(kAttnBwdDq, st,
                 launch_attn_bwd_dq(Qc, dOc, lse_c, D, Kp, Vp, dQc, S, p.Sp, U, h0, G, causal,
                                    RopeArgs{}, st));
    UPIPE_LAUNCH(kUnpackRows, st, launch_unpack_rows(dQc, S, Hq, h0, U, p.Sp, dq, st));
  }
  return UPIPE_OK;
}

}  // namespace upipe

using namespace upipe;

extern "C" {

const char* upipe_status_string(int status) {
  switch (status) {
    case UPIPE_OK: return "UPIPE_OK";
    case UPIPE_ERR_INVALID_ARG: return "UPIPE_ERR_INVALID_ARG";
    case UPIPE_ERR_UNSUPPORTED: return "UPIPE_ERR_UNSUPPORTED";
    case UPIPE_ERR_WORKSPACE: return "UPIPE_ERR_WORKSPACE";
    case UPIPE_ERR_HIP: return "UPIPE_ERR_HIP";
    default: return "UPIPE_ERR_UNKNOWN";
  }
}

int upipe_version(void) { return 100; }

int upipe_gqa_schedule(int H, int Hkv, int C, int U, int* stage_heads,
                       int* kv_stage) {
  if (H < 1 || Hkv < 1 || C < 1 || U < 1 || !stage_heads || !kv_stage)
    return UPIPE_ERR_INVALID_ARG;
  if (H % Hkv || U % C || H % U || H % C || Hkv % C) return UPIPE_ERR_INVALID_ARG;
  const int G = H / Hkv, per_dev = H / C, per_stage = U / C;
  for (int g = 0; g < Hkv; ++g) kv_stage[g] = -1;
  int n = 0;
  for (int s = 0; s < H / U; ++s)
    for (int p = 0; p < C; ++p)
      for (int j = 0; j < per_stage; ++j) {
        const int h = p * per_dev + s * per_stage + j;
        stage_heads[n++] = h;
        if (kv_stage[h / G] < 0) kv_stage[h / G] = s;
      }
  return UPIPE_OK;
}

size_t upipe_attn_fwd_workspace_size(int64_t S, int Hq, int Hkv, int d, int U) {
  if (check_attn_shape(S, Hq, Hkv, d, U) != UPIPE_OK) return 0;
  return plan_attn_fwd(S, Hq, Hkv, U).total;
}

size_t upipe_attn_bwd_workspace_size(int64_t S, int Hq, int Hkv, int d, int U) {
  if (check_attn_shape(S, Hq, Hkv, d, U) != UPIPE_OK) return 0;
  return plan_attn_bwd(S, Hq, Hkv, U).total;
}

static int attn_fwd_batch(const void* q, const void* k, const void* v, void* o, float* lse,
                          int64_t B, int64_t S, int Hq, int Hkv, int d, int causal, int U,
                          void* ws, size_t ws_bytes, hipStream_t stream) {
  try {
    int rc = check_attn_shape(S, Hq, Hkv, d, U);
    if (rc != UPIPE_OK) return rc;
    if (!batch_ok(B, S * Hq * HEAD_DIM)) return UPIPE_ERR_INVALID_ARG;
    if (causal != 0 && causal != 1) return UPIPE_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) ||
        !aligned16(lse) || !aligned16(ws))
      return UPIPE_ERR_INVALID_ARG;
    if (ws_bytes < plan_attn_fwd(S, Hq, Hkv, U).total) return UPIPE_ERR_WORKSPACE;
    // The B sequences run one after another through the same workspace.
    const int64_t qs = S * Hq * HEAD_DIM, ks = S * Hkv * HEAD_DIM, ls = (int64_t)Hq * S;
    for (int64_t b = 0; b < B; ++b) {
      rc = run_attn_fwd((const bf16*)q + b * qs, (const bf16*)k + b * ks,
                        (const bf16*)v + b * ks, (bf16*)o + b * qs, lse + b * ls, S, Hq, Hkv,
                        causal, U, (char*)ws, stream);
      if (rc != UPIPE_OK) return rc;
    }
    return UPIPE_OK;
  } catch (...) {
    return UPIPE_ERR_HIP;
  }
}

int upipe_attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse, int64_t S,
                   int Hq, int Hkv, int d, int causal, int U, void* ws, size_t ws_bytes,
                   hipStream_t stream) {
  return attn_fwd_batch(q, k, v, o, lse, 1, S, Hq, Hkv, d, causal, U, ws, ws_bytes, stream);
}

int upipe_attn_fwd_batch(const void* q, const void* k, const void* v, void* o, float* lse,
                         int64_t B, int64_t S, int Hq, int Hkv, int d, int causal, int U,
                         void* ws, size_t ws_bytes, hipStream_t stream) {
  return attn_fwd_batch(q, k, v, o, lse, B, S, Hq, Hkv, d, causal, U, ws, ws_bytes, stream);
}

size_t upipe_attn_fwd_ring_workspace_size(int64_t Sq, int64_t Skv, int Hq, int Hkv, int d, int U) {
  if (check_attn_shape(Sq, Hq, Hkv, d, U) != UPIPE_OK) return 0;
  if (check_attn_shape(Skv, Hq, Hkv, d, U) != UPIPE_OK) return 0;
  return plan_attn_fwd_ring(Sq, Skv, Hq, Hkv, U).total;
}

int upipe_attn_fwd_ring(const void* q, const void* k, const void* v, void* o, float* lse,
                        int64_t Sq, int64_t Skv, int64_t q_offset, int64_t kv_offset, int Hq,
                        int Hkv, int d, int causal, int U, void* ws, size_t ws_bytes,
                        hipStream_t stream) {
  try {
    int rc = check_attn_shape(Sq, Hq, Hkv, d, U);
    if (rc != UPIPE_OK) return rc;
    rc = check_attn_shape(Skv, Hq, Hkv, d, U);
    if (rc != UPIPE_OK) return rc;
    if (causal != 0 && causal != 1) return UPIPE_ERR_INVALID_ARG;
    const int64_t lim = int64_t(1) << 62;
    if (q_offset < -lim || q_offset > lim || kv_offset < -lim || kv_offset > lim)
      return UPIPE_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) ||
        !aligned16(lse) || !aligned16(ws))
      return UPIPE_ERR_INVALID_ARG;
    int64_t delta;   // q_offset - kv_offset; fits unless it is exactly 2^63
    if (__builtin_sub_overflow(q_offset, kv_offset, &delta)) return UPIPE_ERR_INVALID_ARG;
    if (ws_bytes < plan_attn_fwd_ring(Sq, Skv, Hq, Hkv, U).total) return UPIPE_ERR_WORKSPACE;
    return run_attn_fwd_ring((const bf16*)q, (const bf16*)k, (const bf16*)v, (bf16*)o, lse, Sq,
                             Skv, delta, Hq, Hkv, causal, U, (char*)ws, stream);
  } catch (...) {
    return UPIPE_ERR_HIP;
  }
}

int upipe_lse_merge(void* o, float* lse, const void* o_part, const float* lse_part, int64_t S,
                    int H, int d, hipStream_t stream) {
  try {
    if (S < 1 || H < 1) return UPIPE_ERR_INVALID_ARG;
    if (d != HEAD_DIM) return UPIPE_ERR_UNSUPPORTED;
    if (H > kMaxHeads || S > kMaxSeq) return UPIPE_ERR_UNSUPPORTED;
    if (!aligned16(o) || !aligned16(lse) || !aligned16(o_part) || !aligned16(lse_part))
      return UPIPE_ERR_INVALID_ARG;
    UPIPE_LAUNCH(kLseMerge, stream,
                 launch_lse_merge((bf16*)o, lse, (const bf16*)o_part, lse_part, S, H, stream));
    return UPIPE_OK;
  } catch (...) {
    return UPIPE_ERR_HIP;
  }
}

int upipe_rope(void* x, int64_t S, int H, int d, int64_t pos0, double base, int inverse,
               hipStream_t stream) {
  try {
    if (S < 0 || H < 1 || (inverse != 0 && inverse != 1) || base == 0.0)
      return UPIPE_ERR_INVALID_ARG;
    if (d != HEAD_DIM) return UPIPE_ERR_UNSUPPORTED;
    if (H > kMaxHeads || S > kMaxSeq) return UPIPE_ERR_UNSUPPORTED;
    RopeArgs r;
    const int rc = make_rope(base, pos0, S, &r);
    if (rc != UPIPE_OK) return rc;
    if (!aligned16(x)) return UPIPE_ERR_INVALID_ARG;
    if (S == 0) return UPIPE_OK;
    UPIPE_LAUNCH(kRope, stream,
                 launch_rope((bf16*)x, S, H, (int64_t)H * HEAD_DIM, HEAD_DIM, r, inverse, stream));
    return UPIPE_OK;
  } catch (...) {
    return UPIPE_ERR_HIP;
  }
}

static int attn_bwd_batch(const void* q, const void* k, const void* v, const void* o,
                          const float* lse, const void* dout, void* dq, void* dk, void* dv,
                          int64_t B, int64_t S, int Hq, int Hkv, int d, int causal, int U,
                          void* ws, size_t ws_bytes, hipStream_t stream) {
  try {
    int rc = check_attn_shape(S, Hq, Hkv, d, U);
    if (rc != UPIPE_OK) return rc;
    if (!batch_ok(B, S * Hq * HEAD_DIM)) return UPIPE_ERR_INVALID_ARG;
    if (causal != 0 && causal != 1) return UPIPE_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) ||
        !aligned16(lse) || !aligned16(dout) || !aligned16(dq) || !aligned16(dk) ||
        !aligned16(dv) || !aligned16(ws))
      return UPIPE_ERR_INVALID_ARG;
    if (ws_bytes < plan_attn_bwd(S, Hq, Hkv, U).total) return UPIPE_ERR_WORKSPACE;
    const int64_t qs = S * Hq * HEAD_DIM, ks = S * Hkv * HEAD_DIM, ls = (int64_t)Hq * S;
    for (int64_t b = 0; b < B; ++b) {
      rc = run_attn_bwd((const bf16*)q + b * qs, (const bf16*)k + b * ks,
                        (const bf16*)v + b * ks, (const bf16*)o + b * qs, lse + b * ls,
                        (const bf16*)dout + b * qs, (bf16*)dq + b * qs, (bf16*)dk + b * ks,
                        (bf16*)dv + b * ks, S, Hq, Hkv, causal, U, (char*)ws, stream);
      if (rc != UPIPE_OK) return rc;
    }
    return UPIPE_OK;
  } catch (...) {
    return UPIPE_ERR_HIP;
  }
}

int upipe_attn_bwd(const void* q, const void* k, const void* v, const void* o, const float* lse,
                   const void* dout, void* dq, void* dk, void* dv, int64_t S, int Hq, int Hkv,
                   int d, int causal, int U, void* ws, size_t ws_bytes, hipStream_t stream) {
  return attn_bwd_batch(q, k, v, o, lse, dout, dq, dk, dv, 1, S, Hq, Hkv, d, causal, U, ws,
                        ws_bytes, stream);
}

int upipe_attn_bwd_batch(const void* q, const void* k, const void* v, const void* o,
                         const float* lse, const void* dout, void* dq, void* dk, void* dv,
                         int64_t B, int64_t S, int Hq, int Hkv, int d, int causal, int U,
                         void* ws, size_t ws_bytes, hipStream_t stream) {
  return attn_bwd_batch(q, k, v, o, lse, dout, dq, dk, dv, B, S, Hq, Hkv, d, causal, U, ws,
                        ws_bytes, stream);
}

int upipe_profile_enable(int on) {
  prof().on = on != 0;
  return UPIPE_OK;
}

int upipe_profile_reset(void) {
  Profiler& p = prof();
  for (auto& r : p.recs) {
    p.pool.push_back(r.start);
    p.pool.push_back(r.stop);
  }
  p.recs.clear();
  return UPIPE_OK;
}

int upipe_profile_query(const char* name, int* launches, double* total_ms) {
  if (!name || !launches || !total_ms) return UPIPE_ERR_INVALID_ARG;
  int fam = -1;
  for (int i = 0; i < kNumFamilies; ++i)
    if (strcmp(name, kFamilyNames[i]) == 0) fam = i;
  if (fam < 0) return UPIPE_ERR_INVALID_ARG;
  int n = 0;
  double ms = 0.0;
  for (auto& r : prof().recs) {
    if (r.family != fam) continue;
    if (hipEventSynchronize(r.stop) != hipSuccess) return UPIPE_ERR_HIP;
    float e = 0.f;
    if (hipEventElapsedTime(&e, r.start, r.stop) != hipSuccess) return UPIPE_ERR_HIP;
    ms += e;
    ++n;
  }
  *launches = n;
  *total_ms = ms;
  return UPIPE_OK;
}

const char* upipe_profile_name(int i) {
  return (i >= 0 && i < kNumFamilies) ? kFamilyNames[i] : nullptr;
}

}  // extern "C"
