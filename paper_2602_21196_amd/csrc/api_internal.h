// Host-only internals shared by the ABI translation units.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "common.h"

namespace upipe {

constexpr int kMaxHeads = 64;
// Longest padded sequence: the kernels address one head's [Sp][128] slab and
// its [128][Sp] transpose with 32-bit byte offsets and buffer resources of
// Sp * 256 bytes, which must stay below 2^32.
constexpr int64_t kMaxSeq = (int64_t(1) << 24) - SEQ_PAD;

// Kernel families for event timing; order matches kFamilyNames in api.cpp.
enum Family {
  kPackRows = 0,
  kUnpackRows,
  kRowdotLse,
  kAttnFwd,
  kAttnBwdDkdv,
  kAttnBwdDq,
  kGemm,
  kGemmWgrad,
  kReduceSplitk,
  kLseMerge,
  kRope,
  kSplitMerge,
};

// Records HIP events around one launch when profiling is on.
class ProfScope {
 public:
  ProfScope(int family, hipStream_t st);
  ~ProfScope();

 private:
  hipStream_t st_;
  hipEvent_t start_ = nullptr, stop_ = nullptr;
  int family_ = -1;
};

#define UPIPE_LAUNCH(family, stream, expr)           \
  do {                                               \
    ::upipe::ProfScope _ps((family), (stream));      \
    if ((expr) != hipSuccess) return UPIPE_ERR_HIP;  \
  } while (0)

bool aligned16(const void* p);
// B sequences of `per_seq` elements each address below 2^61 elements (so no
// pointer offset into a batch can overflow); B >= 1.
inline bool batch_ok(int64_t B, int64_t per_seq) {
  return B >= 1 && per_seq >= 1 && B <= (int64_t(1) << 61) / per_seq;
}
// Rotary-embedding arguments from the ABI's (base, pos0) for rows 0..S-1:
// base == 0 means no rotation; otherwise base must be finite and > 0
// (UPIPE_ERR_INVALID_ARG) and positions pos0 .. pos0 + S - 1 must lie in
// [0, kMaxRopePos) (UPIPE_ERR_UNSUPPORTED).
constexpr int64_t kMaxRopePos = int64_t(1) << 32;
int make_rope(double base, int64_t pos0, int64_t S, RopeArgs* out);
int check_attn_shape(int64_t S, int Hq, int Hkv, int d, int U);
bool group_split(int Hq, int Hkv, int U);

// Bump allocator over the caller's workspace (256-byte aligned offsets).
struct Carver {
  size_t used = 0;
  size_t take(size_t bytes);
};

// Token-major keys/values [S, Hkv, d] already are the head-major [Hkv, Sp, d]
// the kernels read when there is one key/value head and no padding: then they
// are read in place instead of being copied into the workspace.
inline bool kv_in_place(int64_t S, int Hkv) { return Hkv == 1 && S % SEQ_PAD == 0; }

struct AttnFwdPlan {
  int64_t Sp = 0;     // query rows, padded
  int64_t Skvp = 0;   // key/value rows, padded
  int ns = 1;         // key splits per query block (their partial results are merged)
  bool kv_direct = false;   // keys/values read in place (no Kp, Vp)
  size_t Kp = 0, Vp = 0, Qc = 0, Oc = 0, lse_part = 0, total = 0;
};

struct AttnBwdPlan {
  int64_t Sp = 0;
  bool carry = false;  // a key/value group spans several chunks
  bool kv_direct = false;   // keys/values read in place (no Kp, Vp)
  size_t Kp = 0, Vp = 0, dK32 = 0, dV32 = 0;
  size_t Qc = 0, dOc = 0, dQc = 0, D = 0, lse_c = 0;
  size_t total = 0;
};

// dK/dV of the chunk of U heads starting at h0 (arguments as for
// launch_attn_bwd_dkdv; Qc, dOc, lse_c, D hold the chunk's U heads).  When
// the fp32 carries exist (dK32 != nullptr: some group spans chunks) or every
// group is one head (G == 1), the heads go one launch each: the same
// additions in the same order as a single launch over the chunk (the carries
// hand each head's sums to the next), but every workgroup of a launch then
// walks one head's query tiles alongside the others and they share L2
// lines, where in one launch over several heads they drift apart.
int run_dkdv_chunk(const bf16* Qc, const bf16* dOc, const float* lse_c, const float* D,
                   const bf16* Kp, const bf16* Vp, float* dK32, float* dV32, bf16* dk, bf16* dv,
                   int64_t kv_row, int64_t kv_head, int64_t S, int64_t Sp, int U, int h0, int G,
                   int causal, hipStream_t st);

AttnFwdPlan plan_attn_fwd(int64_t S, int Hq, int Hkv, int U);
AttnFwdPlan plan_attn_fwd_ring(int64_t Sq, int64_t Skv, int Hq, int Hkv, int U);
AttnBwdPlan plan_attn_bwd(int64_t S, int Hq, int Hkv, int U);

int run_attn_fwd(const bf16* q, const bf16* k, const bf16* v, bf16* o,
                 float* lse, int64_t S, int Hq, int Hkv, int causal, int U,
                 char* ws, hipStream_t st);
int run_attn_fwd_ring(const bf16* q, const bf16* k, const bf16* v, bf16* o, float* lse,
                      int64_t Sq, int64_t Skv, int64_t delta, int Hq, int Hkv, int causal,
                      int U, char* ws, hipStream_t st);
int run_attn_bwd(const bf16* q, const bf16* k, const bf16* v, const bf16* o,
                 const float* lse, const bf16* dout, bf16* dq, bf16* dk,
                 bf16* dv, int64_t S, int Hq, int Hkv, int causal, int U,
                 char* ws, hipStream_t st);

}  // namespace upipe
