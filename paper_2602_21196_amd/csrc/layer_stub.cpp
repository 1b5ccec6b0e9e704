// Placeholder: the attention-block (projection) entry points.
#include "../../include/upipe.h"
extern "C" {
size_t upipe_layer_fwd_workspace_size(int64_t, int, int, int, int, int) { return 0; }
size_t upipe_layer_bwd_workspace_size(int64_t, int, int, int, int, int) { return 0; }
int upipe_layer_fwd(const void*, const void*, const void*, void*, void*, float*, int64_t, int,
                    int, int, int, int, void*, size_t, hipStream_t) {
  return UPIPE_ERR_UNSUPPORTED;
}
int upipe_layer_bwd(const void*, const void*, const void*, const void*, const float*,
                    const void*, void*, void*, void*, int64_t, int, int, int, int, int, void*,
                    size_t, hipStream_t) {
  return UPIPE_ERR_UNSUPPORTED;
}
}
