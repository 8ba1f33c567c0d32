// TEMPORARY placeholder (not committed): the fused path is being written.
#include <hip/hip_runtime.h>
#include "grpo.h"
extern "C" size_t fused_lmhead_workspace_bytes(int64_t, int64_t, int64_t, int32_t, int32_t) { return 0; }
extern "C" int fused_lmhead_grpo(const void*, const void*, int64_t, int64_t, int64_t, int32_t, const int32_t*,
                                 const float*, const float*, const float*, const grpo_segments*,
                                 const grpo_loss_params*, double*, void*, float*, int32_t, grpo_aux*, void*, size_t,
                                 hipStream_t) { return GRPO_ERR_SHAPE; }
