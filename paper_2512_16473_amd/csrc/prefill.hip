// Prefill path placeholder (filled in with the grouped MFMA implementation).
#include <hip/hip_runtime.h>

#include "common.h"
#include "moe_internal.h"

extern "C" {

size_t moe_prefill_workspace_bytes(const moe_prefill_desc *P, int T)
{
    (void)P;
    (void)T;
    return 0;
}

int moe_prefill_forward(const moe_prefill_desc *P, const float *X_dev, int T, float *OUT_dev, int32_t *idx_dev,
                        float *w_dev, void *workspace, size_t workspace_bytes, void *stream)
{
    (void)P; (void)X_dev; (void)T; (void)OUT_dev; (void)idx_dev; (void)w_dev; (void)workspace;
    (void)workspace_bytes; (void)stream;
    moe::set_error("moe_prefill_forward: not available in this build");
    return MOE_ESTATE;
}

}  // extern "C"
