// Latent attention for the decode step's independent stream (placeholder until the MFMA kernel
// lands): validates its arguments and reports the path as unavailable.
#include <hip/hip_runtime.h>

#include "nmm_internal.h"

extern "C" {

size_t nmm_latent_attention_workspace_size(int64_t, int64_t, int64_t, int64_t) { return 0; }

nmm_status nmm_latent_attention(int64_t, int64_t, int64_t, int64_t, const void*, int64_t,
                                const void*, int64_t, float, float*, int64_t, void*, size_t,
                                void*) {
    return NMM_ERR_PATH;
}

}  // extern "C"
