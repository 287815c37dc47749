// Decode-step entry points (filled in with the projection kernels).
#include <hip/hip_runtime.h>

#include "hpd.h"

extern "C" {

size_t hpd_decode_workspace_bytes(const hpd_model_desc *, const hpd_plan *) { return 0; }

hpd_status hpd_decode_step(const hpd_model_desc *, const hpd_plan *, const float *, float *,
                           const void *const *, const void *const *, void *const *, void *const *,
                           void *, size_t, void *) {
  return HPD_ERR_UNSUPPORTED;
}

}  // extern "C"
