// Decoder context entry points (window forward + step). Filled in with the
// forward kernels; until then they report SJD_ENOTSUP.
#include <hip/hip_runtime.h>

#include "sjd.h"

struct sjd_ctx {
  int dummy;
};

extern "C" int sjd_init(const sjd_config*, const sjd_weights*, void*, sjd_ctx** out) {
  if (out) *out = nullptr;
  return SJD_ENOTSUP;
}
extern "C" int sjd_prefill(sjd_ctx*, const int32_t*, int32_t, uint64_t, void*) { return SJD_ENOTSUP; }
extern "C" int sjd_step(sjd_ctx*, float, int32_t, uint64_t, uint32_t, int32_t*, int32_t*, int32_t*, void*) {
  return SJD_ENOTSUP;
}
extern "C" int sjd_forward_window(sjd_ctx*, float*, void*) { return SJD_ENOTSUP; }
extern "C" void sjd_destroy(sjd_ctx*) {}
