// Matrix-core kernels of the backward (placeholder: no shape takes them yet).
#include "moce_internal.h"

namespace moce {

bool bwd_mfma_dalpha(const Shape&, const void*, const void*, const int32_t*, const BwdWs&, hipStream_t, hipError_t*) {
  return false;
}
bool bwd_mfma_dx(const Shape&, const void*, const BwdWs&, void*, hipStream_t, hipError_t*) { return false; }

}  // namespace moce
