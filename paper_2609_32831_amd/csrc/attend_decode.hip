// attend_decode.hip -- bf16 decode attention on matrix cores (placeholder:
// not eligible yet, every call takes the generic path).
#include "uc_common.h"

namespace uc {
bool decode_mfma_eligible(const uc_shape&, const KSegs&, int, int) { return false; }
size_t decode_mfma_workspace(const uc_shape&, const KSegs&, int) { return 0; }
hipError_t launch_decode_mfma(const uc_shape&, const KSegs&, const void*, int, float, float*,
                              float*, float*, void*, hipStream_t) {
  return hipErrorNotSupported;
}
}  // namespace uc
