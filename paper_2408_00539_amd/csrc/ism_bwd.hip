// Backward ISM attention on gfx950 (placeholder until the kernels land).
#include "ism_common.h"
#include "ism_kernels.h"

namespace ism {

hipError_t launch_bwd(const BwdArgs &a, int d, hipStream_t stream) {
  (void)a; (void)d; (void)stream;
  return hipErrorNotSupported;
}

}  // namespace ism
