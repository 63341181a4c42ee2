// One (dtype, head_dim) pair of the step kernel, for every group size; built
// once per pair with KVEC_INST_TT (BF16 or F32) and KVEC_INST_D (64 or 128).
#include "kvec_step.h"

#if !defined(KVEC_INST_TT) || !defined(KVEC_INST_D)
#error "define KVEC_INST_TT and KVEC_INST_D"
#endif

namespace kvec {
namespace step {

template <>
StepFn pick_g<KVEC_INST_TT, KVEC_INST_D>(int G) {
  switch (G) {
    case 1: return step_kernel<KVEC_INST_TT, KVEC_INST_D, 1>;
    case 2: return step_kernel<KVEC_INST_TT, KVEC_INST_D, 2>;
    case 3: return step_kernel<KVEC_INST_TT, KVEC_INST_D, 3>;
    case 4: return step_kernel<KVEC_INST_TT, KVEC_INST_D, 4>;
    case 5: return step_kernel<KVEC_INST_TT, KVEC_INST_D, 5>;
    case 6: return step_kernel<KVEC_INST_TT, KVEC_INST_D, 6>;
    case 7: return step_kernel<KVEC_INST_TT, KVEC_INST_D, 7>;
    default: return step_kernel<KVEC_INST_TT, KVEC_INST_D, 8>;
  }
}

}  // namespace step
}  // namespace kvec
