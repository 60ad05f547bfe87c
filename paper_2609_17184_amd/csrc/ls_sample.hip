// Sampling readouts (temperature > 0): temperature, top-p, softmax, proposal
// draws, the gate and cascade verification with keyed Philox uniforms.
#include "ls_sched.h"

namespace ls {

hipError_t launch_finalize_sample(const Sched&, int, const float*, int, hipStream_t) {
    return hipErrorNotSupported;
}

}  // namespace ls
