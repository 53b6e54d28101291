// scan_grad_f32_trunc.hip -- instantiation of the gradient kernels for
// fp32 inputs, truncated mode.
#include "scan_kernels.h"

namespace ssmk {

hipError_t grad_f32_trunc(const ScanProblem& p, hipStream_t s) { return grad_sel<float, true>(p, s); }

}  // namespace ssmk
