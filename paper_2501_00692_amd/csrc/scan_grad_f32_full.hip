// scan_grad_f32_full.hip -- instantiation of the gradient kernels for
// fp32 inputs, full mode.
#include "scan_kernels.h"

namespace ssmk {

hipError_t grad_f32_full(const ScanProblem& p, hipStream_t s) { return grad_sel<float, false>(p, s); }

}  // namespace ssmk
