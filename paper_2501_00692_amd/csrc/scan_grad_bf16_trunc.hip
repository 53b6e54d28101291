// scan_grad_bf16_trunc.hip -- instantiation of the gradient kernels for
// bf16 inputs, truncated mode.
#include "scan_kernels.h"

namespace ssmk {

hipError_t grad_bf16_trunc(const ScanProblem& p, hipStream_t s) { return grad_sel<uint16_t, true>(p, s); }

}  // namespace ssmk
