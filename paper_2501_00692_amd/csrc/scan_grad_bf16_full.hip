// scan_grad_bf16_full.hip -- instantiation of the gradient kernels for
// bf16 inputs, full mode.
#include "scan_kernels.h"

namespace ssmk {

hipError_t grad_bf16_full(const ScanProblem& p, hipStream_t s) { return grad_sel<uint16_t, false>(p, s); }

}  // namespace ssmk
