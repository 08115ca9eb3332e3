// The decode kernels (decode_kernels.h) instantiated for bf16 activations,
// scales and outputs; a translation unit of its own so that the two element
// types compile in parallel.
#include "decode_kernels.h"

namespace tpdq {

DecodeKernel decode_kernel_bf16(const DecodePlan& p) { return pick_kernel_dt<kBF16>(p); }

}  // namespace tpdq
