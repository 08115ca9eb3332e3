// The gated decode kernels (silu(X W_gate) * (X W_up), decode_kernels.h)
// instantiated for fp16; a translation unit of its own so that the kernel
// families compile in parallel.
#include "decode_kernels.h"

namespace tpdq {

DecodeKernel decode_kernel_gated_f16(const DecodePlan& p) { return pick_gated_dt<kF16>(p); }

}  // namespace tpdq
