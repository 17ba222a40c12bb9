// bf16 fast search kernels for hidden width 64.
#include "mf_bf16_kernel.h"

namespace mfi {

hipError_t launch_bf16_h64(const Bf16Args &a, const FastConst &fc, const Bf16Const &bc, int grid, int kp, int mode,
                           hipStream_t s)
{
    return launch_bf16_for_width<64>(a, fc, bc, grid, kp, mode, s);
}

}  // namespace mfi
