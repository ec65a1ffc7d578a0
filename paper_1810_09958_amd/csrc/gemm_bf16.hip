// bf16-operand instantiations of the MFMA tile kernel (v_mfma_f32_32x32x16_bf16).
#include "gemm_impl.hpp"

namespace isam {
GemmKernelFn gemm_kernel_bf16(int tile, int ta, int tb, int vec) {
    return gemm_kernel_for<bf16_t>(tile, ta, tb, vec);
}
}  // namespace isam
