// fp32-operand instantiations of the MFMA tile kernel (v_mfma_f32_32x32x2_f32).
// gfx950 has no reduced-precision fp32 MFMA shortcut, so fp32 inputs keep
// full fp32 products.
#include "gemm_impl.hpp"

namespace isam {
GemmKernelFn gemm_kernel_f32(int tile, int ta, int tb, int vec) {
    return gemm_kernel_for<float>(tile, ta, tb, vec);
}
}  // namespace isam
