// Instantiations of the direct-to-LDS bf16 GEMM kernel (A K-contiguous;
// B K-contiguous or N-contiguous).
#include "gemm_dma.hpp"

namespace isam {

// 256x256 tiles, 8 waves, K slices of whole 64-deep tiles, two slices summed
// inside the kernel.
GemmKernelFn gemm_dma_fixup_kernel_for(int trans_b) {
    return trans_b ? gemm_dma_kernel<256, 256, true, 2, 4, true, true> : gemm_dma_kernel<256, 256, false, 2, 4, true, true>;
}

GemmKernelFn gemm_dma_kernel_for(int tile, int trans_b, int waves, bool k_full) {
    if (waves == 8) {
        switch (tile) {
            case kTile256x256:
                if (k_full)
                    return trans_b ? gemm_dma_kernel<256, 256, true, 2, 4, true> : gemm_dma_kernel<256, 256, false, 2, 4, true>;
                return trans_b ? gemm_dma_kernel<256, 256, true, 2, 4> : gemm_dma_kernel<256, 256, false, 2, 4>;
            case kTile256x128:
                return trans_b ? gemm_dma_kernel<256, 128, true, 4, 2> : gemm_dma_kernel<256, 128, false, 4, 2>;
            default: break;
        }
    }
    switch (tile) {
        case kTile256x256:
            if (k_full)
                return trans_b ? gemm_dma_kernel<256, 256, true, 2, 2, true> : gemm_dma_kernel<256, 256, false, 2, 2, true>;
            return trans_b ? gemm_dma_kernel<256, 256, true> : gemm_dma_kernel<256, 256, false>;
        case kTile256x128: return trans_b ? gemm_dma_kernel<256, 128, true> : gemm_dma_kernel<256, 128, false>;
        case kTile128x128:
            if (k_full)
                return trans_b ? gemm_dma_kernel<128, 128, true, 2, 2, true> : gemm_dma_kernel<128, 128, false, 2, 2, true>;
            return trans_b ? gemm_dma_kernel<128, 128, true> : gemm_dma_kernel<128, 128, false>;
        default: return nullptr;
    }
}

}  // namespace isam
