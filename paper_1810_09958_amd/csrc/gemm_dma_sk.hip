// Instantiations of the stream-K schedule of the direct-to-LDS bf16 GEMM
// kernel (A K-contiguous; B K-contiguous or N-contiguous).
#include "gemm_dma.hpp"

namespace isam {

// 256x256 tiles with 8 waves (2 x 4 of 128x64), 256x128 with 4 (2 x 2 of 128x64), 128x128
// with 4 (2 x 2 of 64x64).  *threads receives the workgroup size.
GemmKernelFn gemm_dma_sk_kernel_for(int tile, int trans_b, bool k_full, int* threads) {
    switch (tile) {
        case kTile256x256:
            *threads = 512;
            if (k_full)
                return trans_b ? gemm_dma_sk_kernel<256, 256, true, 2, 4, true> : gemm_dma_sk_kernel<256, 256, false, 2, 4, true>;
            return trans_b ? gemm_dma_sk_kernel<256, 256, true, 2, 4, false> : gemm_dma_sk_kernel<256, 256, false, 2, 4, false>;
        case kTile256x128:
            *threads = 256;
            if (k_full)
                return trans_b ? gemm_dma_sk_kernel<256, 128, true, 2, 2, true> : gemm_dma_sk_kernel<256, 128, false, 2, 2, true>;
            return trans_b ? gemm_dma_sk_kernel<256, 128, true, 2, 2, false> : gemm_dma_sk_kernel<256, 128, false, 2, 2, false>;
        case kTile128x128:
            *threads = 256;
            if (k_full)
                return trans_b ? gemm_dma_sk_kernel<128, 128, true, 2, 2, true> : gemm_dma_sk_kernel<128, 128, false, 2, 2, true>;
            return trans_b ? gemm_dma_sk_kernel<128, 128, true, 2, 2, false> : gemm_dma_sk_kernel<128, 128, false, 2, 2, false>;
        default: return nullptr;
    }
}

}  // namespace isam
