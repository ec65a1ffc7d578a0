// GEMM launch: picks the instantiated tile kernel, and reduces split-K
// partials in a fixed order.
#include "gemm_impl.hpp"

namespace isam {

GemmKernelFn gemm_kernel_bf16(int tile, int ta, int tb, int vec);
GemmKernelFn gemm_kernel_f32(int tile, int ta, int tb, int vec);
GemmKernelFn gemm_dma_kernel_for(int tile, int trans_b, int waves);

void tile_dims(int tile, int ab_type, int* bm, int* bn, int* bk) {
    static const int dims[kTileCount][2] = {{256, 256}, {256, 128}, {128, 128},
                                            {128, 64},  {64, 64},   {128, 32}};
    *bm = dims[tile][0];
    *bn = dims[tile][1];
    *bk = ab_type == kBF16 ? 64 : 32;
}

namespace {
// C = (accumulate ? C : 0) + bias + sum over splits s = 0, 1, ... of P[s].
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmArgs a, int splits) {
    const int64_t total = a.M * a.N;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int64_t row = idx / a.N, col = idx - row * a.N;
        float v = 0.0f;
        for (int s = 0; s < splits; ++s) v += a.partial[(int64_t)s * total + idx];
        if (a.bias) v += a.bias[col];
        const int64_t o = row * a.ldc + col;
        if (a.c_type == kF32) {
            float* C = static_cast<float*>(a.C);
            if (a.accumulate) v = C[o] + v;
            C[o] = v;
        } else {
            uint16_t* C = static_cast<uint16_t*>(a.C);
            if (a.accumulate) v = bf16_to_f32(C[o]) + v;
            C[o] = (uint16_t)f32_to_bf16(v);
        }
    }
}
}  // namespace

hipError_t launch_gemm(const GemmArgs& a, const GemmPlan& p, hipStream_t s) {
    if (p.skinny) {
        hipError_t e = launch_skinny(a, p.k_splits, s);
        if (e != hipSuccess || p.k_splits <= 1) return e;
        const int64_t total = a.M * a.N;
        int64_t blocks = (total + 255) / 256;
        if (blocks > 4096) blocks = 4096;
        hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a, p.k_splits);
        return hipGetLastError();
    }
    int bm, bn, bk;
    tile_dims(p.tile, a.ab_type, &bm, &bn, &bk);
    GemmKernelFn fn = nullptr;
    int threads = 256;
    if (p.dma && a.ab_type == kBF16 && !a.trans_a && p.vec) {
        fn = gemm_dma_kernel_for(p.tile, a.trans_b, p.dma_waves);
        if (fn && p.dma_waves == 8 && (p.tile == kTile256x256 || p.tile == kTile256x128)) threads = 512;
        else fn = gemm_dma_kernel_for(p.tile, a.trans_b, 4);
    }
    if (!fn)
        fn = a.ab_type == kBF16 ? gemm_kernel_bf16(p.tile, a.trans_a, a.trans_b, p.vec)
                                : gemm_kernel_f32(p.tile, a.trans_a, a.trans_b, p.vec);
    if (!fn) return hipErrorInvalidValue;
    TileMapArgs t;
    t.tiles_m = (int)((a.M + bm - 1) / bm);
    t.tiles_n = (int)((a.N + bn - 1) / bn);
    t.group_m = p.group_m > 0 ? p.group_m : 1;
    t.xcd_remap = p.xcd_remap;
    t.k_per_split = p.k_splits > 1 ? p.k_per_split : a.K;
    if (t.k_per_split <= 0) t.k_per_split = 1;
    dim3 grid((unsigned)(t.tiles_m * t.tiles_n), (unsigned)(p.k_splits > 1 ? p.k_splits : 1));
    dim3 block(threads);
    hipLaunchKernelGGL(fn, grid, block, 0, s, a, t);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || p.k_splits <= 1) return e;
    const int64_t total = a.M * a.N;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a, p.k_splits);
    return hipGetLastError();
}

}  // namespace isam
