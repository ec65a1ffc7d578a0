// GEMM launch: picks the instantiated tile kernel, and reduces split-K
// partials in a fixed order.
#include "gemm_impl.hpp"

#include <stdio.h>
#include <stdlib.h>

#include <atomic>
#include <random>

namespace isam {

GemmKernelFn gemm_kernel_bf16(int tile, int ta, int tb, int vec);
GemmKernelFn gemm_kernel_f32(int tile, int ta, int tb, int vec);
GemmKernelFn gemm_dma_kernel_for(int tile, int trans_b, int waves, bool k_full);
GemmKernelFn gemm_dma_fixup_kernel_for(int trans_b);
GemmKernelFn gemm_dma_sk_kernel_for(int tile, int trans_b, bool k_full, int* threads);

void tile_dims(int tile, int ab_type, int* bm, int* bn, int* bk) {
    static const int dims[kTileCount][2] = {{256, 256}, {256, 128}, {128, 128},
                                            {128, 64},  {64, 64},   {128, 32}};
    *bm = dims[tile][0];
    *bn = dims[tile][1];
    *bk = ab_type == kBF16 ? 64 : 32;
}

bool gemm_sk_tile(int tile) { return tile == kTile256x256 || tile == kTile256x128 || tile == kTile128x128; }

int gemm_sk_grid(int tile, int cus) { return tile == kTile128x128 ? 2 * cus : cus; }

size_t gemm_sk_ws_bytes(int tile, int grid) {
    int bm, bn, bk;
    tile_dims(tile, kBF16, &bm, &bn, &bk);
    return (size_t)grid * ((size_t)bm * bn * 4 + 128);
}

size_t gemm_fixup_ws_bytes(int64_t M, int64_t N) {
    const size_t tiles = (size_t)((M + 255) / 256) * (size_t)((N + 255) / 256);
    return tiles * (256 * 256 * 4) + tiles * 128;
}

namespace {
// Epochs of in-kernel split sums: a random 64-bit start (so a workspace's
// stale flags cannot match by accident) and then one value per launch.
uint64_t next_fixup_epoch() {
    static std::atomic<uint64_t> next{[] {
        std::random_device rd;
        return ((uint64_t)rd() << 32) ^ (uint64_t)rd();
    }()};
    return next.fetch_add(1, std::memory_order_relaxed);
}

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

// Same sum, four adjacent columns per thread: N, ldc and the C address allow
// whole 4-column groups (16-byte partial loads, 16- or 8-byte C accesses).
__global__ __launch_bounds__(256) void splitk_reduce4_kernel(GemmArgs a, int splits) {
    const int64_t total = a.M * a.N;
    const int64_t groups = total >> 2;
    const float4* P = reinterpret_cast<const float4*>(a.partial);
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < groups;
         q += (int64_t)gridDim.x * blockDim.x) {
        const int64_t idx = q << 2;
        const int64_t row = idx / a.N, col = idx - row * a.N;
        float4 v = P[q];
        for (int s = 1; s < splits; ++s) {
            const float4 w = P[(int64_t)s * groups + q];
            v.x += w.x; v.y += w.y; v.z += w.z; v.w += w.w;
        }
        if (a.bias) {
            v.x += a.bias[col]; v.y += a.bias[col + 1]; v.z += a.bias[col + 2]; v.w += a.bias[col + 3];
        }
        const int64_t o = row * a.ldc + col;
        if (a.c_type == kF32) {
            float4* C = reinterpret_cast<float4*>(static_cast<float*>(a.C) + o);
            if (a.accumulate) {
                const float4 c = *C;
                v.x = c.x + v.x; v.y = c.y + v.y; v.z = c.z + v.z; v.w = c.w + v.w;
            }
            *C = v;
        } else {
            uint2* C = reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.C) + o);
            if (a.accumulate) {
                const uint2 c = *C;
                v.x = bf16lo(c.x) + v.x; v.y = bf16hi(c.x) + v.y;
                v.z = bf16lo(c.y) + v.z; v.w = bf16hi(c.y) + v.w;
            }
            *C = make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
        }
    }
}

hipError_t launch_splitk_reduce(const GemmArgs& a, int splits, hipStream_t s) {
    const int64_t total = a.M * a.N;
    const size_t esz = a.c_type == kF32 ? 4 : 2;
    const bool vec4 = a.N % 4 == 0 && a.ldc % 4 == 0 && ((uintptr_t)a.C % (4 * esz)) == 0 &&
                      ((uintptr_t)a.partial % 16) == 0;
    if (vec4) {
        int64_t blocks = (total / 4 + 255) / 256;
        if (blocks > 8192) blocks = 8192;
        hipLaunchKernelGGL(splitk_reduce4_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a, splits);
    } else {
        int64_t blocks = (total + 255) / 256;
        if (blocks > 4096) blocks = 4096;
        hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a, splits);
    }
    return hipGetLastError();
}
}  // namespace

// Stream-K launch: a persistent grid of p.sk_grid workgroups; the tiles are
// split into one contiguous range per XCD (workgroups are dealt to the 8 XCDs
// in turn, so workgroup b runs on XCD b % 8 and the exchanges of a range stay
// in one L2).
// Returns false, launching nothing, when the device cannot hold the whole grid
// at once (the waits need every workgroup resident); the caller then runs the
// tiles one per workgroup.
static bool launch_gemm_sk(const GemmArgs& a, const GemmPlan& p, hipStream_t s, hipError_t* err) {
    int bm, bn, bk;
    tile_dims(p.tile, a.ab_type, &bm, &bn, &bk);
    int threads = 0;
    GemmKernelFn fn = gemm_dma_sk_kernel_for(p.tile, a.trans_b, a.K % 64 == 0, &threads);
    if (!fn) return false;
    const int per_cu = p.tile == kTile128x128 ? 2 : 1;
    if (resident_per_cu(reinterpret_cast<const void*>(fn), threads, 0) * (p.sk_grid / per_cu) < p.sk_grid) return false;
    TileMapArgs t{};
    t.tiles_m = (int)((a.M + bm - 1) / bm);
    t.tiles_n = (int)((a.N + bn - 1) / bn);
    t.group_m = p.group_m > 0 ? p.group_m : 1;
    t.xcd_remap = 0;
    t.k_per_split = a.K;
    t.sk_parts = p.sk_grid % 8 == 0 ? 8 : 1;
    t.sk_nkt = (int)((a.K + 63) / 64);
    t.sk_keep = p.sk_keep;
    t.epoch = next_fixup_epoch();
    t.expect = t.epoch;
    t.wait_ticks = kFixupTimeoutTicks;
    // Test hook (as for the two-slice sum): owners wait for a value no
    // workgroup writes, under a 1 ms bound, so every tile that has partial
    // sums from other workgroups comes back as NaN.
    if (const char* v = getenv("ISAM_GEMM_TEST_FIXUP_STALL"); v && v[0] == '1') {
        t.expect = t.epoch + 1;
        t.wait_ticks = 100000;
    }
    t.flags = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(a.partial) + (size_t)p.sk_grid * bm * bn * 4);
    if (const char* v = getenv("ISAM_LOG"); v && *v && *v != '0')
        fprintf(stderr, "[isam] stream-K: %d workgroups, %d tiles x %d K tiles in %d ranges\n", p.sk_grid,
                t.tiles_m * t.tiles_n, t.sk_nkt, t.sk_parts);
    hipLaunchKernelGGL(fn, dim3((unsigned)p.sk_grid), dim3(threads), 0, s, a, t);
    *err = hipGetLastError();
    return true;
}

hipError_t launch_gemm(const GemmArgs& a, const GemmPlan& p, hipStream_t s) {
    if (a.batch > 1 && (p.k_splits > 1 || p.skinny || p.small)) return hipErrorInvalidValue;
    if (p.skinny == 2) return launch_skinny_rows(a, s);
    if (p.skinny == 4) return launch_narrow(a, s);
    if (p.small) return launch_gemm_small(a, s);
    if (p.skinny) {
        hipError_t e = launch_skinny(a, p.k_splits, s);
        if (e != hipSuccess || p.k_splits <= 1) return e;
        return launch_splitk_reduce(a, p.k_splits, s);
    }
    int bm, bn, bk;
    tile_dims(p.tile, a.ab_type, &bm, &bn, &bk);
    GemmKernelFn fn = nullptr;
    int threads = 256;
    bool fixup = false;
    const bool dma_ok = p.dma && a.ab_type == kBF16 && !a.trans_a && p.vec;
    if (dma_ok && p.sk && p.k_splits <= 1 && a.batch <= 1 && gemm_sk_tile(p.tile) && a.K > 0 &&
        ((uintptr_t)a.partial & 255) == 0) {
        hipError_t e = hipSuccess;
        if (launch_gemm_sk(a, p, s, &e)) return e;
    }
    if (dma_ok) {
        // every K slice a whole number of 64-deep tiles: copies with base + delta offsets
        const bool k_full = a.K % 64 == 0 && (p.k_splits <= 1 || p.k_per_split % 64 == 0);
        fn = gemm_dma_kernel_for(p.tile, a.trans_b, p.dma_waves, k_full);
        if (fn && p.dma_waves == 8 && (p.tile == kTile256x256 || p.tile == kTile256x128)) threads = 512;
        else fn = gemm_dma_kernel_for(p.tile, a.trans_b, 4, k_full);
        // Two K slices of 256x256 tiles: slice 1 adds slice 0's partial sums
        // itself (the plan has checked that both slices of a tile share an XCD).
        fixup = p.fixup && p.k_splits == 2 && k_full && threads == 512 && p.tile == kTile256x256 &&
                ((uintptr_t)a.partial & 255) == 0;
        if (fixup) fn = gemm_dma_fixup_kernel_for(a.trans_b);
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
    // The symmetric form waits in both slices, so it needs every workgroup
    // resident at once (the plan has checked that the grid is within the CU
    // count); the one-way form's first slice never waits.
    t.fixup = fixup ? ((p.fixup == 2 && resident_per_cu(reinterpret_cast<const void*>(fn), threads, 0) >= 1) ? 2 : 1)
                    : 0;
    t.epoch = fixup ? next_fixup_epoch() : 0;
    t.expect = t.epoch;
    t.wait_ticks = kFixupTimeoutTicks;
    // Test hook: the second slice waits for a value the first never writes, under a 1 ms
    // bound, so every tile of the product comes back as NaN.
    if (const char* v = getenv("ISAM_GEMM_TEST_FIXUP_STALL"); fixup && v && v[0] == '1') {
        t.expect = t.epoch + 1;
        t.wait_ticks = 100000;
    }
    t.flags = fixup ? reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(a.partial) +
                                                   (size_t)t.tiles_m * t.tiles_n * (256 * 256 * 4))
                    : nullptr;
    dim3 grid((unsigned)(t.tiles_m * t.tiles_n), (unsigned)(p.k_splits > 1 ? p.k_splits : 1),
              (unsigned)(a.batch > 1 ? a.batch : 1));
    dim3 block(threads);
    if (fixup) {
        const char* v = getenv("ISAM_LOG");
        if (v && *v && *v != '0')
            fprintf(stderr, "[isam] two K slices summed in the kernel%s\n", t.fixup == 2 ? " (each slice finishes half)" : "");
    }
    hipLaunchKernelGGL(fn, grid, block, 0, s, a, t);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || p.k_splits <= 1 || fixup) return e;
    return launch_splitk_reduce(a, p.k_splits, s);
}

}  // namespace isam
