// Very shallow products: C (+)= A.B of the paper's first listing (Section 2)
// with K <= 256 and N <= 256, bf16 A [M][K] (K-contiguous) and B [K][N]
// (N-contiguous) -- the pointwise half of the separable convolution (Section
// 2.3: M pixels, K input channels, N output channels) when it is not fused
// with the depthwise stencil.  Such a product is bound by streaming A in and
// C out of HBM; a tiled GEMM spends most of each tile in its prologue (load
// latency) and epilogue.  Here B stays in registers for the whole launch and
// A streams through a ring of LDS stages:
//   * persistent workgroups (at most one per CU) take 32-row tiles of A in
//     turn;
//   * 8 consumer waves each own 32 output columns: their slice of B, read
//     once at the start, is the A operand of v_mfma_f32_32x32x16_bf16 for the
//     transposed product C^T = B^T . A^T, whose B operand is the A tile read
//     with ds_read_b128; results leave as 4-column stores straight from the
//     accumulators, so consumers issue no loads after the start;
//   * 4 producer waves copy the tiles into an 8-stage ring with buffer_load
//     ... lds and issue no stores, so their waits on the vector-memory
//     counter count only their own copies (on gfx9 that counter also counts
//     stores);
//   * one workgroup barrier per tile: at barrier i the copies of tile i have
//     landed and every consumer has finished reading tile i-1, whose stage the
//     producers then refill with tile i+7.
// LDS layout of a stage: row r (one pixel, CPR 16-byte chunks), chunk c at
// c ^ swz(r) -- (r ^ r>>3) & 7 for 8-chunk rows, r & 15 for wider rows: the
// 16 rows of every b128 read phase land on 16 different bank groups.
#include "common.hpp"
#include "kernels.hpp"

namespace isam {
namespace {

constexpr int kStreamConsumers = 8;
constexpr int kStreamProducers = 4;
constexpr int kStreamStages = 8;
constexpr int kStreamRows = 32;  // A rows (pixels) per tile

__device__ __forceinline__ void st_dma16(__amdgpu_buffer_rsrc_t rs, uint32_t lds_addr, uint32_t voff) {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %1, %2, 0 offen lds"
        :
        : "s"(lds_addr), "v"(voff), "s"(rs)
        : "memory", "m0");
}

template <int N>
__device__ __forceinline__ void st_vm_wait() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

__device__ __forceinline__ void st_barrier() {
    asm volatile("" : : : "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" : : : "memory");
}

template <int CPR>
__device__ __forceinline__ int st_swz(int r) {
    if constexpr (CPR == 8) return (r ^ (r >> 3)) & 7;
    else return r & 15;
}

// CPR: 16-byte chunks per A row in LDS (8, 16 or 32: K up to 64, 128, 256).
template <int CPR>
__global__ __launch_bounds__(64 * (kStreamConsumers + kStreamProducers)) void gemm_stream_kernel(GemmArgs a) {
    constexpr int STAGE = kStreamRows * CPR * 16;
    constexpr int COPIES = kStreamRows * CPR / 64;         // 1 KB copies per tile
    constexpr int CPW = COPIES / kStreamProducers;          // per producer wave
    constexpr int KS = CPR / 2;                             // 16-deep MFMA steps
    static_assert(COPIES % kStreamProducers == 0, "copies split evenly");
    __shared__ __attribute__((aligned(1024))) char smem[kStreamStages * STAGE];

    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int64_t ntiles = (a.M + kStreamRows - 1) / kStreamRows;
    // this workgroup's tiles: blockIdx.x, blockIdx.x + gridDim.x, ...
    const int nt = (int)((ntiles - blockIdx.x + gridDim.x - 1) / gridDim.x);

    if (wid >= kStreamConsumers) {
        // ---------------- producers ----------------
        const int p = wid - kStreamConsumers;
        const __amdgpu_buffer_rsrc_t rsA = make_rsrc(a.A, (uint32_t)(((a.M - 1) * a.lda + a.K) * 2));
        const uint32_t base = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)smem;
        // per copy q: LDS unit u = (p*CPW + q)*64 + lane -> row r, physical chunk pc
        int row_in[CPW], kof[CPW];
#pragma unroll
        for (int q = 0; q < CPW; ++q) {
            const int u = (p * CPW + q) * 64 + lane;
            const int r = u / CPR, pc = u % CPR;
            row_in[q] = r;
            kof[q] = (pc ^ st_swz<CPR>(r)) * 8;
        }
        // Copies of local tile i (tiles past the last one read nothing).
        auto issue = [&](int i) {
            const int64_t m0 = ((int64_t)blockIdx.x + (int64_t)i * gridDim.x) * kStreamRows;
            const uint32_t st = base + (uint32_t)((i % kStreamStages) * STAGE);
#pragma unroll
            for (int q = 0; q < CPW; ++q) {
                const int64_t m = m0 + row_in[q];
                const bool in = i < nt && m < a.M && kof[q] < a.K;
                st_dma16(rsA, __builtin_amdgcn_readfirstlane(st + (uint32_t)((p * CPW + q) * 1024)),
                         in ? (uint32_t)((m * a.lda + kof[q]) * 2) : kOob);
            }
        };
        for (int i = 0; i < kStreamStages - 1; ++i) issue(i);
        for (int i = 0; i < nt; ++i) {
            // tile i has landed once at most the copies of tiles i+1 .. i+S-2 are in flight
            st_vm_wait<(kStreamStages - 2) * CPW>();
            st_barrier();
            issue(i + kStreamStages - 1);  // into the stage of tile i-1, read before this barrier
        }
        st_vm_wait<0>();  // nothing may still be landing when the workgroup's LDS is released
        return;
    }

    // ---------------- consumers ----------------
    const int64_t n0 = (int64_t)wid * 32;
    const int g = lane >> 5, l32 = lane & 31;
    // B^T slice as MFMA A operands: step s, lane (n = n0 + l32, K group g):
    // B[16 s + 8 g + e][n], e = 0..7
    uint4 bt[KS];
    {
        const __amdgpu_buffer_rsrc_t rsB = make_rsrc(a.B, (uint32_t)(((a.K - 1) * a.ldb + a.N) * 2));
        const int64_t n = n0 + l32;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            uint32_t w[4];
#pragma unroll
            for (int e2 = 0; e2 < 4; ++e2) {
                const int64_t k = 16 * s + 8 * g + 2 * e2;
                const uint32_t lo = buf_load2(rsB, (n < a.N && k < a.K) ? (uint32_t)((k * a.ldb + n) * 2) : kOob);
                const uint32_t hi = buf_load2(rsB, (n < a.N && k + 1 < a.K) ? (uint32_t)(((k + 1) * a.ldb + n) * 2) : kOob);
                w[e2] = (lo & 0xffffu) | (hi << 16);
            }
            bt[s] = make_uint4(w[0], w[1], w[2], w[3]);
        }
    }
    const bool wave_on = n0 < a.N;
    // output columns of this lane: n0 + 8 q + 4 g + (0..3), q = 0..3
    float bias[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        const int64_t n = n0 + 8 * (v >> 2) + 4 * g + (v & 3);
        bias[v] = (a.bias && n < a.N) ? a.bias[n] : 0.0f;
    }
    for (int i = 0; i < nt; ++i) {
        st_barrier();
        if (!wave_on) continue;
        const char* st = smem + (i % kStreamStages) * STAGE;
        f32x16_t acc;
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[v] = 0.0f;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            // A^T fragment: pixel l32, K chunk 2 s + g
            const int c = 2 * s + g;
            const uint4 af = *reinterpret_cast<const uint4*>(st + l32 * (CPR * 16) + ((c ^ st_swz<CPR>(l32)) << 4));
            mfma32_bf16(acc, bt[s], af);
        }
        const int64_t m = ((int64_t)blockIdx.x + (int64_t)i * gridDim.x) * kStreamRows + l32;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int64_t n = n0 + 8 * q + 4 * g;
            // N % 4 == 0: a group of 4 columns is all in or all out
            if (m >= a.M || n >= a.N) continue;
            float o[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) o[e] = acc[4 * q + e] + bias[4 * q + e];
            const int64_t idx = m * a.ldc + n;
            if (a.c_type == kF32) {
                float4* C = reinterpret_cast<float4*>(static_cast<float*>(a.C) + idx);
                if (a.accumulate) {
                    const float4 c4 = *C;
                    o[0] += c4.x; o[1] += c4.y; o[2] += c4.z; o[3] += c4.w;
                }
                *C = make_float4(o[0], o[1], o[2], o[3]);
            } else {
                uint2* C = reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.C) + idx);
                if (a.accumulate) {
                    const uint2 c2 = *C;
                    o[0] += bf16lo(c2.x); o[1] += bf16hi(c2.x); o[2] += bf16lo(c2.y); o[3] += bf16hi(c2.y);
                }
                *C = make_uint2(pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]));
            }
        }
    }
}

}  // namespace

bool gemm_stream_fits(const GemmArgs& a) {
    const int es_c = a.c_type == kF32 ? 4 : 2;
    return a.ab_type == kBF16 && !a.trans_a && !a.trans_b && a.batch <= 1 && a.M > 0 && a.K > 0 && a.K <= 256 &&
           a.N > 0 && a.N <= 32 * kStreamConsumers && a.N % 4 == 0 && a.K % 8 == 0 && a.lda % 8 == 0 &&
           ((uintptr_t)a.A & 15) == 0 && ((uintptr_t)a.C & 15) == 0 && (a.ldc * es_c) % 16 == 0;
}

hipError_t launch_gemm_stream(const GemmArgs& a, int cus, hipStream_t s) {
    if (!gemm_stream_fits(a)) return hipErrorInvalidValue;
    const int64_t ntiles = (a.M + kStreamRows - 1) / kStreamRows;
    const dim3 grid((unsigned)std::min<int64_t>(ntiles, cus)), block(64 * (kStreamConsumers + kStreamProducers));
    if (a.K <= 64) hipLaunchKernelGGL(gemm_stream_kernel<8>, grid, block, 0, s, a);
    else if (a.K <= 128) hipLaunchKernelGGL(gemm_stream_kernel<16>, grid, block, 0, s, a);
    else hipLaunchKernelGGL(gemm_stream_kernel<32>, grid, block, 0, s, a);
    return hipGetLastError();
}

}  // namespace isam
