// Small dense products: C (+)= A.B of the paper's first listing (Section 2)
// when the output has at most 64 tiles of 32x32 and K is moderate -- the
// fp32 128^3 case among them.  The tile kernels give such a product a few
// workgroups that walk K one LDS stage at a time, so the time is the load
// latency of every stage plus the MFMAs of one SIMD.  Here one workgroup owns
// one 32x32 output tile and its four waves split K: each wave issues all the
// loads of its K range at once (fragments straight from global memory, no
// LDS staging), runs its MFMAs, and the four partial tiles are summed through
// LDS in wave order (deterministic), followed by the usual epilogue (bias,
// accumulate, fp32 or bf16 output).
//
// Requirements (checked by the planner): A K-contiguous (no transpose),
// 16-byte aligned operands and leading dimensions, K a multiple of the
// 16-byte element count, batch 1.
#include "common.hpp"
#include "kernels.hpp"

namespace isam {
namespace {

constexpr int kSmallWaves = 4;
constexpr int kSmallBatch = 8;  // K blocks whose loads are issued together

template <typename T, bool TB>
__global__ __launch_bounds__(64 * kSmallWaves) void gemm_small_kernel(GemmArgs a) {
    constexpr int E = 16 / (int)sizeof(T);  // K values per lane per fragment
    constexpr int KB = 2 * E;               // K values per MFMA step (two lane halves)
    constexpr int64_t es = (int64_t)sizeof(T);
    __shared__ float red[kSmallWaves][16][64];

    const int tiles_n = (int)((a.N + 31) / 32);
    const int64_t m0 = (int64_t)(blockIdx.x / tiles_n) * 32, n0 = (int64_t)(blockIdx.x % tiles_n) * 32;
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const int half = lane >> 5;
    const int64_t row = m0 + (lane & 31), col = n0 + (lane & 31);
    const int64_t nkb = (a.K + KB - 1) / KB;
    const int64_t kb_lo = nkb * wid / kSmallWaves, kb_hi = nkb * (wid + 1) / kSmallWaves;

    const int64_t a_ext = (a.M - 1) * a.lda + a.K;
    const int64_t b_ext = TB ? ((a.N - 1) * a.ldb + a.K) : ((a.K - 1) * a.ldb + a.N);
    const __amdgpu_buffer_rsrc_t rsA = make_rsrc(a.A, (uint32_t)(a_ext * es));
    const __amdgpu_buffer_rsrc_t rsB = make_rsrc(a.B, (uint32_t)(b_ext * es));
    const bool row_ok = row < a.M, col_ok = col < a.N;

    f32x16_t acc;
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[v] = 0.0f;
    for (int64_t kb0 = kb_lo; kb0 < kb_hi; kb0 += kSmallBatch) {
        uint4 af[kSmallBatch], bfr[kSmallBatch];
#pragma unroll
        for (int u = 0; u < kSmallBatch; ++u) {
            const int64_t kb = kb0 + u;
            const int64_t k = kb * KB + half * E;
            const bool kok = kb < kb_hi && k < a.K;  // K % E == 0: a piece is all in or all out
            af[u] = buf_load16(rsA, (kok && row_ok) ? (uint32_t)((row * a.lda + k) * es) : kOob);
            if constexpr (TB) {
                bfr[u] = buf_load16(rsB, (kok && col_ok) ? (uint32_t)((col * a.ldb + k) * es) : kOob);
            } else {
                // B[k..k+E)[col]: E strided elements gathered into one fragment
                uint32_t w[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if constexpr (sizeof(T) == 4) {
                        w[q] = buf_load4(rsB, (kok && col_ok) ? (uint32_t)(((k + q) * a.ldb + col) * es) : kOob);
                    } else {
                        const uint32_t lo = buf_load2(rsB, (kok && col_ok) ? (uint32_t)(((k + 2 * q) * a.ldb + col) * es) : kOob);
                        const uint32_t hi = buf_load2(rsB, (kok && col_ok) ? (uint32_t)(((k + 2 * q + 1) * a.ldb + col) * es) : kOob);
                        w[q] = (lo & 0xffffu) | (hi << 16);
                    }
                }
                bfr[u] = make_uint4(w[0], w[1], w[2], w[3]);
            }
        }
        // all of the batch's loads are in flight before the first MFMA waits
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < kSmallBatch; ++u) {
            if (kb0 + u >= kb_hi) break;  // wave-uniform: the rest of the batch is zeros
            if constexpr (sizeof(T) == 2) mfma32_bf16(acc, af[u], bfr[u]);
            else mfma32_f32x4(acc, af[u], bfr[u]);
        }
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) red[wid][v][lane] = acc[v];
    __syncthreads();
    // Element (v, l) of the tile: row 8*(v/4) + 4*(l/32) + v%4, column l%32;
    // consecutive threads take consecutive columns of one row.
    for (int idx = threadIdx.x; idx < 16 * 64; idx += 64 * kSmallWaves) {
        const int v = idx >> 6, l = idx & 63;
        const int64_t r = m0 + 8 * (v >> 2) + 4 * (l >> 5) + (v & 3), c = n0 + (l & 31);
        if (r >= a.M || c >= a.N) continue;
        float s = red[0][v][l];
#pragma unroll
        for (int w = 1; w < kSmallWaves; ++w) s += red[w][v][l];
        if (a.bias) s += a.bias[c];
        const int64_t o = r * a.ldc + c;
        if (a.c_type == kF32) {
            float* C = static_cast<float*>(a.C);
            if (a.accumulate) s += C[o];
            C[o] = s;
        } else {
            uint16_t* C = static_cast<uint16_t*>(a.C);
            if (a.accumulate) s += bf16_to_f32(C[o]);
            C[o] = (uint16_t)f32_to_bf16(s);
        }
    }
}

}  // namespace

bool gemm_small_fits(int64_t M, int64_t N, int64_t K) {
    return M > 0 && N > 0 && K > 0 && K <= kSmallMaxK && ((M + 31) / 32) * ((N + 31) / 32) <= kSmallMaxTiles;
}

hipError_t launch_gemm_small(const GemmArgs& a, hipStream_t s) {
    if (a.trans_a || a.batch > 1 || !gemm_small_fits(a.M, a.N, a.K)) return hipErrorInvalidValue;
    const unsigned grid = (unsigned)(((a.M + 31) / 32) * ((a.N + 31) / 32));
    const dim3 block(64 * kSmallWaves);
    if (a.ab_type == kBF16) {
        if (a.trans_b) hipLaunchKernelGGL((gemm_small_kernel<uint16_t, true>), dim3(grid), block, 0, s, a);
        else hipLaunchKernelGGL((gemm_small_kernel<uint16_t, false>), dim3(grid), block, 0, s, a);
    } else {
        if (a.trans_b) hipLaunchKernelGGL((gemm_small_kernel<float, true>), dim3(grid), block, 0, s, a);
        else hipLaunchKernelGGL((gemm_small_kernel<float, false>), dim3(grid), block, 0, s, a);
    }
    return hipGetLastError();
}

}  // namespace isam
