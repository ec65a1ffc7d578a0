// Operand packing for the products of the paper's first listing (Section 2)
// whose rows cannot be fetched in 16-byte pieces: a contiguous dimension that
// is not a multiple of 8 bf16 / 4 fp32 values, or a base pointer or leading
// dimension off 16 bytes.  The MFMA kernels copy operands into LDS 16 bytes at
// a time, so such a product would otherwise run on the element-wise tile
// kernel.  These kernels copy a row-major matrix into a dense buffer whose row
// length is a multiple of 16 bytes -- optionally transposed, so that K becomes
// the contiguous dimension -- and write zeros everywhere outside the source.
// Padded K positions are then zero in both operands, so they add exact zeros
// to every dot product and the result is that of the unpadded product.
//
// The values are moved as opaque 2- or 4-byte words (the zero bit pattern is
// +0.0 in both formats); no arithmetic is done on them.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace isam {
namespace {

constexpr int kPackThreads = 256;
constexpr int kPackTile = 64;  // edge of the transposed tile

// dst[i][j] = src[i][j] (i < s_rows, j < s_cols), else 0; one 16-byte group
// of a destination row per lane and step, read as G-byte pieces (G: the
// largest power of two up to 16 that divides the source base and row pitch).
template <typename T, int G>
__global__ __launch_bounds__(kPackThreads) void pack_copy_kernel(const T* __restrict__ src, int64_t s_rows,
                                                                  int64_t s_cols, int64_t ld, T* __restrict__ dst,
                                                                  int64_t d_rows, int64_t d_cols) {
    constexpr int E = 16 / (int)sizeof(T);
    constexpr int P = 16 / G;  // pieces per group
    // the destination is below 2^31 bytes: unit and row indices fit 32 bits
    const uint32_t upr = (uint32_t)(d_cols / E), units = (uint32_t)d_rows * upr;
    for (uint32_t u = blockIdx.x * kPackThreads + threadIdx.x; u < units; u += gridDim.x * kPackThreads) {
        const uint32_t i = u / upr;
        const int64_t j0 = (int64_t)(u - i * upr) * E;
        uint4 v;
        if ((int64_t)i < s_rows && j0 + E <= s_cols) {
            const char* q = reinterpret_cast<const char*>(src + (int64_t)i * ld + j0);
            uint32_t w[4];
            if constexpr (G == 16) {
                v = *reinterpret_cast<const uint4*>(q);
            } else if constexpr (G == 8) {
                const uint2 a = reinterpret_cast<const uint2*>(q)[0], b = reinterpret_cast<const uint2*>(q)[1];
                v = make_uint4(a.x, a.y, b.x, b.y);
            } else if constexpr (G == 4) {
#pragma unroll
                for (int p = 0; p < P; ++p) w[p] = reinterpret_cast<const uint32_t*>(q)[p];
                v = make_uint4(w[0], w[1], w[2], w[3]);
            } else {
                uint32_t h[8];
#pragma unroll
                for (int p = 0; p < 8; ++p) h[p] = reinterpret_cast<const uint16_t*>(q)[p];
                v = make_uint4(h[0] | h[1] << 16, h[2] | h[3] << 16, h[4] | h[5] << 16, h[6] | h[7] << 16);
            }
        } else {
            T e[E];
#pragma unroll
            for (int k = 0; k < E; ++k) {
                const int64_t j = j0 + k;
                e[k] = ((int64_t)i < s_rows && j < s_cols) ? src[(int64_t)i * ld + j] : T(0);
            }
            v = __builtin_bit_cast(uint4, e);
        }
        *reinterpret_cast<uint4*>(dst + (int64_t)i * d_cols + j0) = v;
    }
}

// bf16 transpose with 16-byte source rows: dst[i][j] = src[j][i] (j < s_rows,
// i < s_cols), else 0.  A lane reads an 8x8 block (8 source rows, 16 bytes
// each), transposes it in registers and writes 8 destination rows of 16 bytes;
// the lanes of a wave cover 64x64 (8 lanes per 128-byte run on both sides),
// the 4 waves of a workgroup 64 source rows x 256 source columns.
__global__ __launch_bounds__(kPackThreads) void pack_transpose8_kernel(const uint16_t* __restrict__ src,
                                                                        int64_t s_rows, int64_t s_cols, int64_t ld,
                                                                        uint16_t* __restrict__ dst, int64_t d_rows,
                                                                        int64_t d_cols) {
    const int64_t tiles_k = (d_cols + 63) / 64;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int64_t k = (int64_t)(blockIdx.x % tiles_k) * 64 + 8 * (lane >> 3);
    const int64_t m = (int64_t)(blockIdx.x / tiles_k) * 256 + 64 * w + 8 * (lane & 7);
    uint4 in[8], out[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int64_t r = k + e;
        if (r < s_rows && m + 8 <= s_cols) {
            in[e] = *reinterpret_cast<const uint4*>(src + r * ld + m);
        } else {
            uint32_t h[8];
#pragma unroll
            for (int c = 0; c < 8; ++c) h[c] = (r < s_rows && m + c < s_cols) ? src[r * ld + m + c] : 0u;
            in[e] = make_uint4(h[0] | h[1] << 16, h[2] | h[3] << 16, h[4] | h[5] << 16, h[6] | h[7] << 16);
        }
    }
    transpose8x8_b16(in, out);
    if (k >= d_cols) return;
#pragma unroll
    for (int c = 0; c < 8; ++c)
        if (m + c < d_rows) *reinterpret_cast<uint4*>(dst + (m + c) * d_cols + k) = out[c];
}

// dst[i][j] = src[j][i] (j < s_rows, i < s_cols), else 0.  A workgroup moves
// one 64x64 block through LDS: lanes read along a source row and write along
// a destination row, so both sides are contiguous per wave.  Row stride 65
// words: a lane column of the block falls on 64 different banks.
template <typename T>
__global__ __launch_bounds__(kPackThreads) void pack_transpose_kernel(const T* __restrict__ src, int64_t s_rows,
                                                                       int64_t s_cols, int64_t ld,
                                                                       T* __restrict__ dst, int64_t d_rows,
                                                                       int64_t d_cols) {
    __shared__ uint32_t blk[kPackTile][kPackTile + 1];
    const int64_t tiles_c = (d_cols + kPackTile - 1) / kPackTile;
    const int64_t i0 = (int64_t)(blockIdx.x / tiles_c) * kPackTile, j0 = (int64_t)(blockIdx.x % tiles_c) * kPackTile;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    // block rows: source rows j0 + r (destination columns), lanes: source
    // columns i0 + lane (destination rows)
    for (int r = w; r < kPackTile; r += kPackThreads / 64) {
        const int64_t sr = j0 + r, sc = i0 + lane;
        blk[r][lane] = (sr < s_rows && sc < s_cols) ? (uint32_t)src[sr * ld + sc] : 0u;
    }
    __syncthreads();
    for (int r = w; r < kPackTile; r += kPackThreads / 64) {
        const int64_t i = i0 + r, j = j0 + lane;
        if (i < d_rows && j < d_cols) dst[i * d_cols + j] = (T)blk[lane][r];
    }
}

// fp32 operand split for the bf16-term product (see split3_pair): a source
// value becomes its three bf16 terms, written into six K blocks of Kp values
// in the order the 2-bit fields of `pattern` give (0 = h, 1 = m, 2 = l), so
// that one bf16 product over K' = 6 Kp sums the six significant term
// products.  Zeros outside the source.  KROWS = false: K is the contiguous
// source dimension (src [rows][K]); dst [rows][6 Kp], block b at column b Kp.
// KROWS = true: K is the source row (src [K][cols]); dst [6 Kp][cols], block b
// at row b Kp.  One 8-value group of a destination row per lane and step.
template <bool KROWS>
__global__ __launch_bounds__(kPackThreads) void split6_kernel(const float* __restrict__ src, int64_t s_rows,
                                                               int64_t s_cols, int64_t ld, uint16_t* __restrict__ dst,
                                                               int64_t d_rows, int64_t d_cols, int64_t kp,
                                                               uint32_t pattern, int vec) {
    const uint32_t upr = (uint32_t)(d_cols / 8), units = (uint32_t)d_rows * upr;
    for (uint32_t u = blockIdx.x * kPackThreads + threadIdx.x; u < units; u += gridDim.x * kPackThreads) {
        const uint32_t r = u / upr;
        const int64_t c0 = (int64_t)(u - r * upr) * 8;
        float x[8];
        const float* q = src + (int64_t)r * ld + c0;
        if (vec && (int64_t)r < s_rows && c0 + 8 <= s_cols) {
            const float4 a = reinterpret_cast<const float4*>(q)[0], b = reinterpret_cast<const float4*>(q)[1];
            x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) x[e] = ((int64_t)r < s_rows && c0 + e < s_cols) ? q[e] : 0.0f;
        }
        uint32_t t[4][3];
#pragma unroll
        for (int p = 0; p < 4; ++p) split3_pair(x[2 * p], x[2 * p + 1], t[p]);
#pragma unroll
        for (int b = 0; b < 6; ++b) {
            const int term = (pattern >> (2 * b)) & 3;
            const uint4 v = make_uint4(t[0][term], t[1][term], t[2][term], t[3][term]);
            const int64_t off = KROWS ? ((int64_t)b * kp + r) * d_cols + c0 : (int64_t)r * 6 * kp + (int64_t)b * kp + c0;
            *reinterpret_cast<uint4*>(dst + off) = v;
        }
    }
}

}  // namespace

hipError_t launch_pack(const void* src, int64_t s_rows, int64_t s_cols, int64_t ld, void* dst, int64_t d_rows,
                       int64_t d_cols, int esize, bool transpose, int cus, hipStream_t s) {
    if (d_rows <= 0 || d_cols <= 0) return hipSuccess;
    // widest piece that the source base and row pitch allow
    int g = 16;
    while (g > esize && (((uintptr_t)src % g) != 0 || (ld * esize) % g != 0)) g /= 2;
    if (transpose && esize == 2 && g == 16 && d_cols % 8 == 0 && (uintptr_t)dst % 16 == 0) {
        const int64_t n = ((d_rows + 255) / 256) * ((d_cols + 63) / 64);
        hipLaunchKernelGGL(pack_transpose8_kernel, dim3((unsigned)n), dim3(kPackThreads), 0, s,
                           static_cast<const uint16_t*>(src), s_rows, s_cols, ld, static_cast<uint16_t*>(dst), d_rows,
                           d_cols);
    } else if (transpose) {
        const int64_t n = ((d_rows + kPackTile - 1) / kPackTile) * ((d_cols + kPackTile - 1) / kPackTile);
        if (esize == 2)
            hipLaunchKernelGGL(pack_transpose_kernel<uint16_t>, dim3((unsigned)n), dim3(kPackThreads), 0, s,
                               static_cast<const uint16_t*>(src), s_rows, s_cols, ld, static_cast<uint16_t*>(dst),
                               d_rows, d_cols);
        else
            hipLaunchKernelGGL(pack_transpose_kernel<uint32_t>, dim3((unsigned)n), dim3(kPackThreads), 0, s,
                               static_cast<const uint32_t*>(src), s_rows, s_cols, ld, static_cast<uint32_t*>(dst),
                               d_rows, d_cols);
    } else {
        const int64_t units = d_rows * (d_cols * esize / 16);
        const int64_t blocks = std::min<int64_t>((units + kPackThreads - 1) / kPackThreads, (int64_t)cus * 16);
        auto go = [&](auto kern, auto* tsrc, auto* tdst) {
            hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kPackThreads), 0, s, tsrc, s_rows, s_cols, ld, tdst,
                               d_rows, d_cols);
        };
        const uint16_t* s16 = static_cast<const uint16_t*>(src);
        const uint32_t* s32 = static_cast<const uint32_t*>(src);
        uint16_t* d16 = static_cast<uint16_t*>(dst);
        uint32_t* d32 = static_cast<uint32_t*>(dst);
        if (esize == 2) {
            if (g == 16) go(pack_copy_kernel<uint16_t, 16>, s16, d16);
            else if (g == 8) go(pack_copy_kernel<uint16_t, 8>, s16, d16);
            else if (g == 4) go(pack_copy_kernel<uint16_t, 4>, s16, d16);
            else go(pack_copy_kernel<uint16_t, 2>, s16, d16);
        } else {
            if (g == 16) go(pack_copy_kernel<uint32_t, 16>, s32, d32);
            else if (g == 8) go(pack_copy_kernel<uint32_t, 8>, s32, d32);
            else go(pack_copy_kernel<uint32_t, 4>, s32, d32);
        }
    }
    return hipGetLastError();
}

hipError_t launch_split6(const float* src, int64_t s_rows, int64_t s_cols, int64_t ld, uint16_t* dst,
                         int64_t d_rows, int64_t d_cols, int64_t kp, bool k_rows, uint32_t pattern, int cus,
                         hipStream_t s) {
    if (d_rows <= 0 || d_cols <= 0) return hipSuccess;
    const int vec = ((uintptr_t)src % 16 == 0 && (ld * 4) % 16 == 0) ? 1 : 0;
    const int64_t units = d_rows * (d_cols / 8);
    const int64_t blocks = std::min<int64_t>((units + kPackThreads - 1) / kPackThreads, (int64_t)cus * 16);
    if (k_rows)
        hipLaunchKernelGGL(split6_kernel<true>, dim3((unsigned)blocks), dim3(kPackThreads), 0, s, src, s_rows, s_cols,
                           ld, dst, d_rows, d_cols, kp, pattern, vec);
    else
        hipLaunchKernelGGL(split6_kernel<false>, dim3((unsigned)blocks), dim3(kPackThreads), 0, s, src, s_rows,
                           s_cols, ld, dst, d_rows, d_cols, kp, pattern, vec);
    return hipGetLastError();
}

}  // namespace isam
