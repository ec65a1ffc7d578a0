// Depthwise half of the separable depthwise convolution (the paper's third
// listing, after the pointwise weight is factored out of the (di, dj)
// reduction, Section 2.3):
//   Y[b][i][j][c*q + r] = sum_{di, dj} X~[b][s*i + di - pad][s*j + dj - pad][q] * D[di][dj][q][r]
// with X~ zero outside the image.  NHWC in, NHWC out; fp32 accumulation.
//
// Fast path (3x3, stride 1, depth multiplier 1, C a multiple of the 16-byte
// vector): each thread owns one 16-byte channel vector of one output column
// over a segment of output rows and slides a 3x3 window of input vectors down
// the image, so every input vector is fetched from L2 about (1 + 2/RS) times
// and from HBM once.  A wave covers 64 / (C / E) adjacent columns, so its
// loads of one input row are one contiguous run of pixels.  The kernel is
// HBM-bound: X is read once and Y written once.
//
// Generic path: one thread per output element, any kernel size, stride,
// padding and depth multiplier.
#include "common.hpp"
#include "kernels.hpp"

namespace isam {
namespace {

constexpr int kRowsPerSeg = 8;

template <typename T>
__device__ __forceinline__ void unpack16(uint4 v, float* f);
template <>
__device__ __forceinline__ void unpack16<bf16_t>(uint4 v, float* f) {
    f[0] = bf16lo(v.x); f[1] = bf16hi(v.x); f[2] = bf16lo(v.y); f[3] = bf16hi(v.y);
    f[4] = bf16lo(v.z); f[5] = bf16hi(v.z); f[6] = bf16lo(v.w); f[7] = bf16hi(v.w);
}
template <>
__device__ __forceinline__ void unpack16<float>(uint4 v, float* f) {
    f[0] = __uint_as_float(v.x); f[1] = __uint_as_float(v.y);
    f[2] = __uint_as_float(v.z); f[3] = __uint_as_float(v.w);
}

template <typename T, typename TY>
__device__ __forceinline__ void store_vec(TY* y, const float* acc);
template <>
__device__ __forceinline__ void store_vec<bf16_t, bf16_t>(bf16_t* y, const float* a) {
    *reinterpret_cast<uint4*>(y) = make_uint4(pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3]),
                                              pack_bf16x2(a[4], a[5]), pack_bf16x2(a[6], a[7]));
}
template <>
__device__ __forceinline__ void store_vec<bf16_t, float>(float* y, const float* a) {
    reinterpret_cast<float4*>(y)[0] = make_float4(a[0], a[1], a[2], a[3]);
    reinterpret_cast<float4*>(y)[1] = make_float4(a[4], a[5], a[6], a[7]);
}
template <>
__device__ __forceinline__ void store_vec<float, float>(float* y, const float* a) {
    *reinterpret_cast<float4*>(y) = make_float4(a[0], a[1], a[2], a[3]);
}
template <>
__device__ __forceinline__ void store_vec<float, bf16_t>(bf16_t* y, const float* a) {
    *reinterpret_cast<uint2*>(y) = make_uint2(pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3]));
}

template <typename T, typename TY>
__global__ __launch_bounds__(256) void dw3x3_s1_kernel(DwArgs a) {
    constexpr int E = 16 / (int)sizeof(T);
    const int CV = (int)(a.C / E);
    const int64_t nseg = (a.Ho + kRowsPerSeg - 1) / kRowsPerSeg;
    const int64_t total = a.batch * nseg * a.Wo * CV;
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total) return;
    const int cv = (int)(idx % CV);
    int64_t t = idx / CV;
    const int64_t j = t % a.Wo;
    t /= a.Wo;
    const int64_t seg = t % nseg;
    const int64_t b = t / nseg;
    const int64_t i0 = seg * kRowsPerSeg;
    const int64_t i1 = min(a.Ho, i0 + kRowsPerSeg);
    const int64_t c0 = (int64_t)cv * E;

    // Filter taps for these E channels, fp32.
    float w[9][E];
    const T* wp = static_cast<const T*>(a.w);
#pragma unroll
    for (int tap = 0; tap < 9; ++tap) {
        uint4 v = *reinterpret_cast<const uint4*>(wp + tap * a.C + c0);
        unpack16<T>(v, w[tap]);
    }

    const T* xp = static_cast<const T*>(a.x) + b * a.H * a.W * a.C + c0;
    // win[r][dj][e]: input rows (i - pad + r), columns (j - pad + dj)
    float win[3][3][E];
    auto load_row = [&](int64_t y, float (*dst)[E]) {
#pragma unroll
        for (int dj = 0; dj < 3; ++dj) {
            const int64_t x = j - a.pad + dj;
            if (y >= 0 && y < a.H && x >= 0 && x < a.W) {
                uint4 v = *reinterpret_cast<const uint4*>(xp + (y * a.W + x) * a.C);
                unpack16<T>(v, dst[dj]);
            } else {
#pragma unroll
                for (int e = 0; e < E; ++e) dst[dj][e] = 0.0f;
            }
        }
    };
    load_row(i0 - a.pad + 0, win[0]);
    load_row(i0 - a.pad + 1, win[1]);
    TY* yp = static_cast<TY*>(a.y) + ((b * a.Ho) * a.Wo + j) * a.C + c0;
    for (int64_t i = i0; i < i1; ++i) {
        load_row(i - a.pad + 2, win[2]);
        float acc[E];
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = 0.0f;
#pragma unroll
        for (int di = 0; di < 3; ++di)
#pragma unroll
            for (int dj = 0; dj < 3; ++dj)
#pragma unroll
                for (int e = 0; e < E; ++e) acc[e] = fmaf(win[di][dj][e], w[di * 3 + dj][e], acc[e]);
        store_vec<T, TY>(yp + i * a.Wo * a.C, acc);
#pragma unroll
        for (int dj = 0; dj < 3; ++dj)
#pragma unroll
            for (int e = 0; e < E; ++e) {
                win[0][dj][e] = win[1][dj][e];
                win[1][dj][e] = win[2][dj][e];
            }
    }
}

template <typename T>
__device__ __forceinline__ float ld1(const void* p, int64_t i) {
    if constexpr (sizeof(T) == 2) return bf16_to_f32(static_cast<const uint16_t*>(p)[i]);
    else return static_cast<const float*>(p)[i];
}

template <typename T>
__global__ __launch_bounds__(256) void dw_generic_kernel(DwArgs a) {
    const int64_t Cm = a.C * a.cm;
    const int64_t total = a.batch * a.Ho * a.Wo * Cm;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int64_t m = idx % Cm;
        int64_t t = idx / Cm;
        const int64_t j = t % a.Wo;
        t /= a.Wo;
        const int64_t i = t % a.Ho;
        const int64_t b = t / a.Ho;
        const int64_t q = m / a.cm, r = m - q * a.cm;
        float acc = 0.0f;
        for (int64_t di = 0; di < a.kh; ++di) {
            const int64_t y = a.stride * i + di - a.pad;
            if (y < 0 || y >= a.H) continue;
            for (int64_t dj = 0; dj < a.kw; ++dj) {
                const int64_t x = a.stride * j + dj - a.pad;
                if (x < 0 || x >= a.W) continue;
                acc = fmaf(ld1<T>(a.x, ((b * a.H + y) * a.W + x) * a.C + q),
                           ld1<T>(a.w, ((di * a.kw + dj) * a.C + q) * a.cm + r), acc);
            }
        }
        if (a.y_type == kF32) static_cast<float*>(a.y)[idx] = acc;
        else static_cast<uint16_t*>(a.y)[idx] = (uint16_t)f32_to_bf16(acc);
    }
}

}  // namespace

hipError_t launch_depthwise(const DwArgs& a, hipStream_t s) {
    const int E = a.in_type == kBF16 ? 8 : 4;
    const bool fast = a.kh == 3 && a.kw == 3 && a.stride == 1 && a.cm == 1 && a.C % E == 0 &&
                      (reinterpret_cast<uintptr_t>(a.x) & 15) == 0 &&
                      (reinterpret_cast<uintptr_t>(a.w) & 15) == 0 &&
                      (reinterpret_cast<uintptr_t>(a.y) & 15) == 0;
    if (fast) {
        const int64_t nseg = (a.Ho + kRowsPerSeg - 1) / kRowsPerSeg;
        const int64_t total = a.batch * nseg * a.Wo * (a.C / E);
        const dim3 grid((unsigned)((total + 255) / 256)), block(256);
        if (a.in_type == kBF16) {
            if (a.y_type == kBF16) hipLaunchKernelGGL((dw3x3_s1_kernel<bf16_t, bf16_t>), grid, block, 0, s, a);
            else hipLaunchKernelGGL((dw3x3_s1_kernel<bf16_t, float>), grid, block, 0, s, a);
        } else {
            if (a.y_type == kBF16) hipLaunchKernelGGL((dw3x3_s1_kernel<float, bf16_t>), grid, block, 0, s, a);
            else hipLaunchKernelGGL((dw3x3_s1_kernel<float, float>), grid, block, 0, s, a);
        }
    } else {
        const int64_t total = a.batch * a.Ho * a.Wo * a.C * a.cm;
        int64_t blocks = (total + 255) / 256;
        if (blocks > 65536) blocks = 65536;
        if (blocks < 1) blocks = 1;
        if (a.in_type == kBF16) hipLaunchKernelGGL(dw_generic_kernel<bf16_t>, dim3((unsigned)blocks), dim3(256), 0, s, a);
        else hipLaunchKernelGGL(dw_generic_kernel<float>, dim3((unsigned)blocks), dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

}  // namespace isam
