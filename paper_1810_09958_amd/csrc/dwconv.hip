// Depthwise half of the separable depthwise convolution (the paper's third
// listing, after the pointwise weight is factored out of the (di, dj)
// reduction, Section 2.3):
//   Y[b][i][j][c*q + r] = sum_{di, dj} X~[b][s*i + di - pad][s*j + dj - pad][q] * D[di][dj][q][r]
// with X~ zero outside the image.  NHWC in, NHWC out; fp32 accumulation.
//
// Fast paths (3x3, stride 1, depth multiplier 1, C a multiple of the 16-byte
// vector): with padding 1 and a pixel's channel vectors fitting one workgroup,
// the LDS-staged kernel below (dw3x3_lds_kernel); otherwise the register-window
// kernel: each thread owns one 16-byte channel vector of one output column
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

#include <algorithm>
#include <cstdlib>

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

// LDS-staged 3x3 stride-1 pad-1 kernel.  A workgroup owns RS output rows x
// SW output columns x all C channels of one image; thread (column cc, channel
// vector v) computes its column over the RS rows.  The input block it needs --
// RS+2 rows x SW+2 columns x C, rows and columns outside the image as zeros --
// is one contiguous run of SW+2 pixels per row in NHWC, so it is copied straight
// into LDS with buffer_load ... lds (64 consecutive 16-byte units per
// instruction; out-of-image units are fetched at an out-of-range offset and
// land as zeros), after the 9 x C filter taps, all copies of the workgroup at
// once.  Each thread then slides its 3x3 window down its column, reading three
// 16-byte LDS vectors per output row (a wave's 64 lanes read 64 consecutive
// units: conflict-free); the three window rows rotate through three register
// slots (the row loop is unrolled by three), so no values are moved.  bf16
// input: each window row is kept as (x-1, x) bf16 pairs per channel plus x+1
// in fp32, and an output channel is three v_dot2_f32_bf16 (the (dj 0, dj 1)
// tap pairs) and three FMAs (dj 2), di by di; fp32 input: nine FMAs in (di, dj)
// order.  The stores of one output row are one contiguous run of SW pixels.
__device__ __forceinline__ void dw_dma16(__amdgpu_buffer_rsrc_t rs, uint32_t lds_addr, uint32_t voff) {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %1, %2, 0 offen lds"
        :
        : "s"(lds_addr), "v"(voff), "s"(rs)
        : "memory", "m0");
}

typedef __bf16 dw_bf16x2_t __attribute__((ext_vector_type(2)));
typedef float dw_f32x2_t __attribute__((ext_vector_type(2)));
// Two fp32 values to a bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t dw_pack_bf16(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((dw_f32x2_t){lo, hi}, dw_bf16x2_t));
}

// Window row of one thread: bf16 -> (x-1, x) pairs + x+1 in fp32; fp32 -> the
// three vectors.
template <typename T>
struct DwSlot;
template <>
struct DwSlot<bf16_t> {
    uint32_t pr[8];
    float sg[8];
    __device__ __forceinline__ void load(const uint4* p, int stride) {
        const uint4 b0 = p[0], b1 = p[stride], b2 = p[2 * stride];
        const uint32_t a0[4] = {b0.x, b0.y, b0.z, b0.w}, a1[4] = {b1.x, b1.y, b1.z, b1.w},
                       a2[4] = {b2.x, b2.y, b2.z, b2.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            pr[2 * q] = __builtin_amdgcn_perm(a1[q], a0[q], 0x05040100u);
            pr[2 * q + 1] = __builtin_amdgcn_perm(a1[q], a0[q], 0x07060302u);
            sg[2 * q] = bf16lo(a2[q]);
            sg[2 * q + 1] = bf16hi(a2[q]);
        }
    }
};
template <>
struct DwSlot<float> {
    float x[3][4];
    __device__ __forceinline__ void load(const uint4* p, int stride) {
#pragma unroll
        for (int dj = 0; dj < 3; ++dj) unpack16<float>(p[dj * stride], x[dj]);
    }
};

// Taps of one thread's channels, laid out to match its window slots.
template <typename T>
struct DwTaps;
template <>
struct DwTaps<bf16_t> {
    uint32_t w01[3][8];
    float w2[3][8];
    __device__ __forceinline__ void load(const uint4* taps, int CV, int v) {
#pragma unroll
        for (int di = 0; di < 3; ++di) {
            const uint4 t0 = taps[(di * 3 + 0) * CV + v], t1 = taps[(di * 3 + 1) * CV + v],
                        t2 = taps[(di * 3 + 2) * CV + v];
            const uint32_t a0[4] = {t0.x, t0.y, t0.z, t0.w}, a1[4] = {t1.x, t1.y, t1.z, t1.w},
                           a2[4] = {t2.x, t2.y, t2.z, t2.w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                w01[di][2 * q] = __builtin_amdgcn_perm(a1[q], a0[q], 0x05040100u);
                w01[di][2 * q + 1] = __builtin_amdgcn_perm(a1[q], a0[q], 0x07060302u);
                w2[di][2 * q] = bf16lo(a2[q]);
                w2[di][2 * q + 1] = bf16hi(a2[q]);
            }
        }
    }
    // out[c] for window rows (top, mid, bottom)
    __device__ __forceinline__ void apply(const DwSlot<bf16_t>& r0, const DwSlot<bf16_t>& r1,
                                          const DwSlot<bf16_t>& r2, float* out) const {
        const DwSlot<bf16_t>* rows[3] = {&r0, &r1, &r2};
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            float a = 0.0f;
#pragma unroll
            for (int di = 0; di < 3; ++di) {
                a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(dw_bf16x2_t, rows[di]->pr[c]),
                                                    __builtin_bit_cast(dw_bf16x2_t, w01[di][c]), a, false);
                a = fmaf(rows[di]->sg[c], w2[di][c], a);
            }
            out[c] = a;
        }
    }
};
template <>
struct DwTaps<float> {
    float w[9][4];
    __device__ __forceinline__ void load(const uint4* taps, int CV, int v) {
#pragma unroll
        for (int tap = 0; tap < 9; ++tap) unpack16<float>(taps[tap * CV + v], w[tap]);
    }
    __device__ __forceinline__ void apply(const DwSlot<float>& r0, const DwSlot<float>& r1,
                                          const DwSlot<float>& r2, float* out) const {
        const DwSlot<float>* rows[3] = {&r0, &r1, &r2};
#pragma unroll
        for (int e = 0; e < 4; ++e) out[e] = 0.0f;
#pragma unroll
        for (int di = 0; di < 3; ++di)
#pragma unroll
            for (int dj = 0; dj < 3; ++dj)
#pragma unroll
                for (int e = 0; e < 4; ++e) out[e] = fmaf(rows[di]->x[dj][e], w[di * 3 + dj][e], out[e]);
    }
};

template <typename T, typename TY>
__device__ __forceinline__ void dw_store(TY* y, const float* a) {
    constexpr int E = 16 / (int)sizeof(T);
    if constexpr (sizeof(TY) == 2) {
        if constexpr (E == 8)
            *reinterpret_cast<uint4*>(y) = make_uint4(dw_pack_bf16(a[0], a[1]), dw_pack_bf16(a[2], a[3]),
                                                      dw_pack_bf16(a[4], a[5]), dw_pack_bf16(a[6], a[7]));
        else
            *reinterpret_cast<uint2*>(y) = make_uint2(dw_pack_bf16(a[0], a[1]), dw_pack_bf16(a[2], a[3]));
    } else {
#pragma unroll
        for (int q = 0; q < E / 4; ++q)
            reinterpret_cast<float4*>(y)[q] = make_float4(a[4 * q], a[4 * q + 1], a[4 * q + 2], a[4 * q + 3]);
    }
}

constexpr int kDwLdsThreads = 256;

template <typename T, typename TY>
__global__ __launch_bounds__(kDwLdsThreads) void dw3x3_lds_kernel(DwArgs a, int RS, int SW) {
    extern __shared__ __attribute__((aligned(1024))) char dw_lds[];
    constexpr int E = 16 / (int)sizeof(T);
    constexpr int NW = kDwLdsThreads / 64;
    const int CV = (int)(a.C / E);
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int64_t nstrip = (a.Wo + SW - 1) / SW, nseg = (a.Ho + RS - 1) / RS;
    // Workgroups are dispatched round-robin over the 8 XCDs; give each XCD a
    // contiguous range of blocks, so blocks that share halo rows and columns
    // run on one L2 at about the same time.
    int64_t u = blockIdx.x;
    if (gridDim.x % 8 == 0) u = (u % 8) * (gridDim.x / 8) + u / 8;
    const int64_t strip = u % nstrip;
    u /= nstrip;
    const int64_t seg = u % nseg;
    const int64_t b = u / nseg;
    const int64_t i0 = seg * RS, x0 = strip * SW;
    const uint32_t base = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)dw_lds;

    // 1. Copies: taps [9][CV] units first, then input rows i0-1 .. i0+RS,
    //    columns x0-1 .. x0+SW as [row][column][vector] units.
    const int tap_units = 9 * CV, tap_copies = (tap_units + 63) / 64;
    const __amdgpu_buffer_rsrc_t rsW = make_rsrc(a.w, (uint32_t)(tap_units * 16));
    for (int q = wid; q < tap_copies; q += NW) {
        const int unit = q * 64 + lane;
        dw_dma16(rsW, __builtin_amdgcn_readfirstlane(base + (uint32_t)q * 1024u),
                 unit < tap_units ? (uint32_t)unit * 16u : kOob);
    }
    const int upr = (SW + 2) * CV;  // units per LDS row
    const int units = (RS + 2) * upr;
    const int ncopy = (units + 63) / 64;
    const int64_t img = a.H * a.W * a.C;  // elements of one image
    const __amdgpu_buffer_rsrc_t rsX =
        make_rsrc(static_cast<const T*>(a.x) + b * img, (uint32_t)(img * (int64_t)sizeof(T)));
    const uint32_t xbase = base + (uint32_t)tap_copies * 1024u;
    for (int q = wid; q < ncopy; q += NW) {
        const int unit = q * 64 + lane;
        const int r = unit / upr, rem = unit - r * upr;
        const int cc = rem / CV, v = rem - cc * CV;
        const int64_t y = i0 - 1 + r, x = x0 - 1 + cc;
        const bool in = unit < units && y >= 0 && y < a.H && x >= 0 && x < a.W;
        const uint32_t off = in ? (uint32_t)(((y * a.W + x) * a.C + (int64_t)v * E) * (int64_t)sizeof(T)) : kOob;
        dw_dma16(rsX, __builtin_amdgcn_readfirstlane(xbase + (uint32_t)q * 1024u), off);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();

    // 2. The stencil, one output row per step, window rows in rotating slots.
    const int cc = tid / CV, v = tid - cc * CV;
    if (cc >= SW || x0 + cc >= a.Wo) return;
    DwTaps<T> taps;
    taps.load(reinterpret_cast<const uint4*>(dw_lds), CV, v);
    const uint4* L = reinterpret_cast<const uint4*>(dw_lds + tap_copies * 1024) + cc * CV + v;
    const int rows = (int)min((int64_t)RS, a.Ho - i0);
    TY* yp = static_cast<TY*>(a.y) + ((b * a.Ho + i0) * a.Wo + x0 + cc) * a.C + (int64_t)v * E;
    const int64_t ystride = a.Wo * a.C;
    DwSlot<T> s0, s1, s2;
    s0.load(L, CV);
    s1.load(L + upr, CV);
    float acc[E];
    int i = 0;
    for (; i + 3 <= rows; i += 3) {
        s2.load(L + (i + 2) * upr, CV);
        taps.apply(s0, s1, s2, acc);
        dw_store<T, TY>(yp + i * ystride, acc);
        s0.load(L + (i + 3) * upr, CV);
        taps.apply(s1, s2, s0, acc);
        dw_store<T, TY>(yp + (i + 1) * ystride, acc);
        s1.load(L + (i + 4) * upr, CV);
        taps.apply(s2, s0, s1, acc);
        dw_store<T, TY>(yp + (i + 2) * ystride, acc);
    }
    if (i < rows) {
        s2.load(L + (i + 2) * upr, CV);
        taps.apply(s0, s1, s2, acc);
        dw_store<T, TY>(yp + i * ystride, acc);
    }
    if (i + 1 < rows) {
        s0.load(L + (i + 3) * upr, CV);
        taps.apply(s1, s2, s0, acc);
        dw_store<T, TY>(yp + (i + 1) * ystride, acc);
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
    // LDS-staged path: 3x3 stride-1 pad-1, a channel-vector count that fits
    // one workgroup, and images addressable with 32-bit offsets.
    const int64_t CV = a.C / E;
    const int64_t es = a.in_type == kBF16 ? 2 : 4;
    // Rows per workgroup (measured on the 32x56x56x128 image batch: bf16 10 rows
    // 16.6 us against 17-18 for 4-8; fp32 4 rows 26.5 us against 28-30 for 8-14);
    // ISAM_DW_RS overrides, 0 takes the register-window kernel.
    const char* rs_env = getenv("ISAM_DW_RS");
    const int rs_sel = rs_env ? atoi(rs_env) : (a.in_type == kBF16 ? 10 : 4);
    if (fast && a.pad == 1 && rs_sel > 0 && CV <= kDwLdsThreads && a.H * a.W * a.C * es < (1ll << 31)) {
        const int64_t per = kDwLdsThreads / CV;                 // columns one workgroup can own
        const int64_t nstrip = (a.Wo + per - 1) / per;
        const int SW = (int)((a.Wo + nstrip - 1) / nstrip);     // balanced strips
        // rows per workgroup: the requested count, fewer if the block would
        // take more than 64 KB of LDS (at least two workgroups per CU)
        auto lds_for = [&](int64_t rs) { return (size_t)((9 * CV + 63) / 64 + ((rs + 2) * (SW + 2) * CV + 63) / 64) * 1024; };
        int RS = (int)std::min<int64_t>(rs_sel, a.Ho);
        while (RS > 1 && lds_for(RS) > 64 * 1024) --RS;
        const size_t lds = lds_for(RS);
        if (lds <= 64 * 1024) {
            const int64_t nseg = (a.Ho + RS - 1) / RS;
            const dim3 grid((unsigned)(a.batch * nseg * nstrip)), block(kDwLdsThreads);
            // at most 64 KB of dynamic LDS: within the default limit, no attribute needed
            if (a.in_type == kBF16) {
                if (a.y_type == kBF16) hipLaunchKernelGGL((dw3x3_lds_kernel<bf16_t, bf16_t>), grid, block, lds, s, a, RS, SW);
                else hipLaunchKernelGGL((dw3x3_lds_kernel<bf16_t, float>), grid, block, lds, s, a, RS, SW);
            } else {
                if (a.y_type == kBF16) hipLaunchKernelGGL((dw3x3_lds_kernel<float, bf16_t>), grid, block, lds, s, a, RS, SW);
                else hipLaunchKernelGGL((dw3x3_lds_kernel<float, float>), grid, block, lds, s, a, RS, SW);
            }
            return hipGetLastError();
        }
    }
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
