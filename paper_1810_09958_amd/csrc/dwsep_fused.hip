// Fused separable depthwise convolution (bf16 inputs): the third listing of
// the paper, factored as in Section 2.3 into a 3x3 depthwise stencil followed
// by the pointwise matrix product, with the intermediate kept on chip -- the
// inter-operation fusion the paper credits for its GRU results
// (Section 6.2.2) applied to this layer.
//
// One workgroup produces R full output rows of one image (R*W pixels, padded
// to 128 MFMA rows) for all C_out channels:
//   1. copies P ([C][C_out], padded to 256 columns) and the R+2 input rows it
//      needs (contiguous in NHWC; rows outside the image arrive as zeros)
//      into LDS with buffer_load ... lds;
//   2. computes the depthwise result for its pixels in fp32 from LDS (each
//      thread owns one channel vector of one column and reuses the vertical
//      window in registers), rounds it to bf16 and stores it as the A tile
//      [128][C] in LDS;
//   3. runs the [128 x C] . [C x 256] product on MFMA (A with ds_read_b128,
//      P with ds_read_b64_tr_b16) and writes the output tile.
// Supported: bf16 input, 3x3, stride 1, pad 1, depth multiplier 1,
// C in {64, 128}, C_out % 8 == 0, C_out <= 256, W <= 128 / R, and
// the LDS footprint within the device limit; everything else uses the
// two-kernel path.
#include "common.hpp"
#include "gemm_impl.hpp"
#include "kernels.hpp"

namespace isam {
namespace {

typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16_t lds_v4i16_t;

constexpr int kFBM = 128;     // MFMA rows per workgroup
constexpr int kFBN = 256;     // output channels per workgroup (padded)
constexpr int kPRow = kFBN * 2;  // bytes of one P row in LDS

__device__ __forceinline__ void f_dma16(__amdgpu_buffer_rsrc_t rs, uint32_t lds_addr, uint32_t voff) {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %1, %2, 0 offen lds"
        :
        : "s"(lds_addr), "v"(voff), "s"(rs)
        : "memory", "m0");
}
__device__ __forceinline__ uint32_t f_lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}
// A tile [128][C] bf16: 16-byte chunk c of row r at chunk c ^ (r & 7).
__device__ __forceinline__ uint32_t f_a_off(int r, int c, int row_bytes) {
    return (uint32_t)(r * row_bytes + ((c ^ (r & 7)) << 4));
}
// P rows [k][256] bf16: 32-byte block b of row k at block b ^ (k & 3).
__device__ __forceinline__ uint32_t f_p_off(int k, int n) {
    return (uint32_t)(k * kPRow + ((((n >> 4) ^ (k & 3))) << 5) + (n & 15) * 2);
}

template <int R, typename TO>
__global__ __launch_bounds__(256) void dwsep_fused_kernel(DwArgs d, const void* pw, void* out, int64_t C_out,
                                                          int out_type) {
    extern __shared__ __attribute__((aligned(1024))) char smem[];
    const int C = (int)d.C, W = (int)d.W, H = (int)d.H;
    const int CV = C / 8;                       // 16-byte channel vectors per pixel
    const int pix_bytes = C * 2;
    const int xrow_bytes = W * pix_bytes;
    const int xt_bytes = (R + 2) * xrow_bytes;
    char* sP = smem;                                  // [C][256] bf16
    char* sX = smem + C * kPRow;                      // [R+2][W][C] bf16
    char* sA = sX + ((xt_bytes + 1023) & ~1023);      // [128][C] bf16
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;

    // Tile: image b, output rows i0 .. i0+R-1.  Consecutive tiles of one
    // image go to one XCD (dispatch is round robin over the 8 XCDs), so the
    // halo rows two tiles share are reused from that XCD's L2.
    int bid = blockIdx.x;
    const int G = gridDim.x;
    if ((G & 7) == 0) bid = (bid & 7) * (G >> 3) + (bid >> 3);
    const int tiles_per_img = (H + R - 1) / R;
    const int b = bid / tiles_per_img, i0 = (bid % tiles_per_img) * R;

    // 1. Copies: P, then the input rows i0-1 .. i0+R.
    const __amdgpu_buffer_rsrc_t rsP = make_rsrc(pw, (uint32_t)(C * C_out * 2));
    const __amdgpu_buffer_rsrc_t rsX = make_rsrc(d.x, (uint32_t)(d.batch * (int64_t)H * W * C * 2));
    {
        const int p_instr = C * kPRow / 1024;  // C/2 copies of 1 KiB
        for (int q = wid; q < p_instr; q += 4) {
            const int unit = q * 64 + lane;        // 16-byte unit of the P region
            const int k = unit / (kPRow / 16), pu = unit % (kPRow / 16);
            const int n = (((pu >> 1) ^ (k & 3)) << 4) + (pu & 1) * 8;
            const uint32_t off = (n < C_out) ? (uint32_t)((k * C_out + n) * 2) : kOob;
            f_dma16(rsP, __builtin_amdgcn_readfirstlane(f_lds_addr(sP + q * 1024)), off);
        }
        const int x_instr = (xt_bytes + 1023) / 1024;
        const int64_t row0 = (int64_t)b * H + i0 - 1;  // global image row of tile row 0
        for (int q = wid; q < x_instr; q += 4) {
            const int o = q * 1024 + lane * 16;
            const int tr = o / xrow_bytes;
            const int64_t ir = i0 - 1 + tr;
            const bool ok = o < xt_bytes && ir >= 0 && ir < H;
            const uint32_t off = ok ? (uint32_t)((row0 * xrow_bytes) + o) : kOob;
            f_dma16(rsX, __builtin_amdgcn_readfirstlane(f_lds_addr(sX + q * 1024)), off);
        }
    }

    // Depthwise filter of this thread's channel vector, fp32 (taps di*3+dj).
    const int cv = tid % CV;
    const int jstep = 256 / CV;
    float wv[9][8];
    {
        const uint16_t* wp = static_cast<const uint16_t*>(d.w);
#pragma unroll
        for (int tap = 0; tap < 9; ++tap) {
            const uint4 v = *reinterpret_cast<const uint4*>(wp + tap * C + cv * 8);
            wv[tap][0] = bf16lo(v.x); wv[tap][1] = bf16hi(v.x); wv[tap][2] = bf16lo(v.y); wv[tap][3] = bf16hi(v.y);
            wv[tap][4] = bf16lo(v.z); wv[tap][5] = bf16hi(v.z); wv[tap][6] = bf16lo(v.w); wv[tap][7] = bf16hi(v.w);
        }
    }
    __builtin_amdgcn_s_waitcnt(0);  // every copy of this wave has landed
    __syncthreads();

    // 2. Depthwise into the A tile.  Rows R*W .. 127 of the tile are zero.
    const int a_row_bytes = C * 2;
    // every (column, channel vector) pair has exactly one owner thread
    for (int j = tid / CV; tid < CV * jstep && j < W; j += jstep) {
        float col[R + 2][3][8];
#pragma unroll
        for (int rr = 0; rr < R + 2; ++rr)
#pragma unroll
            for (int dj = 0; dj < 3; ++dj) {
                const int x = j + dj - 1;
                if (x >= 0 && x < W) {
                    const uint4 v = *reinterpret_cast<const uint4*>(sX + rr * xrow_bytes + x * pix_bytes + cv * 16);
                    col[rr][dj][0] = bf16lo(v.x); col[rr][dj][1] = bf16hi(v.x);
                    col[rr][dj][2] = bf16lo(v.y); col[rr][dj][3] = bf16hi(v.y);
                    col[rr][dj][4] = bf16lo(v.z); col[rr][dj][5] = bf16hi(v.z);
                    col[rr][dj][6] = bf16lo(v.w); col[rr][dj][7] = bf16hi(v.w);
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e) col[rr][dj][e] = 0.0f;
                }
            }
#pragma unroll
        for (int rl = 0; rl < R; ++rl) {
            float acc[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[e] = 0.0f;
#pragma unroll
            for (int di = 0; di < 3; ++di)
#pragma unroll
                for (int dj = 0; dj < 3; ++dj)
#pragma unroll
                    for (int e = 0; e < 8; ++e) acc[e] = fmaf(col[rl + di][dj][e], wv[di * 3 + dj][e], acc[e]);
            const int px = rl * W + j;
            // rows past the image bottom are computed from zero input and never stored
            *reinterpret_cast<uint4*>(sA + f_a_off(px, cv, a_row_bytes)) =
                make_uint4(pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]),
                           pack_bf16x2(acc[4], acc[5]), pack_bf16x2(acc[6], acc[7]));
        }
    }
    for (int q = R * W * CV + tid; q < kFBM * CV; q += 256)
        *reinterpret_cast<uint4*>(sA + f_a_off(q / CV, q % CV, a_row_bytes)) = make_uint4(0, 0, 0, 0);
    __syncthreads();

    // 3. MFMA: waves 2x2 over the 128 x 256 tile, 64 x 128 each.
    constexpr int MI = 2, NI = 4;
    const int wm = wid >> 1, wn = wid & 1;
    f32x16_t acc[MI][NI];
    static_for<MI>([&](auto i) {
        static_for<NI>([&](auto jj) {
            static_for<16>([&](auto v) { acc[i][jj][decltype(v)::value] = 0.0f; });
        });
    });
    const int g = lane >> 4, li = lane & 15;
    for (int ks = 0; ks < C / 16; ++ks) {
        uint4 af[MI], bfr[NI];
        const int ch = ks * 2 + (lane >> 5);
        static_for<MI>([&](auto i) {
            af[i] = *reinterpret_cast<const uint4*>(sA + f_a_off(wm * 64 + i * 32 + (lane & 31), ch, a_row_bytes));
        });
        static_for<NI>([&](auto jj) {
            const int n = wn * 128 + jj * 32 + (g & 1) * 16 + 4 * (li & 3);
            uint32_t w[4];
            static_for<2>([&](auto rr) {
                const int k = ks * 16 + (g >> 1) * 8 + rr * 4 + (li >> 2);
                v4i16_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(sP + f_p_off(k, n)));
                const uint2 u = __builtin_bit_cast(uint2, v);
                w[rr * 2] = u.x;
                w[rr * 2 + 1] = u.y;
            });
            bfr[jj] = make_uint4(w[0], w[1], w[2], w[3]);
        });
        static_for<MI>([&](auto i) {
            static_for<NI>([&](auto jj) { mfma32_bf16(acc[i][jj], af[i], bfr[jj]); });
        });
    }
    __syncthreads();

    // 4. Epilogue through LDS (the X and A regions are free now): output rows
    //    are the tile's pixels, contiguous in NHWC.
    constexpr int WTN = 128;
    constexpr int EPI_LD = WTN * 4 + 16;
    char* epi = sX + wid * 32 * EPI_LD;
    const int valid_rows = min(R, H - i0) * W;
    const int64_t m0 = ((int64_t)b * H + i0) * W;
    constexpr int Q = WTN / 4;
    static_for<MI>([&](auto i) {
        static_for<NI>([&](auto jj) {
            static_for<16>([&](auto v) {
                constexpr int vv = decltype(v)::value;
                const int r = 8 * (vv >> 2) + 4 * (lane >> 5) + (vv & 3);
                *reinterpret_cast<float*>(epi + r * EPI_LD + (jj * 32 + (lane & 31)) * 4) = acc[i][jj][vv];
            });
        });
        __syncthreads();
        for (int q = lane; q < 32 * Q; q += 64) {
            const int r = q / Q, c4 = q - r * Q;
            const int prow = wm * 64 + i * 32 + r;
            const int64_t col = wn * WTN + c4 * 4;
            if (prow >= valid_rows || col >= C_out) continue;
            const float4 v4 = *reinterpret_cast<const float4*>(epi + r * EPI_LD + c4 * 16);
            const int64_t idx = (m0 + prow) * C_out + col;  // C_out % 8 == 0: whole float4 in range
            if constexpr (sizeof(TO) == 4) {
                *reinterpret_cast<float4*>(static_cast<float*>(out) + idx) = v4;
            } else {
                *reinterpret_cast<uint2*>(static_cast<uint16_t*>(out) + idx) =
                    make_uint2(pack_bf16x2(v4.x, v4.y), pack_bf16x2(v4.z, v4.w));
            }
        }
        __syncthreads();
    });
}

template <int R>
size_t fused_lds(const DwArgs& d) {
    const size_t xt = (size_t)(R + 2) * d.W * d.C * 2;
    return (size_t)d.C * kPRow + ((xt + 1023) & ~(size_t)1023) + (size_t)kFBM * d.C * 2;
}

}  // namespace

// Rows per tile for this shape, or 0 when the fused kernel does not apply.
int dwsep_fused_rows(const DwArgs& d, int64_t C_out, int lds_max) {
    if (d.in_type != kBF16 || d.kh != 3 || d.kw != 3 || d.stride != 1 || d.pad != 1 || d.cm != 1) return 0;
    // C in {64, 128}: 8 or 16 chunks per A-tile row, as the XOR swizzle needs
    if (d.C % 64 || d.C > 128 || C_out % 8 || C_out > kFBN) return 0;
    if (d.batch * d.H * d.W * d.C * 2 > (int64_t(1) << 31) - 1) return 0;
    if ((reinterpret_cast<uintptr_t>(d.x) & 15) || (reinterpret_cast<uintptr_t>(d.w) & 15)) return 0;
    const int r = d.W <= 32 ? 4 : d.W <= 64 ? 2 : d.W <= 128 ? 1 : 0;
    if (!r) return 0;
    const size_t lds = r == 4 ? fused_lds<4>(d) : r == 2 ? fused_lds<2>(d) : fused_lds<1>(d);
    // epilogue staging (4 waves x 32 rows) reuses the X and A regions
    const size_t epi = 4 * 32 * (128 * 4 + 16);
    const size_t xa = lds - (size_t)d.C * kPRow;
    if (lds > (size_t)lds_max || epi > xa) return 0;
    return r;
}

hipError_t launch_dwsep_fused(const DwArgs& d, const void* pw, void* out, int64_t C_out, int out_type, int R,
                              hipStream_t s) {
    const size_t lds = R == 4 ? fused_lds<4>(d) : R == 2 ? fused_lds<2>(d) : fused_lds<1>(d);
    const int tiles = (int)(d.batch * ((d.H + R - 1) / R));
    void* fn = nullptr;
#define ISAM_FUSED_FN(RR)                                                                        \
    fn = out_type == kF32 ? reinterpret_cast<void*>(dwsep_fused_kernel<RR, float>)               \
                          : reinterpret_cast<void*>(dwsep_fused_kernel<RR, uint16_t>)
    if (R == 4) ISAM_FUSED_FN(4);
    else if (R == 2) ISAM_FUSED_FN(2);
    else ISAM_FUSED_FN(1);
#undef ISAM_FUSED_FN
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    DwArgs dd = d;
    void* args[] = {&dd, const_cast<void**>(&pw), &out, &C_out, &out_type};
    return hipLaunchKernel(fn, dim3(tiles), dim3(256), args, lds, s);
}

}  // namespace isam
