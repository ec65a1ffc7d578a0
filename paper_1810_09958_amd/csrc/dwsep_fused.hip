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
//      window in registers; taps are paired for v_dot2_f32_bf16), rounds it
//      to bf16 and stores it as the A tile [128][C] in LDS;
//   3. runs the product on MFMA, transposed ([256 x C] . [C x 128]: P with
//      ds_read_b64_tr_b16 as the A operand, the tile with ds_read_b128 as
//      the B operand) and writes the output channels of each pixel straight
//      from the accumulators.
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
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef unsigned u32x2_t __attribute__((vector_size(2 * sizeof(unsigned))));

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

template <int N>
__device__ __forceinline__ void f_vm_wait() {
    asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}
__device__ __forceinline__ void f_vm_wait_rt(int n) {
    switch (n) {
        case 0: f_vm_wait<0>(); break;
        case 1: f_vm_wait<1>(); break;
        case 2: f_vm_wait<2>(); break;
        case 3: f_vm_wait<3>(); break;
        default: f_vm_wait<4>(); break;
    }
}
__device__ __forceinline__ void f_barrier() {
    asm volatile("" : : : "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" : : : "memory");
}

constexpr int kFWaves = 8;
constexpr int kARegion = 32768;        // A tile (<= 128 x 128 bf16)
constexpr int kXBuf = 32768;           // bytes of one input half-tile buffer
constexpr int kXInstr = kXBuf / 1024 / kFWaves;  // copies per wave per half (4)
constexpr int kStoresPerWave = 16;     // output stores per wave per tile (MI x NI x 4)

// Persistent form: one workgroup per CU walks its tiles (tile = R output rows
// of one image).  LDS: P [C][256] (copied once) | A [128][C] | two buffers of
// one channel half of the input tile.  Per tile, all 8 waves in lockstep:
//   depthwise of channel half 0 -> A     (half 1 of this tile is landing)
//   wait, barrier; copy half 0 of the next tile
//   depthwise of channel half 1 -> A
//   barrier; copy half 1 of the next tile
//   MFMA [128 x C] . [C x 256]           (next tile's copies land meanwhile)
//   wait for next half 0, barrier; store this tile from the accumulators
template <int R, typename TO>
__global__ __launch_bounds__(64 * kFWaves) void dwsep_fused_kernel(DwArgs d, const void* pw, void* out,
                                                                   int64_t C_out) {
    extern __shared__ __attribute__((aligned(1024))) char smem[];
    const int C = (int)d.C, W = (int)d.W, H = (int)d.H;
    const int CH = C / 2;                 // channels per half
    const int UH = CH / 8;                // 16-byte units per pixel per half
    const int half_bytes = (R + 2) * W * CH * 2;
    char* sP = smem;                                   // [C][256] bf16
    char* sA = smem + C * kPRow;                       // [128][C] bf16
    char* sX0 = sA + kARegion;                         // two [R+2][W][CH] bf16 buffers
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int a_row_bytes = C * 2;
    const int tiles_per_img = (H + R - 1) / R;
    const int n_tiles = (int)d.batch * tiles_per_img;

    const __amdgpu_buffer_rsrc_t rsP = make_rsrc(pw, (uint32_t)(C * C_out * 2));
    const __amdgpu_buffer_rsrc_t rsX = make_rsrc(d.x, (uint32_t)(d.batch * (int64_t)H * W * C * 2));
    const __amdgpu_buffer_rsrc_t rsO =
        make_rsrc(out, (uint32_t)(d.batch * (int64_t)H * W * C_out * (int64_t)sizeof(TO)));

    // Copy channel half h of tile `tile`'s input rows into buffer h.
    auto copy_half = [&](int tile, int h) {
        const int b = tile / tiles_per_img, i0 = (tile % tiles_per_img) * R;
        char* dst = sX0 + h * kXBuf;
#pragma unroll
        for (int qq = 0; qq < kXInstr; ++qq) {
            const int q = wid * kXInstr + qq;
            const int unit = q * 64 + lane;              // 16-byte unit of the half tile
            const int pix = unit / UH, u = unit % UH;    // pixel index within the (R+2) x W rows
            const int rr = pix / W, x = pix % W;
            const int ir = i0 - 1 + rr;
            const bool ok = tile < n_tiles && rr < R + 2 && ir >= 0 && ir < H;
            const uint32_t off = ok ? (uint32_t)(((((int64_t)b * H + ir) * W + x) * C + h * CH + u * 8) * 2) : kOob;
            f_dma16(rsX, __builtin_amdgcn_readfirstlane(f_lds_addr(dst + q * 1024)), off);
        }
    };

    // Prologue: P once, both halves of the first tile.
    {
        const int p_instr = C * kPRow / 1024;
        for (int q = wid; q < p_instr; q += kFWaves) {
            const int unit = q * 64 + lane;
            const int k = unit / (kPRow / 16), pu = unit % (kPRow / 16);
            const int n = (((pu >> 1) ^ (k & 3)) << 4) + (pu & 1) * 8;
            const uint32_t off = (n < C_out) ? (uint32_t)((k * C_out + n) * 2) : kOob;
            f_dma16(rsP, __builtin_amdgcn_readfirstlane(f_lds_addr(sP + q * 1024)), off);
        }
    }
    int tile = blockIdx.x;
    copy_half(tile, 0);
    copy_half(tile, 1);
    f_vm_wait<0>();
    f_barrier();

    // Depthwise of one channel half into the A tile: thread tid < W*UH owns
    // item (column j, channel unit u) = (tid / UH, tid % UH) in both halves
    // (W*UH <= 512 is checked at dispatch), so its filter taps are fixed and
    // are loaded once, before the tile loop.  Taps (di, 0) and (di, 1) of
    // channel c are paired as bf16x2 for v_dot2_f32_bf16; tap (di, 2) is
    // applied with an fp32 FMA.
    const uint16_t* wp = static_cast<const uint16_t*>(d.w);
    const bool dw_item = tid < W * UH;
    const int dj_col = dw_item ? tid / UH : 0, dj_u = dw_item ? tid % UH : 0;
    uint32_t w01[2][3][8];
    float w2[2][3][8];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int cv = h * UH + dj_u;
#pragma unroll
        for (int di = 0; di < 3; ++di) {
            uint4 t0 = make_uint4(0, 0, 0, 0), t1 = t0, t2 = t0;
            if (dw_item) {
                t0 = *reinterpret_cast<const uint4*>(wp + (di * 3 + 0) * C + cv * 8);
                t1 = *reinterpret_cast<const uint4*>(wp + (di * 3 + 1) * C + cv * 8);
                t2 = *reinterpret_cast<const uint4*>(wp + (di * 3 + 2) * C + cv * 8);
            }
            const uint32_t a0[4] = {t0.x, t0.y, t0.z, t0.w}, a1[4] = {t1.x, t1.y, t1.z, t1.w},
                           a2[4] = {t2.x, t2.y, t2.z, t2.w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                w01[h][di][2 * q] = (a0[q] & 0xffffu) | (a1[q] << 16);
                w01[h][di][2 * q + 1] = (a0[q] >> 16) | (a1[q] & 0xffff0000u);
                w2[h][di][2 * q] = bf16lo(a2[q]);
                w2[h][di][2 * q + 1] = bf16hi(a2[q]);
            }
        }
    }
    auto depthwise_half = [&](auto h_c) {
        constexpr int h = decltype(h_c)::value;
        if (!dw_item) return;
        const char* xs = sX0 + h * kXBuf;
        const int j = dj_col, u = dj_u;
        const int cv = h * UH + u;  // channel vector within C
        uint32_t pr[3][8];  // sliding window of rows: (x=j-1, x=j) pairs per channel
        float sg[3][8];     // x=j+1 values per channel
        auto load_row = [&](int rr, int slot) {
            uint4 v[3];
#pragma unroll
            for (int dj = 0; dj < 3; ++dj) {
                const int x = j + dj - 1;
                v[dj] = (x >= 0 && x < W) ? *reinterpret_cast<const uint4*>(xs + ((rr * W + x) * UH + u) * 16)
                                          : make_uint4(0, 0, 0, 0);
            }
            const uint32_t b0[4] = {v[0].x, v[0].y, v[0].z, v[0].w}, b1[4] = {v[1].x, v[1].y, v[1].z, v[1].w},
                           b2[4] = {v[2].x, v[2].y, v[2].z, v[2].w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                pr[slot][2 * q] = (b0[q] & 0xffffu) | (b1[q] << 16);
                pr[slot][2 * q + 1] = (b0[q] >> 16) | (b1[q] & 0xffff0000u);
                sg[slot][2 * q] = bf16lo(b2[q]);
                sg[slot][2 * q + 1] = bf16hi(b2[q]);
            }
        };
        load_row(0, 0);
        load_row(1, 1);
#pragma unroll
        for (int rl = 0; rl < R; ++rl) {
            load_row(rl + 2, (rl + 2) % 3);
            float acc[8];
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                float a = 0.0f;
#pragma unroll
                for (int di = 0; di < 3; ++di) {
                    const int slot = (rl + di) % 3;
                    a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pr[slot][c]),
                                                        __builtin_bit_cast(bf16x2_t, w01[h][di][c]), a, false);
                    a = fmaf(sg[slot][c], w2[h][di][c], a);
                }
                acc[c] = a;
            }
            const int px = rl * W + j;
            *reinterpret_cast<uint4*>(sA + f_a_off(px, cv, a_row_bytes)) =
                make_uint4(pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]),
                           pack_bf16x2(acc[4], acc[5]), pack_bf16x2(acc[6], acc[7]));
        }
    };
    // Rows R*W .. 127 of the A tile stay zero for every tile.
    for (int q = R * W * (C / 8) + tid; q < kFBM * (C / 8); q += 64 * kFWaves)
        *reinterpret_cast<uint4*>(sA + f_a_off(q / (C / 8), q % (C / 8), a_row_bytes)) = make_uint4(0, 0, 0, 0);

    // The product is formed transposed, out^T[cout][pixel] = P^T . A^T: the
    // P fragments (read with ds_read_b64_tr_b16) are the MFMA A operand and
    // the pixel fragments of the A tile (ds_read_b128) the B operand, so each
    // accumulator holds 4 consecutive output channels of one pixel and goes
    // straight to memory as one 16-byte (fp32) or 8-byte (bf16) store.
    // Waves: 4 blocks of 64 output channels x 2 blocks of 64 pixels.
    constexpr int MI = 2, NI = 2;  // wave tile 64 couts x 64 pixels
    const int cb = wid & 3, pb = wid >> 2;
    const int g = lane >> 4, li = lane & 15;

    for (; tile < n_tiles; tile += gridDim.x) {
        const int next = tile + (int)gridDim.x;
        depthwise_half(std::integral_constant<int, 0>{});
        // Half 1 of this tile has landed once at most the previous tile's
        // kStoresPerWave stores (issued after it) are still in flight.
        if (tile == (int)blockIdx.x) f_vm_wait<0>();
        else f_vm_wait<kStoresPerWave>();
        f_barrier();
        copy_half(next, 0);
        depthwise_half(std::integral_constant<int, 1>{});
        f_barrier();               // A complete, buffer 1 free
        copy_half(next, 1);

        f32x16_t acc[MI][NI];
        static_for<MI>([&](auto i) {
            static_for<NI>([&](auto jj) {
                static_for<16>([&](auto v) { acc[i][jj][decltype(v)::value] = 0.0f; });
            });
        });
        for (int ks = 0; ks < C / 16; ++ks) {
            uint4 pf[MI], yf[NI];
            const int ch = ks * 2 + (lane >> 5);
            static_for<MI>([&](auto i) {
                const int n = cb * 64 + i * 32 + (g & 1) * 16 + 4 * (li & 3);
                uint32_t w[4];
                static_for<2>([&](auto rr) {
                    const int k = ks * 16 + (g >> 1) * 8 + rr * 4 + (li >> 2);
                    v4i16_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(sP + f_p_off(k, n)));
                    const uint2 uu = __builtin_bit_cast(uint2, v);
                    w[rr * 2] = uu.x;
                    w[rr * 2 + 1] = uu.y;
                });
                pf[i] = make_uint4(w[0], w[1], w[2], w[3]);
            });
            static_for<NI>([&](auto jj) {
                yf[jj] = *reinterpret_cast<const uint4*>(sA + f_a_off(pb * 64 + jj * 32 + (lane & 31), ch, a_row_bytes));
            });
            static_for<MI>([&](auto i) {
                static_for<NI>([&](auto jj) { mfma32_bf16(acc[i][jj], pf[i], yf[jj]); });
            });
        }
        // Every wave is done reading the A tile before the next depthwise
        // overwrites it; the next tile's half 0 (issued before this wave's
        // half-1 copies) has landed.
        f_vm_wait<kXInstr>();
        f_barrier();

        // Store: accumulator element v of lane l is output channel
        // cb*64 + i*32 + 8*(v/4) + 4*(l/32) + v%4 of pixel pb*64 + jj*32 + l%32.
        // Every lane issues its stores (pixels past the tile's valid rows and
        // channels past C_out go to an offset beyond the buffer and are
        // dropped), so each wave issues exactly kStoresPerWave.
        const int b = tile / tiles_per_img, i0 = (tile % tiles_per_img) * R;
        const int valid_rows = min(R, H - i0) * W;
        const int64_t m0 = ((int64_t)b * H + i0) * W;
        static_for<MI>([&](auto i) {
            static_for<NI>([&](auto jj) {
                static_for<4>([&](auto v4c) {
                    constexpr int v4 = decltype(v4c)::value;
                    const int px = pb * 64 + jj * 32 + (lane & 31);
                    const int64_t co = cb * 64 + i * 32 + 8 * v4 + 4 * (lane >> 5);
                    const bool ok = px < valid_rows && co < C_out;
                    const int64_t idx = (m0 + px) * C_out + co;
                    const float x0 = acc[i][jj][4 * v4], x1 = acc[i][jj][4 * v4 + 1];
                    const float x2 = acc[i][jj][4 * v4 + 2], x3 = acc[i][jj][4 * v4 + 3];
                    if constexpr (sizeof(TO) == 4)
                        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4_t, make_float4(x0, x1, x2, x3)), rsO,
                                                               ok ? (int)(idx * 4) : (int)kOob, 0, 0);
                    else
                        __builtin_amdgcn_raw_buffer_store_b64(
                            __builtin_bit_cast(u32x2_t, make_uint2(pack_bf16x2(x0, x1), pack_bf16x2(x2, x3))), rsO,
                            ok ? (int)(idx * 2) : (int)kOob, 0, 0);
                });
            });
        });
    }
    f_vm_wait<0>();
}

template <int R>
size_t fused_lds(const DwArgs& d) {
    return (size_t)d.C * kPRow + (size_t)kARegion + 2 * (size_t)kXBuf;
}

}  // namespace

// Rows per tile for this shape, or 0 when the fused kernel does not apply.
int dwsep_fused_rows(const DwArgs& d, int64_t C_out, int lds_max) {
    if (d.in_type != kBF16 || d.kh != 3 || d.kw != 3 || d.stride != 1 || d.pad != 1 || d.cm != 1) return 0;
    // C in {64, 128}: 8 or 16 chunks per A-tile row, as the XOR swizzle needs
    if (d.C % 64 || d.C > 128 || C_out % 8 || C_out > kFBN) return 0;
    if (d.batch * d.H * d.W * d.C * 2 > (int64_t(1) << 31) - 1) return 0;
    if ((reinterpret_cast<uintptr_t>(d.x) & 15) || (reinterpret_cast<uintptr_t>(d.w) & 15)) return 0;
    const int r = d.W <= 32 ? 4 : d.W <= 64 ? 2 : 0;
    if (!r) return 0;
    // one channel half of the R+2 input rows must fit one copy buffer
    if ((int64_t)(r + 2) * d.W * (d.C / 2) * 2 > kXBuf) return 0;
    const size_t lds = r == 4 ? fused_lds<4>(d) : fused_lds<2>(d);
    if (lds > (size_t)lds_max) return 0;
    return r;
}

hipError_t launch_dwsep_fused(const DwArgs& d, const void* pw, void* out, int64_t C_out, int out_type, int R,
                              int cus, hipStream_t s) {
    const size_t lds = R == 4 ? fused_lds<4>(d) : fused_lds<2>(d);
    const int tiles = (int)(d.batch * ((d.H + R - 1) / R));
    const int grid = tiles < cus ? tiles : cus;
    void* fn = nullptr;
    if (R == 4)
        fn = out_type == kF32 ? reinterpret_cast<void*>(dwsep_fused_kernel<4, float>)
                              : reinterpret_cast<void*>(dwsep_fused_kernel<4, uint16_t>);
    else
        fn = out_type == kF32 ? reinterpret_cast<void*>(dwsep_fused_kernel<2, float>)
                              : reinterpret_cast<void*>(dwsep_fused_kernel<2, uint16_t>);
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    DwArgs dd = d;
    void* args[] = {&dd, const_cast<void**>(&pw), &out, &C_out};
    return hipLaunchKernel(fn, dim3(grid), dim3(64 * kFWaves), args, lds, s);
}

}  // namespace isam
