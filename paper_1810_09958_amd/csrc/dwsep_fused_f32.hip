// Fused separable depthwise convolution, fp32 end to end: the third listing
// of the paper factored as in Section 2.3 (3x3 depthwise, then the pointwise
// matrix product), with the depthwise result kept on chip as the operand of
// the product (the inter-operation fusion of Section 6.2.2).
//
// The pointwise product keeps fp32 accuracy without the fp32 matrix rate:
// every fp32 operand x is split into three bf16 terms, x = h + m + l + e
// (h = bf16(x), m = bf16(x - h), l = bf16(x - h - m); each difference is
// exact in fp32 and |e| <= 2^-24 |x|), and a.b is formed as the six bf16
// products h.h + h.m + m.h + h.l + l.h + m.m with fp32 accumulation on the
// bf16 matrix cores (v_mfma_f32_16x16x32_bf16, 16 times the fp32 MFMA
// rate).  The dropped terms m.l, l.m, l.l are below 2^-23 |a.b|, the same
// order as the rounding of one fp32 product.  The product is computed
// transposed, out^T[cout][pixel] = P^T[cout][k] . Y^T[k][pixel]:
//   * each wave owns 32 output channels; the three bf16 terms of its slice
//     of P (32 x C) live in registers for the whole kernel as MFMA A
//     operands;
//   * the depthwise result Y of a tile (R output rows x W pixels) is built
//     in LDS one 32-channel chunk at a time, as three bf16 term planes, and
//     read as MFMA B operands with ds_read_b128 (8 consecutive channels of
//     one pixel per lane);
//   * the accumulators hold 4 consecutive output channels of one pixel per
//     lane, so results go straight from registers to memory as 16-byte
//     stores.
// Per tile (persistent workgroups walk the tiles), per 32-channel chunk c:
//   wait for chunk c's input copies, barrier
//   issue the copies of the next chunk (direct to LDS, other buffer)
//   depthwise of chunk c -> Y chunk in LDS, barrier
//   MFMAs over the chunk
// Input chunk layout: [R+2 rows][W][32 channels] fp32 (128 bytes per pixel,
// one whole cache line per copied segment).  Y chunk layout: term t, channel
// unit u (8 channels), pixel p: 16 bytes at t*kYTerm + u*kYUnit + p*16.  The
// B-operand reads of 16 lanes take 16 consecutive pixels of one unit (256
// contiguous bytes); the unit stride is 64 bytes past a multiple of 256 so
// that the depthwise writes of a wave (8 pixels x 4 units x 2 halves) fall on
// distinct banks.
// Supported: fp32 in and out, 3x3, stride 1, pad 1, depth multiplier 1,
// C % 32 == 0 and C <= 128, C_out % 16 == 0 and C_out <= 256, W % 8 == 0 and
// W <= 64; everything else uses the two-kernel path.
#include "common.hpp"
#include "kernels.hpp"

namespace isam {
namespace {

constexpr int kWaves32 = 8;
constexpr int kR32 = 2;          // output rows per tile
constexpr int kKC = 32;          // channels per chunk
constexpr int kMaxW = 64;
constexpr int kMaxC = 128;
constexpr int kNT = kR32 * kMaxW / 16;   // pixel tiles of 16 per workgroup tile (max)
constexpr int kKB = kMaxC / kKC;         // 32-deep K blocks = chunks (max)
constexpr int kYUnit = kR32 * kMaxW * 16 + 64;
constexpr int kYTerm = 4 * kYUnit;
constexpr int kYBytes = 3 * kYTerm;

__device__ __forceinline__ void f32_dma16(__amdgpu_buffer_rsrc_t rs, uint32_t lds_addr, uint32_t voff) {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %1, %2, 0 offen lds"
        :
        : "s"(lds_addr), "v"(voff), "s"(rs)
        : "memory", "m0");
}
__device__ __forceinline__ uint32_t f32_lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}
__device__ __forceinline__ void f32_barrier() {
    asm volatile("" : : : "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" : : : "memory");
}
__device__ __forceinline__ uint32_t y_off(int t, int u, int p) { return (uint32_t)(t * kYTerm + u * kYUnit + p * 16); }

__host__ __device__ __forceinline__ int xbuf_bytes(int W) { return ((kR32 + 2) * W * kKC * 4 + 1023) / 1024 * 1024; }
__host__ __device__ __forceinline__ size_t f32_fused_lds(int W, int C) {
    return 2 * (size_t)xbuf_bytes(W) + (size_t)kYBytes + (size_t)9 * C * 4;
}

template <int NT>
__global__ __launch_bounds__(64 * kWaves32) void dwsep_fused_f32_kernel(DwArgs d, const float* pw, float* out,
                                                                        int64_t C_out) {
    extern __shared__ __attribute__((aligned(1024))) char smem[];
    const int C = (int)d.C, W = (int)d.W, H = (int)d.H;
    const int NCH = C / kKC;
    const int xb = xbuf_bytes(W);
    char* sX = smem;                                   // 2 x [R+2][W][32] fp32
    char* sY = smem + 2 * xb;                          // 3 term planes of the Y chunk
    float* sT = reinterpret_cast<float*>(sY + kYBytes);  // taps [9][C]
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int tiles_per_img = (H + kR32 - 1) / kR32;
    const int n_tiles = (int)d.batch * tiles_per_img;
    const int npx = kR32 * W;                          // pixels per tile (NT * 16)

    const __amdgpu_buffer_rsrc_t rsX = make_rsrc(d.x, (uint32_t)(d.batch * (int64_t)H * W * C * 4));
    const __amdgpu_buffer_rsrc_t rsO = make_rsrc(out, (uint32_t)(d.batch * (int64_t)H * W * C_out * 4));

    // Taps into LDS.
    const float* taps = static_cast<const float*>(d.w);
    for (int i = tid; i < 9 * C; i += 64 * kWaves32) sT[i] = taps[i];

    // The three bf16 terms of this wave's P slice as MFMA A operands: output
    // channel o = co0 + mt*16 + lane%16 and, in 32-deep block kb, the K
    // indices kb*32 + 8*(lane/16) + 0..7 (the B operands use the same).
    const int co0 = wid * 32;
    const int g = lane >> 4, li = lane & 15;
    uint4 pt[2][kKB][3];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int kb = 0; kb < kKB; ++kb) {
            uint32_t w[3][4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int o = co0 + mt * 16 + li, k = kb * 32 + 8 * g + 2 * e;
                const float x0 = (o < C_out && k < C) ? pw[(int64_t)k * C_out + o] : 0.0f;
                const float x1 = (o < C_out && k + 1 < C) ? pw[(int64_t)(k + 1) * C_out + o] : 0.0f;
                uint32_t t[3];
                split3_pair(x0, x1, t);
                w[0][e] = t[0];
                w[1][e] = t[1];
                w[2][e] = t[2];
            }
#pragma unroll
            for (int t = 0; t < 3; ++t) pt[mt][kb][t] = make_uint4(w[t][0], w[t][1], w[t][2], w[t][3]);
        }
    const bool wave_active = co0 < C_out;

    // Copy chunk c (channels c*32 .. +32) of tile `tile`'s input rows into buffer `buf`.
    const int units = (kR32 + 2) * W * 8;             // 16-byte units per chunk
    const int n_instr = (units + 63) / 64;
    auto copy_chunk = [&](int tile, int c, int buf) {
        if (tile >= n_tiles) return;
        const int b = tile / tiles_per_img, i0 = (tile % tiles_per_img) * kR32;
        char* dst = sX + buf * xb;
        for (int q = wid; q < n_instr; q += kWaves32) {
            const int unit = q * 64 + lane;
            const int pix = unit >> 3, u = unit & 7;
            const int rr = pix / W, x = pix - rr * W;
            const int ir = i0 - 1 + rr;
            const bool ok = unit < units && ir >= 0 && ir < H;
            const uint32_t off = ok ? (uint32_t)(((((int64_t)b * H + ir) * W + x) * C + c * kKC + u * 4) * 4) : kOob;
            f32_dma16(rsX, __builtin_amdgcn_readfirstlane(f32_lds_addr(dst + q * 1024)), off);
        }
    };

    // Depthwise of chunk c from buffer `buf` into the Y chunk: thread tid < W*8
    // owns (column j, channel unit u of 4 channels) for all R output rows.
    const bool dw_item = tid < W * 8;
    const int dj = dw_item ? tid >> 3 : 0, du = tid & 7;
    auto depthwise = [&](int c, int buf) {
        if (!dw_item) return;
        const char* xs = sX + buf * xb;
        const int ch = c * kKC + du * 4;
        float4 t[9];
#pragma unroll
        for (int q = 0; q < 9; ++q) t[q] = *reinterpret_cast<const float4*>(sT + q * C + ch);
        float4 win[3][3];  // sliding window: [row slot][column offset]
        auto load_row = [&](int rr, int slot) {
#pragma unroll
            for (int dx = 0; dx < 3; ++dx) {
                const int x = dj + dx - 1;
                win[slot][dx] = (x >= 0 && x < W) ? *reinterpret_cast<const float4*>(xs + ((rr * W + x) * 8 + du) * 16)
                                                  : make_float4(0.f, 0.f, 0.f, 0.f);
            }
        };
        load_row(0, 0);
        load_row(1, 1);
#pragma unroll
        for (int rl = 0; rl < kR32; ++rl) {
            load_row(rl + 2, (rl + 2) % 3);
            float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int di = 0; di < 3; ++di) {
                const int slot = (rl + di) % 3;
#pragma unroll
                for (int dx = 0; dx < 3; ++dx) {
                    const float4 v = win[slot][dx], w = t[di * 3 + dx];
                    a.x = fmaf(v.x, w.x, a.x);
                    a.y = fmaf(v.y, w.y, a.y);
                    a.z = fmaf(v.z, w.z, a.z);
                    a.w = fmaf(v.w, w.w, a.w);
                }
            }
            // channels du*4 .. +3 = half (du & 1) of unit du / 2
            uint32_t t01[3], t23[3];
            split3_pair(a.x, a.y, t01);
            split3_pair(a.z, a.w, t23);
#pragma unroll
            for (int t = 0; t < 3; ++t)
                *reinterpret_cast<uint2*>(sY + y_off(t, du >> 1, rl * W + dj) + (du & 1) * 8) = make_uint2(t01[t], t23[t]);
        }
    };

    int tile = blockIdx.x;
    copy_chunk(tile, 0, 0);
    int buf = 0;
    for (; tile < n_tiles; tile += gridDim.x) {
        f32x4_t acc[2][NT];
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        for (int c = 0; c < NCH; ++c) {
            // This wave's copies of chunk c (and the previous tile's stores)
            // are complete; after the barrier everyone's are, every wave is
            // done reading the Y chunk of c-1, and the other buffer is free.
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            f32_barrier();
            if (c + 1 < NCH) copy_chunk(tile, c + 1, buf ^ 1);
            else copy_chunk(tile + (int)gridDim.x, 0, buf ^ 1);
            depthwise(c, buf);
            f32_barrier();
            buf ^= 1;
            if (wave_active) {
                // pt's K block index must be a compile-time constant.
#pragma unroll
                for (int kk = 0; kk < kKB; ++kk) {
                    if (kk != c) continue;
                    // Pixel tiles in pairs; term products outermost, so
                    // consecutive MFMAs go to 4 different accumulators and
                    // none waits for the previous result.  Smallest terms
                    // first: (P term, Y term) = (m,m) (l,h) (h,l) (m,h) (h,m) (h,h).
                    constexpr int TA[6] = {1, 2, 0, 1, 0, 0}, TB[6] = {1, 0, 2, 0, 1, 0};
#pragma unroll
                    for (int n0 = 0; n0 < NT; n0 += 2) {
                        uint4 yb[2][3];
#pragma unroll
                        for (int j = 0; j < 2; ++j)
#pragma unroll
                            for (int t = 0; t < 3; ++t)
                                if (n0 + j < NT) yb[j][t] = *reinterpret_cast<const uint4*>(sY + y_off(t, g, (n0 + j) * 16 + li));
#pragma unroll
                        for (int e = 0; e < 6; ++e)
#pragma unroll
                            for (int j = 0; j < 2; ++j)
#pragma unroll
                                for (int mt = 0; mt < 2; ++mt)
                                    if (n0 + j < NT) mfma16_bf16(acc[mt][n0 + j], pt[mt][kk][TA[e]], yb[j][TB[e]]);
                    }
                }
            }
        }
        // Store: lane holds output channels co0 + mt*16 + 4*(lane/16) + 0..3 of
        // pixel nt*16 + lane%16; pixels past the image and channels past
        // C_out go to an offset beyond the buffer and are dropped.
        if (wave_active) {
            const int b = tile / tiles_per_img, i0 = (tile % tiles_per_img) * kR32;
            const int valid = min(kR32, H - i0) * W;
            const int64_t pix0 = ((int64_t)b * H + i0) * W;
#pragma unroll
            for (int mt = 0; mt < 2; ++mt)
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) {
                    const int p = nt * 16 + li;
                    const int o = co0 + mt * 16 + 4 * g;
                    const bool ok = p < valid && p < npx && o < C_out;
                    const int64_t idx = (pix0 + p) * C_out + o;
                    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4_t, acc[mt][nt]), rsO,
                                                           ok ? (int)(idx * 4) : (int)kOob, 0, 0);
                }
        }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

}  // namespace

// Whether the fp32 fused kernel applies to this shape.
bool dwsep_fused_f32_ok(const DwArgs& d, int64_t C_out, int lds_max) {
    if (d.in_type != kF32 || d.kh != 3 || d.kw != 3 || d.stride != 1 || d.pad != 1 || d.cm != 1) return false;
    if (d.C % kKC || d.C > kMaxC || C_out % 16 || C_out > 256) return false;
    if (d.W % 8 || d.W > kMaxW) return false;
    if (d.batch * d.H * d.W * d.C * 4 > (int64_t(1) << 31) - 1) return false;
    if (d.batch * d.H * d.W * C_out * 4 > (int64_t(1) << 31) - 1) return false;
    if (reinterpret_cast<uintptr_t>(d.x) & 15) return false;
    return f32_fused_lds((int)d.W, (int)d.C) <= (size_t)lds_max;
}

hipError_t launch_dwsep_fused_f32(const DwArgs& d, const void* pw, void* out, int64_t C_out, int cus,
                                  hipStream_t s) {
    const size_t lds = f32_fused_lds((int)d.W, (int)d.C);
    const int tiles = (int)(d.batch * ((d.H + kR32 - 1) / kR32));
    const int grid = tiles < cus ? tiles : cus;
    const int nt = kR32 * (int)d.W / 16;
    void* fn = nullptr;
    switch (nt) {  // pixel tiles per workgroup tile: R*W/16 with W % 8 == 0
        case 1: fn = reinterpret_cast<void*>(dwsep_fused_f32_kernel<1>); break;
        case 2: fn = reinterpret_cast<void*>(dwsep_fused_f32_kernel<2>); break;
        case 3: fn = reinterpret_cast<void*>(dwsep_fused_f32_kernel<3>); break;
        case 4: fn = reinterpret_cast<void*>(dwsep_fused_f32_kernel<4>); break;
        case 5: fn = reinterpret_cast<void*>(dwsep_fused_f32_kernel<5>); break;
        case 6: fn = reinterpret_cast<void*>(dwsep_fused_f32_kernel<6>); break;
        case 7: fn = reinterpret_cast<void*>(dwsep_fused_f32_kernel<7>); break;
        case 8: fn = reinterpret_cast<void*>(dwsep_fused_f32_kernel<8>); break;
        default: return hipErrorInvalidValue;
    }
    hipError_t e = ensure_dynamic_lds(fn, lds);
    if (e != hipSuccess) return e;
    DwArgs dd = d;
    const float* p = static_cast<const float*>(pw);
    float* o = static_cast<float*>(out);
    void* args[] = {&dd, &p, &o, &C_out};
    return hipLaunchKernel(fn, dim3(grid), dim3(64 * kWaves32), args, lds, s);
}

}  // namespace isam
