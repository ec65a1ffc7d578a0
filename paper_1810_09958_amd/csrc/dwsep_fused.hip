// Fused separable depthwise convolution (bf16 inputs): the third listing of
// the paper, factored as in Section 2.3 into a 3x3 depthwise stencil followed
// by the pointwise matrix product, with the intermediate kept on chip -- the
// inter-operation fusion the paper credits for its GRU results
// (Section 6.2.2) applied to this layer.
//
// A tile is R output rows of one image (R*W <= 64 pixels); each workgroup
// (one per CU) takes a contiguous range of tiles, so consecutive tiles share
// all but R of their R+2 input rows.  The 8 waves are specialised:
//   * producer waves 0-3 each own a quarter of the channels.  A wave streams
//     its channel slice of every input row it needs into a private LDS ring
//     (buffer_load ... lds; each row with a zero column on either side, rows
//     outside the image arrive as zeros), up to the ring's depth ahead,
//     computes the depthwise result of its channels for the tile in fp32
//     (taps in registers, the two left taps of a row paired for
//     v_dot2_f32_bf16), rounds it to bf16 and writes it into one of two A
//     tiles [64 px][C].  Depthwise is per channel, so a producer reads only
//     what it copied itself and waits only on its own copies.
//   * consumer waves 4-7 each own 64 output channels, keep that slice of P
//     in registers for the whole launch, form out^T = P^T . A^T on MFMA
//     (P fragments as the A operand, pixel fragments of the A tile read with
//     ds_read_b128 as the B operand) and store 4 consecutive output channels
//     of a pixel per lane straight from the accumulators.  They issue no
//     loads, so their stores are never waited on.
// One workgroup barrier per tile hands A tile t from the producers to the
// consumers while the producers fill the other A tile with tile t+1.
// Supported: bf16 input, 3x3, stride 1, pad 1, depth multiplier 1,
// C in {64, 128}, C_out % 8 == 0, C_out <= 256, W <= 64; everything else
// uses the two-kernel path.
#include "common.hpp"
#include "gemm_impl.hpp"
#include "kernels.hpp"

namespace isam {
namespace {

typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16_t lds_v4i16_t;
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef unsigned u32x2_t __attribute__((vector_size(2 * sizeof(unsigned))));

constexpr int kProducers = 4;    // depthwise waves, a quarter of the channels each
constexpr int kConsumers = 4;    // MFMA + store waves, 64 output channels each
constexpr int kFWaves = kProducers + kConsumers;
constexpr int kFPix = 64;        // MFMA pixel columns per tile
constexpr int kFBN = 256;        // output channels (4 consumer waves x 64)
constexpr int kMaxSlots = 16;    // input rows per producer ring

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
// A tile [64 px][C] bf16, 16-byte chunk c of pixel row px.  C = 128: chunk
// c ^ (px & 15); C = 64: chunk c ^ ((px >> 1) & 7).  Both make the consumer
// reads (16 pixel rows, one logical chunk per 16-lane phase) conflict-free.
template <int C>
__device__ __forceinline__ uint32_t f_a_off(int px, int c) {
    if constexpr (C == 128) return (uint32_t)(px * 256 + ((c ^ (px & 15)) << 4));
    else return (uint32_t)(px * 128 + ((c ^ ((px >> 1) & 7)) << 4));
}
// A consumer's staged P slice [k][64] bf16 (128-byte rows): 32-byte block b
// of row k at block b ^ (k & 3) -- conflict-free for ds_read_b64_tr_b16.
__device__ __forceinline__ uint32_t f_p_off(int k, int n) {
    return (uint32_t)(k * 128 + ((((n >> 4) ^ (k & 3))) << 5) + (n & 15) * 2);
}

typedef float f32x2_v __attribute__((ext_vector_type(2)));
// Two fp32 values to a bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t f_pack_bf16(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_v){lo, hi}, bf16x2_t));
}

template <int N>
__device__ __forceinline__ void f_vm_wait() {
    asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}
// Wait until at most n vector-memory operations are outstanding; counts past
// the largest case wait for that case (stricter, never looser).
__device__ __forceinline__ void f_vm_wait_rt(int n) {
#define ISAM_VMW(k) \
    case k: f_vm_wait<k>(); break;
    switch (n) {
        ISAM_VMW(0) ISAM_VMW(1) ISAM_VMW(2) ISAM_VMW(3) ISAM_VMW(4) ISAM_VMW(5) ISAM_VMW(6) ISAM_VMW(7)
        ISAM_VMW(8) ISAM_VMW(9) ISAM_VMW(10) ISAM_VMW(11) ISAM_VMW(12) ISAM_VMW(13) ISAM_VMW(14)
        ISAM_VMW(15) ISAM_VMW(16) ISAM_VMW(17) ISAM_VMW(18) ISAM_VMW(19) ISAM_VMW(20) ISAM_VMW(21)
        ISAM_VMW(22) ISAM_VMW(23) ISAM_VMW(24) ISAM_VMW(25) ISAM_VMW(26) ISAM_VMW(27) ISAM_VMW(28)
        ISAM_VMW(29) ISAM_VMW(30)
        default: f_vm_wait<31>(); break;
    }
#undef ISAM_VMW
}
__device__ __forceinline__ void f_lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
__device__ __forceinline__ void f_barrier() {
    asm volatile("" : : : "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" : : : "memory");
}

template <int C>
constexpr int a_tile_bytes() { return kFPix * C * 2; }

// Producer ring rows: logical 16-byte unit (unit column x, channel unit u) of
// a row, at a physical unit rotated within blocks of 16 units (256 bytes):
//   4 channel units per column (C = 128): unit (x, u) at
//     16 (x/4) + (4 (x%4) + u + 4 ((x/4)%4)) % 16;
//   2 channel units per column (C = 64): unit (x, u) at
//     16 (x/8) + (2 (x%8) + u + 2 ((x/8)%2)) % 16.
// A stencil read has lane (jl, ul) = (lane / UPW, lane % UPW) at column
// CPL jl + dj.  The jl of every 16-lane ds_read_b128 phase ({0-3, 12-15,
// 20-27}, {4-11, 16-19, 28-31}, and + 32) differ mod 4 (C = 128) or mod 8
// (C = 64), so the 16 lanes of a phase hit 16 different groups of 4 banks;
// unrotated, 4 (C = 128) or 2 (C = 64) lanes shared each group.
template <int UPW>
__device__ __forceinline__ int ring_pos(int x, int u) {
    static_assert(UPW == 4 || UPW == 2, "ring layout defined for 2 or 4 channel units per column");
    if constexpr (UPW == 4) return 16 * (x >> 2) + ((4 * (x & 3) + u + 4 * ((x >> 2) & 3)) & 15);
    else return 16 * (x >> 3) + ((2 * (x & 7) + u + 2 * ((x >> 3) & 1)) & 15);
}
// Inverse of ring_pos: the logical unit x * UPW + u held at physical unit p.
template <int UPW>
__device__ __forceinline__ int ring_unit(int p) {
    const int b = p >> 4;
    if constexpr (UPW == 4) return 16 * b + (((p & 15) - 4 * (b & 3)) & 15);
    else return 16 * b + (((p & 15) - 2 * (b & 1)) & 15);
}

template <int R, int C, typename TO, int NP = kProducers>
__global__ __launch_bounds__(64 * (NP + kConsumers)) void dwsep_fused_kernel(DwArgs d, const void* pw, void* out,
                                                                   int64_t C_out, int n_slots, int row_instr) {
    extern __shared__ __attribute__((aligned(1024))) char smem[];
    constexpr int UPW = C / (8 * NP);  // 16-byte channel units per producer wave
    constexpr int SLOTS = 64 / UPW;  // column runs per producer wave (lanes per channel unit)
    constexpr int CPL = kFPix / SLOTS;  // columns per run: SLOTS * CPL = 64 >= W, one pass
    constexpr int KS = C / 16;       // MFMA K steps
    constexpr int kA = a_tile_bytes<C>();
    const int W = (int)d.W, H = (int)d.H;
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int slot_bytes = row_instr * 1024;
    char* sA = smem;                 // two A tiles, C*256 bytes
    char* sT = smem + 2 * kA;        // C*256 more bytes: P staging of consumers 2, 3
    char* sX = sT + 2 * kA;          // producer rings
    const int tiles_per_img = (H + R - 1) / R;
    const int64_t n_tiles = d.batch * tiles_per_img;
    const int t_lo = (int)(n_tiles * blockIdx.x / gridDim.x);
    const int n_local = (int)(n_tiles * (blockIdx.x + 1) / gridDim.x) - t_lo;

    const __amdgpu_buffer_rsrc_t rsP = make_rsrc(pw, (uint32_t)(C * C_out * 2));
    const __amdgpu_buffer_rsrc_t rsX = make_rsrc(d.x, (uint32_t)(d.batch * (int64_t)H * W * C * 2));
    const __amdgpu_buffer_rsrc_t rsO =
        make_rsrc(out, (uint32_t)(d.batch * (int64_t)H * W * C_out * (int64_t)sizeof(TO)));
    const bool producer = wid < NP;
    const int pw4 = producer ? wid : wid - NP;  // producer index / consumer index

    // Producer lane: channel unit ug (8 channels) of the CPL adjacent columns
    // jl*CPL .. jl*CPL + CPL-1.  Its taps are fixed: (di, 0) and (di, 1)
    // paired as bf16x2, (di, 2) fp32.
    const int ul = lane % UPW, jl = lane / UPW, ug = pw4 * UPW + ul;
    uint32_t w01[3][8];
    float w2[3][8];
    // Consumer: P^T fragments of its 64 output channels (MFMA A operand,
    // lane l: channel l % 32 of the block, K values 8*(l/32) .. +7 of a step).
    const int g = lane >> 4, li = lane & 15;
    uint4 pf[2][KS];

    char* ring = sX + pw4 * n_slots * slot_bytes;
    // Input rows form one sequence: tile t reads the R+2 rows ending at
    // sequence number e_t; a tile continuing the previous one in the same
    // image adds R new rows, any other R+2.  Row s lives in slot s % n_slots.
    auto new_rows = [&](int t) {
        const int i0 = ((t_lo + t) % tiles_per_img) * R;
        return (t == 0 || i0 == 0) ? R + 2 : R;
    };
    int nx_tile = 0, nx_k = 0, issued = 0, nx_slot = 0;
    auto issue_row = [&]() {
        const int tg = t_lo + nx_tile;
        const int img = tg / tiles_per_img, i0 = (tg % tiles_per_img) * R;
        const int nr = new_rows(nx_tile);
        const int ir = i0 - 1 + (R + 2 - nr) + nx_k;
        char* dst = ring + nx_slot * slot_bytes;
        const bool row_ok = ir >= 0 && ir < H;
        for (int q = 0; q < row_instr; ++q) {
            // physical unit q * 64 + lane holds logical unit v: column v / UPW - 1 (zero halo at -1
            // and W), channel unit v % UPW
            const int v = ring_unit<UPW>(q * 64 + lane);
            const int x = v / UPW - 1, u = v % UPW;
            const bool ok = row_ok && x >= 0 && x < W;
            const uint32_t off =
                ok ? (uint32_t)(((((int64_t)img * H + ir) * W + x) * C + (pw4 * UPW + u) * 8) * 2) : kOob;
            f_dma16(rsX, __builtin_amdgcn_readfirstlane(f_lds_addr(dst + q * 1024)), off);
        }
        ++issued;
        nx_slot = nx_slot + 1 == n_slots ? 0 : nx_slot + 1;
        if (++nx_k == nr) {
            nx_k = 0;
            ++nx_tile;
        }
    };

    if (producer) {
        // The rings do not overlap the P staging: stream the first tile's
        // rows at once, then load the taps (the compiler's wait for them
        // also covers those rows, which the first tile needs anyway), then
        // fill the rest of the ring.
        while (nx_tile < n_local && issued < R + 2) issue_row();
        const uint16_t* wp = static_cast<const uint16_t*>(d.w);
#pragma unroll
        for (int di = 0; di < 3; ++di) {
            const uint4 t0 = *reinterpret_cast<const uint4*>(wp + (di * 3 + 0) * C + ug * 8);
            const uint4 t1 = *reinterpret_cast<const uint4*>(wp + (di * 3 + 1) * C + ug * 8);
            const uint4 t2 = *reinterpret_cast<const uint4*>(wp + (di * 3 + 2) * C + ug * 8);
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
        // Pin the taps here, before the next copies are issued.
#pragma unroll
        for (int di = 0; di < 3; ++di)
#pragma unroll
            for (int c = 0; c < 8; ++c) asm volatile("" : : "v"(w01[di][c]), "v"(w2[di][c]));
        // Only the next tile's rows now: every workgroup requests its first
        // rows at the same moment, and a shorter burst lands them sooner.
        while (nx_tile < n_local && issued < min(n_slots, 2 * R + 2)) issue_row();
    } else {
        // Stage this wave's P slice [C][64] (columns past C_out read as zero),
        // then read its fragments; no other wave touches this staging area.
        char* st = (pw4 < 2 ? sA : sT) + (pw4 & 1) * (C * 128);
        constexpr int p_instr = C * 128 / 1024;
#pragma unroll
        for (int q = 0; q < p_instr; ++q) {
            const int unit = q * 64 + lane;
            const int k = unit >> 3, pu = unit & 7;
            const int n = pw4 * 64 + (((pu >> 1) ^ (k & 3)) << 4) + (pu & 1) * 8;
            const uint32_t off = (n < C_out) ? (uint32_t)((k * C_out + n) * 2) : kOob;
            f_dma16(rsP, __builtin_amdgcn_readfirstlane(f_lds_addr(st + q * 1024)), off);
        }
        f_vm_wait<0>();
#pragma unroll
        for (int i = 0; i < 2; ++i) {
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                const int n = i * 32 + (g & 1) * 16 + 4 * (li & 3);
                uint32_t w[4];
#pragma unroll
                for (int rr = 0; rr < 2; ++rr) {
                    const int k = s * 16 + (g >> 1) * 8 + rr * 4 + (li >> 2);
                    v4i16_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(st + f_p_off(k, n)));
                    const uint2 uu = __builtin_bit_cast(uint2, v);
                    w[rr * 2] = uu.x;
                    w[rr * 2 + 1] = uu.y;
                }
                pf[i][s] = make_uint4(w[0], w[1], w[2], w[3]);
            }
        }
        f_lds_wait();
    }
    f_barrier();  // every P slice is in registers: the staging areas are free

    if (producer) {
        int e = 0;
        for (int t = 0; t < n_local; ++t) {
            e += new_rows(t);
            const int first = e - (R + 2);  // oldest row this tile reads
            while (nx_tile < n_local && issued < first + n_slots) issue_row();
            f_vm_wait_rt((issued - e) * row_instr);  // rows up to e - 1 have landed

            char* A = sA + (t & 1) * kA;
            const char* rowp[R + 2];  // this tile's input rows in the ring
#pragma unroll
            for (int k = 0; k < R + 2; ++k) {
                int sl = first % n_slots + k;
                if (sl >= n_slots) sl -= n_slots;
                rowp[k] = ring + sl * slot_bytes;
            }
            // One pass: the lane reads columns j0-1 .. j0+CPL of each of the
            // R+2 rows (the halo columns make every read unconditional; a run
            // past the image is not stored), all reads
            // in flight at once, then computes its CPL x R outputs: each
            // loaded column serves up to three outputs instead of being read
            // once per output.
            // Unit columns past W+1 feed only outputs past the image (not
            // stored); they are clamped to the row's last unit column, which
            // keeps every read inside the row and (unlike a clamp at W+1)
            // adds no bank conflicts.
            const int j0 = jl * CPL, xcap = row_instr * 64 / UPW - 1;
            uint4 v[R + 2][CPL + 2];
#pragma unroll
            for (int k = 0; k < R + 2; ++k)
#pragma unroll
                for (int dj = 0; dj < CPL + 2; ++dj) {
                    const int x = min(j0 + dj, xcap);  // unit column x holds image column x-1
                    v[k][dj] = *reinterpret_cast<const uint4*>(rowp[k] + ring_pos<UPW>(x, ul) * 16);
                }
#pragma unroll
            for (int cl = 0; cl < CPL; ++cl) {
                const int j = j0 + cl;
                if (j >= W) break;
                uint32_t pr[R + 2][8];  // per row: (x=j-1, x=j) pairs per channel
                float sg[R + 2][8];     // per row: x=j+1 per channel
#pragma unroll
                for (int k = 0; k < R + 2; ++k) {
                    const uint4 c0 = v[k][cl], c1 = v[k][cl + 1], c2 = v[k][cl + 2];
                    const uint32_t b0[4] = {c0.x, c0.y, c0.z, c0.w}, b1[4] = {c1.x, c1.y, c1.z, c1.w},
                                   b2[4] = {c2.x, c2.y, c2.z, c2.w};
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        pr[k][2 * q] = __builtin_amdgcn_perm(b1[q], b0[q], 0x05040100u);
                        pr[k][2 * q + 1] = __builtin_amdgcn_perm(b1[q], b0[q], 0x07060302u);
                        sg[k][2 * q] = bf16lo(b2[q]);
                        sg[k][2 * q + 1] = bf16hi(b2[q]);
                    }
                }
#pragma unroll
                for (int rl = 0; rl < R; ++rl) {
                    float acc[8];
#pragma unroll
                    for (int c = 0; c < 8; ++c) {
                        float a = 0.0f;
#pragma unroll
                        for (int di = 0; di < 3; ++di) {
                            a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pr[rl + di][c]),
                                                                __builtin_bit_cast(bf16x2_t, w01[di][c]), a, false);
                            a = fmaf(sg[rl + di][c], w2[di][c], a);
                        }
                        acc[c] = a;
                    }
                    *reinterpret_cast<uint4*>(A + f_a_off<C>(rl * W + j, ug)) =
                        make_uint4(f_pack_bf16(acc[0], acc[1]), f_pack_bf16(acc[2], acc[3]),
                                   f_pack_bf16(acc[4], acc[5]), f_pack_bf16(acc[6], acc[7]));
                }
            }
            f_lds_wait();
            f_barrier();  // A tile t complete
        }
    } else {
        const int cb = wid - NP;
        const bool active = cb * 64 < C_out;
        for (int t = 0; t < n_local; ++t) {
            f_barrier();  // A tile t complete; A tile t-1 may be overwritten after the next barrier
            if (!active) continue;
            const char* A = sA + (t & 1) * kA;
            f32x16_t acc[2][2];
            static_for<2>([&](auto i) {
                static_for<2>([&](auto jj) {
                    static_for<16>([&](auto v) { acc[i][jj][decltype(v)::value] = 0.0f; });
                });
            });
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                uint4 yf[2];
#pragma unroll
                for (int jj = 0; jj < 2; ++jj)
                    yf[jj] = *reinterpret_cast<const uint4*>(A + f_a_off<C>(jj * 32 + (lane & 31), 2 * s + (lane >> 5)));
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int jj = 0; jj < 2; ++jj) mfma32_bf16(acc[i][jj], pf[i][s], yf[jj]);
            }
            // Accumulator element v of lane l: output channel
            // cb*64 + i*32 + 8*(v/4) + 4*(l/32) + v%4 of pixel jj*32 + l%32.
            const int tg = t_lo + t;
            const int img = tg / tiles_per_img, i0 = (tg % tiles_per_img) * R;
            const int valid_px = min(R, H - i0) * W;
            const int64_t m0 = ((int64_t)img * H + i0) * W;
            // Output through the wave's part of the P staging area (free
            // after the prologue), 32 pixels at a time: a pixel's 64 channels
            // of this wave are one contiguous piece of the output row (128
            // bytes bf16, 256 fp32), so every store instruction writes whole
            // pieces instead of 32 scattered 8- or 16-byte ones.  16-byte chunk
            // c of staged pixel p sits at chunk c ^ (p & (CH-1)).
            constexpr int RB = 64 * (int)sizeof(TO), CH = RB / 16;
            constexpr bool kStaged = 32 * RB * kConsumers <= 2 * kA;
            if constexpr (kStaged) {
                char* stg = sT + cb * (32 * RB);
                static_for<2>([&](auto jjc) {
                    constexpr int jj = decltype(jjc)::value;
                    const int p = lane & 31;
                    static_for<2>([&](auto ic) {
                        constexpr int i = decltype(ic)::value;
                        static_for<4>([&](auto v4c) {
                            constexpr int v4 = decltype(v4c)::value;
                            const int byte = (i * 32 + 8 * v4 + 4 * (lane >> 5)) * (int)sizeof(TO);
                            char* dst = stg + p * RB + ((((byte >> 4) ^ (p & (CH - 1)))) << 4) + (byte & 15);
                            const float x0 = acc[i][jj][4 * v4], x1 = acc[i][jj][4 * v4 + 1];
                            const float x2 = acc[i][jj][4 * v4 + 2], x3 = acc[i][jj][4 * v4 + 3];
                            if constexpr (sizeof(TO) == 4)
                                *reinterpret_cast<float4*>(dst) = make_float4(x0, x1, x2, x3);
                            else
                                *reinterpret_cast<uint2*>(dst) = make_uint2(f_pack_bf16(x0, x1), f_pack_bf16(x2, x3));
                        });
                    });
                    f_lds_wait();  // this wave's staging writes before its reads (no other wave uses the area)
#pragma unroll
                    for (int r = 0; r < 32 * CH / 64; ++r) {
                        const int q = r * 64 + lane, pp = q / CH, c = q % CH;
                        const uint4 val = *reinterpret_cast<const uint4*>(stg + pp * RB + ((c ^ (pp & (CH - 1))) << 4));
                        const int px = jj * 32 + pp;
                        const int64_t co = cb * 64 + c * (16 / (int)sizeof(TO));
                        const bool ok = px < valid_px && co < C_out;
                        const int64_t idx = (m0 + px) * C_out + co;
                        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4_t, val), rsO,
                                                               ok ? (int)(idx * (int64_t)sizeof(TO)) : (int)kOob, 0, 0);
                    }
                });
            } else
            static_for<2>([&](auto i) {
                static_for<2>([&](auto jj) {
                    static_for<4>([&](auto v4c) {
                        constexpr int v4 = decltype(v4c)::value;
                        const int px = jj * 32 + (lane & 31);
                        const int64_t co = cb * 64 + i * 32 + 8 * v4 + 4 * (lane >> 5);
                        const bool ok = px < valid_px && co < C_out;
                        const int64_t idx = (m0 + px) * C_out + co;
                        const float x0 = acc[i][jj][4 * v4], x1 = acc[i][jj][4 * v4 + 1];
                        const float x2 = acc[i][jj][4 * v4 + 2], x3 = acc[i][jj][4 * v4 + 3];
                        if constexpr (sizeof(TO) == 4)
                            __builtin_amdgcn_raw_buffer_store_b128(
                                __builtin_bit_cast(i32x4_t, make_float4(x0, x1, x2, x3)), rsO,
                                ok ? (int)(idx * 4) : (int)kOob, 0, 0);
                        else
                            __builtin_amdgcn_raw_buffer_store_b64(
                                __builtin_bit_cast(u32x2_t, make_uint2(f_pack_bf16(x0, x1), f_pack_bf16(x2, x3))), rsO,
                                ok ? (int)(idx * 2) : (int)kOob, 0, 0);
                    });
                });
            });
        }
    }
}

struct FusedPlan {
    int R = 0, n_slots = 0, row_instr = 0;
    size_t lds = 0;
};

FusedPlan fused_plan(const DwArgs& d, int64_t C_out, int lds_max) {
    FusedPlan p;
    if (d.in_type != kBF16 || d.kh != 3 || d.kw != 3 || d.stride != 1 || d.pad != 1 || d.cm != 1) return p;
    if ((d.C != 64 && d.C != 128) || C_out % 8 || C_out > kFBN || C_out <= 0) return p;
    // buffer offsets are 32-bit: input and (fp32) output extents below 2^31
    if (d.batch * d.H * d.W * d.C * 2 > (int64_t(1) << 31) - 1) return p;
    if (d.batch * d.H * d.W * C_out * 4 > (int64_t(1) << 31) - 1) return p;
    if ((reinterpret_cast<uintptr_t>(d.x) & 15) || (reinterpret_cast<uintptr_t>(d.w) & 15)) return p;
    if (d.W <= 0 || d.W > kFPix || d.H <= 0) return p;
    const int R = d.W <= kFPix / 2 ? 2 : 1;
    const int upw = (int)d.C / (8 * kProducers);
    const int row_instr = (int)(((d.W + 2) * upw + 63) / 64);  // a row with its zero halo
    // two A tiles (C*256 bytes) and as much again for the P staging of the
    // other two consumers, then the four producer rings
    const size_t fixed = 2 * (size_t)kFPix * d.C * 2 * 2;
    const size_t set_bytes = kProducers * (size_t)row_instr * 1024;  // one slot of each producer ring
    if ((size_t)lds_max <= fixed) return p;
    const int n_slots = (int)std::min<size_t>(kMaxSlots, ((size_t)lds_max - fixed) / set_bytes);
    if (n_slots < R + 2) return p;
    p.R = R;
    p.n_slots = n_slots;
    p.row_instr = row_instr;
    p.lds = fixed + (size_t)n_slots * set_bytes;
    return p;
}

template <int R, int C>
void* fused_fn(int out_type) {
    return out_type == kF32 ? reinterpret_cast<void*>(dwsep_fused_kernel<R, C, float>)
                            : reinterpret_cast<void*>(dwsep_fused_kernel<R, C, uint16_t>);
}

}  // namespace

// Rows per tile for this shape, or 0 when the fused kernel does not apply.
int dwsep_fused_rows(const DwArgs& d, int64_t C_out, int lds_max) { return fused_plan(d, C_out, lds_max).R; }

hipError_t launch_dwsep_fused(const DwArgs& d, const void* pw, void* out, int64_t C_out, int out_type, int lds_max,
                              int cus, hipStream_t s) {
    const FusedPlan p = fused_plan(d, C_out, lds_max);
    if (!p.R) return hipErrorInvalidValue;
    const int64_t tiles = d.batch * ((d.H + p.R - 1) / p.R);
    const int grid = (int)std::min<int64_t>(tiles, cus);
    void* fn = p.R == 2 ? (d.C == 128 ? fused_fn<2, 128>(out_type) : fused_fn<2, 64>(out_type))
                        : (d.C == 128 ? fused_fn<1, 128>(out_type) : fused_fn<1, 64>(out_type));
    hipError_t e = ensure_dynamic_lds(fn, p.lds);
    if (e != hipSuccess) return e;
    DwArgs dd = d;
    int n_slots = p.n_slots, row_instr = p.row_instr;
    void* args[] = {&dd, const_cast<void**>(&pw), &out, &C_out, &n_slots, &row_instr};
    return hipLaunchKernel(fn, dim3(grid), dim3(64 * kFWaves), args, p.lds, s);
}

}  // namespace isam
