// bf16 MFMA GEMM fed by direct global->LDS loads (gfx950).
//
// Same contraction as the register-staged tile kernel (the paper's first
// listing), with the HBM -> LDS -> VGPR path of Section 3.5 rebuilt around
// the CDNA4 data movers:
//   * buffer_load ... lds (16 bytes per lane) copies A and B tiles straight
//     into LDS: no staging registers and no ds_write instructions;
//   * the K depth of a stage is 64, so every copied row segment is a whole
//     128-byte cache line (row segments of 64 bytes leave half of each line
//     fetched into the vector L1 unused and cap the L1 -> LDS stream at about
//     two thirds of its full-line rate); two stages, and the copies of tile
//     t+2 are issued during the last K step of tile t, a whole tile of MFMAs
//     ahead of their use;
//   * a copy instruction writes 64 consecutive 16-byte LDS units, so the
//     bank swizzle is applied by choosing which global chunk each lane
//     fetches; out-of-range chunks are fetched at an offset past the buffer
//     end and arrive as zeros;
//   * A (K-contiguous) is read with ds_read_b128.  B is read with
//     ds_read_b128 when K-contiguous, and with ds_read_b64_tr_b16 when
//     N-contiguous: within each 16-lane group that instruction hands lane j
//     element j%4 of the 8-byte pieces addressed by lanes j/4 + 4e
//     (e = 0..3), so pieces taken from four consecutive K rows arrive as
//     four consecutive K values of one column -- the MFMA B operand -- with
//     no transpose pass.
// LDS layouts (one stage, bf16), chosen for the gfx950 LDS as measured: 64
// banks of 4 bytes; a ds_read_b128 is served in four 16-lane phases, lanes
// {0-3, 12-15, 20-27}, {4-11, 16-19, 28-31} and the same sets + 32; a
// ds_read_b64_tr_b16 in two 32-lane phases.  A phase with two different
// addresses on one bank takes an extra pass.
//   A / K-contiguous B: row r (128 bytes = 64 K values), logical 16-byte
//     chunk c at physical chunk c ^ ((r ^ (r >> 3)) & 7): the 16 rows of a
//     b128 phase then cover all 16 bank groups of 16 bytes;
//   N-contiguous B: K row k (BN*2 bytes), logical 32-byte block b at physical
//     block b ^ (2 * (k & 3)): the 4 K rows x 2 column blocks of a 32-lane
//     transpose-read phase land in 8 different 32-byte bank groups.
#pragma once

#include "common.hpp"
#include "gemm_impl.hpp"

namespace isam {

typedef __attribute__((address_space(3))) void lds_void_t;
typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16_t lds_v4i16_t;

__device__ __forceinline__ int dma_a_swz(int r) { return (r ^ (r >> 3)) & 7; }
__device__ __forceinline__ int dma_b_swz(int k) { return 2 * (k & 3); }

__device__ __forceinline__ uint32_t dma_a_off(int r, int c) {
    return (uint32_t)(r * 128 + ((c ^ dma_a_swz(r)) << 4));
}

// The copies are issued with inline assembly so that the compiler, which
// cannot tell which LDS bytes an in-flight copy will write, does not drain
// every outstanding copy before each LDS read and barrier.  Completion is
// tracked explicitly: vm_wait<N>() returns once at most N of this wave's
// copies are still in flight (they complete in issue order), and
// block_sync() is a plain workgroup barrier without a memory fence.
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t rs, uint32_t lds_addr, uint32_t voff) {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %1, %2, 0 offen lds"
        :
        : "s"(lds_addr), "v"(voff), "s"(rs)
        : "memory", "m0");
}

template <int N>
__device__ __forceinline__ void vm_wait() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

__device__ __forceinline__ void block_sync() {
    asm volatile("" : : : "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" : : : "memory");
}

__device__ __forceinline__ uint32_t lds_addr_of(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}

// Per-lane copy plan for one workgroup's A and B tiles (K depth 64 per
// tile): byte offsets relative to the tile origin, with -1 for chunks outside
// the M / N range.  Copy instruction Q of an operand fills the 1 KB LDS
// block Q of this wave inside the operand's region: 8 rows x 128 bytes for a
// K-contiguous operand, 1024 / (BN*2) K rows for N-contiguous B.
template <int BM, int BN, bool TB, int NW>
struct DmaCopier {
    static constexpr int A_INSTR = BM * 128 / 1024 / NW, B_INSTR = BN * 128 / 1024 / NW;
    static_assert(A_INSTR >= 1 && B_INSTR >= 1, "tile too small for one copy per wave");
    static_assert(TB || BN >= 128, "N-contiguous B swizzle needs 8 column blocks per K row");
    __amdgpu_buffer_rsrc_t rsA, rsB;
    int64_t a_row_off[A_INSTR], b_off[B_INSTR];
    int a_k[A_INSTR], b_k[B_INSTR];
    // Byte offsets of each copy for the K tile at k = 0 (kOob outside M / N):
    // for a K tile wholly inside K the offset is base + a wave-uniform delta.
    uint32_t a_base[A_INSTR], b_base[B_INSTR];
    int64_t ldb, kend;
    int wid;

    __device__ __forceinline__ DmaCopier(const GemmArgs& a, int64_t m0, int64_t n0, int64_t kend_, int wid_, int lane)
        : ldb(a.ldb), kend(kend_), wid(wid_) {
        const int64_t a_ext = (a.M - 1) * a.lda + a.K;
        const int64_t b_ext = TB ? ((a.N - 1) * a.ldb + a.K) : ((a.K - 1) * a.ldb + a.N);
        rsA = make_rsrc(a.A, (uint32_t)(a_ext * 2));
        rsB = make_rsrc(a.B, (uint32_t)(b_ext * 2));
#pragma unroll
        for (int q = 0; q < A_INSTR; ++q) {
            const int unit = (wid * A_INSTR + q) * 64 + lane;  // 16-byte LDS unit within the A region
            const int r = unit >> 3, pc = unit & 7;
            a_k[q] = (pc ^ dma_a_swz(r)) * 8;
            a_row_off[q] = (m0 + r < a.M) ? (m0 + r) * a.lda : -1;
            a_base[q] = a_row_off[q] >= 0 ? (uint32_t)((a_row_off[q] + a_k[q]) * 2) : kOob;
        }
#pragma unroll
        for (int q = 0; q < B_INSTR; ++q) {
            const int unit = (wid * B_INSTR + q) * 64 + lane;
            if constexpr (TB) {
                const int r = unit >> 3, pc = unit & 7;
                b_k[q] = (pc ^ dma_a_swz(r)) * 8;
                b_off[q] = (n0 + r < a.N) ? (n0 + r) * a.ldb : -1;
            } else {
                constexpr int UPR = BN / 8;  // 16-byte units per K row
                const int k = unit / UPR, u = unit % UPR;
                const int b = (u >> 1) ^ dma_b_swz(k);
                const int64_t n = n0 + b * 16 + (u & 1) * 8;
                b_k[q] = k;
                b_off[q] = (n < a.N) ? n : -1;
            }
            if constexpr (TB) b_base[q] = b_off[q] >= 0 ? (uint32_t)((b_off[q] + b_k[q]) * 2) : kOob;
            else b_base[q] = b_off[q] >= 0 ? (uint32_t)((b_k[q] * ldb + b_off[q]) * 2) : kOob;
        }
    }
    // Copies of a K tile wholly inside K: offset = base + the tile's delta
    // (k0 * 2 bytes for A and K-contiguous B, k0 * ldb * 2 for N-contiguous B).
    // live == false (a K tile past the last one): every lane reads past the
    // buffer end, so the copy moves zeros and touches no memory.
    template <int Q>
    __device__ __forceinline__ void a_part_full(uint32_t delta, uint32_t dst, bool live = true) const {
        dma16(rsA, __builtin_amdgcn_readfirstlane(dst + (uint32_t)((wid * A_INSTR + Q) * 1024)), live ? a_base[Q] + delta : kOob);
    }
    template <int Q>
    __device__ __forceinline__ void b_part_full(uint32_t delta, uint32_t dst, bool live = true) const {
        dma16(rsB, __builtin_amdgcn_readfirstlane(dst + (uint32_t)((wid * B_INSTR + Q) * 1024)), live ? b_base[Q] + delta : kOob);
    }
    // A copy instruction Q of the K tile starting at k0 into the A region at
    // LDS address `dst` (a wave-uniform 32-bit LDS address, so no generic-
    // pointer conversion is redone per copy).
    template <int Q>
    __device__ __forceinline__ void a_part(int64_t k0, uint32_t dst) const {
        const int64_t k = k0 + a_k[Q];
        const uint32_t off = (a_row_off[Q] >= 0 && k < kend) ? (uint32_t)((a_row_off[Q] + k) * 2) : kOob;
        dma16(rsA, __builtin_amdgcn_readfirstlane(dst + (uint32_t)((wid * A_INSTR + Q) * 1024)), off);
    }
    template <int Q>
    __device__ __forceinline__ void b_part(int64_t k0, uint32_t dst) const {
        const int64_t k = k0 + b_k[Q];
        uint32_t off;
        if constexpr (TB) off = (b_off[Q] >= 0 && k < kend) ? (uint32_t)((b_off[Q] + k) * 2) : kOob;
        else off = (b_off[Q] >= 0 && k < kend) ? (uint32_t)((k * ldb + b_off[Q]) * 2) : kOob;
        dma16(rsB, __builtin_amdgcn_readfirstlane(dst + (uint32_t)((wid * B_INSTR + Q) * 1024)), off);
    }
};

// MFMA operands of one 16-deep K step: MI A blocks and NI B blocks (32x32 each).
template <int MI, int NI>
struct Frag {
    uint4 a[MI], b[NI];
};

// LDS read number IDX of a fragment set (K step ks of the tile whose A / B
// regions are sa / sb): A blocks first (one ds_read_b128 each), then B
// blocks (one ds_read_b128, or two ds_read_b64_tr_b16 when N-contiguous).
// arow / bcol: the wave's first A row / B column inside the tile.
template <int IDX, int MI, int NI, bool TB, int BN>
__device__ __forceinline__ void read_frag_part(Frag<MI, NI>& f, const char* sa, const char* sb, int ks, int arow,
                                               int bcol, int lane) {
    const int ch = ks * 2 + (lane >> 5);
    if constexpr (IDX < MI) {
        const int r = arow + IDX * 32 + (lane & 31);
        f.a[IDX] = *reinterpret_cast<const uint4*>(sa + dma_a_off(r, ch));
    } else if constexpr (TB) {
        constexpr int j = IDX - MI;
        const int r = bcol + j * 32 + (lane & 31);
        f.b[j] = *reinterpret_cast<const uint4*>(sb + dma_a_off(r, ch));
    } else {
        constexpr int j = (IDX - MI) / 2, rr = (IDX - MI) % 2;
        const int g = lane >> 4, li = lane & 15;
        const int n = bcol + j * 32 + (g & 1) * 16 + 4 * (li & 3);
        const int k = ks * 16 + (g >> 1) * 8 + rr * 4 + (li >> 2);
        const int b = (n >> 4) ^ dma_b_swz(k);
        const char* p = sb + k * (BN * 2) + b * 32 + (n & 15) * 2;
        v4i16_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)p);
        const uint2 u = __builtin_bit_cast(uint2, v);
        if constexpr (rr == 0) {
            f.b[j].x = u.x;
            f.b[j].y = u.y;
        } else {
            f.b[j].z = u.x;
            f.b[j].w = u.y;
        }
    }
}

// Main loop of the three-stage ring (see the kernel's comment).  One operand
// (B, or A when A3) has three stages, the other two: layout A stages then B
// stages, each A_BYTES / B_BYTES.
template <int BM, int BN, bool TB, int WM, int WN, bool KFULL, bool A3, int MI, int NI, typename Copier>
__device__ __forceinline__ void ring3_main_loop(f32x16_t (&acc)[MI][NI], char* smem, uint32_t smem_base, const Copier& cp,
                                                const GemmArgs& a, int64_t kbeg, int nk, int wm, int wn, int lane) {
    constexpr int BK = 64, A_BYTES = BM * 128, B_BYTES = BN * 128;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int A_ST = A3 ? 3 : 2;
    const uint32_t bbase = smem_base + (uint32_t)(A_ST * A_BYTES);
    // KFULL: offsets as base + per-tile delta; otherwise range-checked (a K
    // tile past the end is wholly out of range and reads nothing either way)
    auto copy_a = [&](int tt, int ast, auto q_c) {
        const int64_t k0 = kbeg + (int64_t)tt * BK;
        const uint32_t dst = smem_base + (uint32_t)(ast * A_BYTES);
        if constexpr (KFULL) cp.template a_part_full<decltype(q_c)::value>((uint32_t)(k0 * 2), dst, tt < nk);
        else cp.template a_part<decltype(q_c)::value>(k0, dst);
    };
    auto copy_b = [&](int tt, int bst, auto q_c) {
        const int64_t k0 = kbeg + (int64_t)tt * BK;
        const uint32_t dst = bbase + (uint32_t)(bst * B_BYTES);
        if constexpr (KFULL) cp.template b_part_full<decltype(q_c)::value>((uint32_t)(TB ? k0 * 2 : k0 * a.ldb * 2), dst, tt < nk);
        else cp.template b_part<decltype(q_c)::value>(k0, dst);
    };
    // the three-stage operand (stage s3) and the two-stage one (stage tt & 1)
    constexpr int Q3 = A3 ? Copier::A_INSTR : Copier::B_INSTR, Q2 = A3 ? Copier::B_INSTR : Copier::A_INSTR;
    auto copy3 = [&](int tt, int s3, auto q_c) {
        if constexpr (A3) copy_a(tt, s3, q_c);
        else copy_b(tt, s3, q_c);
    };
    auto copy2 = [&](int tt, auto q_c) {
        if constexpr (A3) copy_b(tt, tt & 1, q_c);
        else copy_a(tt, tt & 1, q_c);
    };
    using F = Frag<MI, NI>;
    constexpr int N_READS = MI + NI * (TB ? 1 : 2);
    // s2: stage of the two-stage operand, s3: of the three-stage one
    auto read_part = [&](F& f, int s2, int s3, int ks, auto idx_c) {
        const int ast = A3 ? s3 : s2, bst = A3 ? s2 : s3;
        read_frag_part<decltype(idx_c)::value, MI, NI, TB, BN>(f, smem + ast * A_BYTES, smem + A_ST * A_BYTES + bst * B_BYTES,
                                                               ks, wm * WTM, wn * WTN, lane);
    };
    // MFMAs of f, with the reads of step ks (stages s2 / s3) into g and then
    // the copies CK spread over the MFMA slots (0: none; 1, 2, 3: the first
    // half, third quarter and last quarter of the three-stage operand's
    // copies of tile t+2, into its stage r2; 4: every copy of the two-stage
    // operand for tile t+2).
    auto step = [&](const F& f, F& g, int s2, int s3, int ks, auto ck_c, int t, int r2) {
        constexpr int CK = decltype(ck_c)::value;
        // copies of this step: [0, Q3/2), [Q3/2, 3Q3/4), [3Q3/4, Q3) of the three-stage operand, [0, Q2) of the other
        constexpr int QLO = CK == 1 ? 0 : CK == 2 ? Q3 / 2 : CK == 3 ? 3 * Q3 / 4 : 0;
        constexpr int NC = CK == 0 ? 0 : CK == 1 ? Q3 / 2 : CK == 2 ? 3 * Q3 / 4 - Q3 / 2 : CK == 3 ? Q3 - 3 * Q3 / 4 : Q2;
        static_for<MI * NI>([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            mfma32_bf16(acc[k / NI][k % NI], f.a[k / NI], f.b[k % NI]);
            constexpr int SL = MI * NI, NOPS = N_READS + NC;
            constexpr int lo = (k * NOPS + SL - 1) / SL, hi = ((k + 1) * NOPS + SL - 1) / SL;
            static_for<hi - lo>([&](auto d) {
                constexpr int o = lo + decltype(d)::value;
                if constexpr (o < N_READS) {
                    read_part(g, s2, s3, ks, std::integral_constant<int, o>{});
                } else {
                    constexpr int c = o - N_READS;
                    if constexpr (CK >= 1 && CK <= 3) copy3(t + 2, r2, std::integral_constant<int, QLO + c>{});
                    if constexpr (CK == 4) copy2(t + 2, std::integral_constant<int, c>{});
                }
            });
            __builtin_amdgcn_sched_barrier(0);
        });
    };
    using C0 = std::integral_constant<int, 0>;
    using C1 = std::integral_constant<int, 1>;
    using C2 = std::integral_constant<int, 2>;
    using C3 = std::integral_constant<int, 3>;
    using C4 = std::integral_constant<int, 4>;

    // tiles 0 and 1 whole (tile 1 reads nothing when nk == 1), then wait for tile 0
    static_for<Q2>([&](auto q) { copy2(0, q); });
    static_for<Q3>([&](auto q) { copy3(0, 0, q); });
    static_for<Q2>([&](auto q) { copy2(1, q); });
    static_for<Q3>([&](auto q) { copy3(1, 1, q); });
    vm_wait<Q2 + Q3>();
    block_sync();
    F f0, f1;
    static_for<N_READS>([&](auto idx) { read_part(f0, 0, 0, 0, idx); });
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
    int r0 = 0, r1 = 1, r2 = 2;          // three-stage operand: stages of tiles t, t+1, t+2
    for (int t = 0; t < nk - 1; ++t) {
        const int st = t & 1;
        __builtin_amdgcn_sched_barrier(0);
        step(f0, f1, st, r0, 1, C1{}, t, r2);
        __builtin_amdgcn_s_waitcnt(0xc07f);
        step(f1, f0, st, r0, 2, C2{}, t, r2);
        __builtin_amdgcn_s_waitcnt(0xc07f);
        step(f0, f1, st, r0, 3, C3{}, t, r2);
        __builtin_amdgcn_s_waitcnt(0xc07f);
        vm_wait<Q3>();  // only the three-stage operand's copies of tile t+2 may still be in flight
        block_sync();   // every wave's share of tile t+1 landed; two-stage stage st is free
        step(f1, f0, st ^ 1, r1, 0, C4{}, t, r2);
        __builtin_amdgcn_s_waitcnt(0xc07f);
        const int rt = r0;
        r0 = r1;
        r1 = r2;
        r2 = rt;
    }
    // last K tile: no copies, no barrier
    const int st = (nk - 1) & 1;
    __builtin_amdgcn_sched_barrier(0);
    step(f0, f1, st, r0, 1, C0{}, 0, 0);
    __builtin_amdgcn_s_waitcnt(0xc07f);
    step(f1, f0, st, r0, 2, C0{}, 0, 0);
    __builtin_amdgcn_s_waitcnt(0xc07f);
    step(f0, f1, st, r0, 3, C0{}, 0, 0);
    static_for<MI * NI>([&](auto kc) {
        constexpr int k = decltype(kc)::value;
        mfma32_bf16(acc[k / NI][k % NI], f1.a[k / NI], f1.b[k % NI]);
    });
}

// Exchange of one workgroup tile's fp32 accumulators between workgroups of
// one XCD (the in-kernel split sums): a partial-sum tile of BM x BN floats,
// each wave's accumulators in register order (16-byte pieces, lane-
// contiguous: piece p of wave w at byte ((w * pieces + p) * 1024 + lane * 16)),
// and a 128-byte flag line holding a 64-bit epoch.  Stores use workgroup-
// scope write-through of L1, so they sit in the XCD's L2; loads bypass L1 and
// read the L2's copy.  The per-lane part of every address is lane * 16 and the
// rest is wave-uniform (a scalar offset), so no per-piece address registers
// are needed and all of a block's loads can be in flight at once.
template <int BM, int BN>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t partial_rsrc(float* base, int slot) {
    constexpr uint32_t TILE_BYTES = (uint32_t)BM * BN * 4;
    return make_rsrc(reinterpret_cast<char*>(base) + (size_t)slot * TILE_BYTES, TILE_BYTES);
}
// Stores the accumulators, waits until every wave's stores are in L2, then
// raises the flag to `epoch`.
// This wave's accumulators into its part of the tile's partial-sum area
// (workgroup-scope write-through, so they sit in the XCD's L2), then a wait
// until they are there.
template <int MI, int NI>
__device__ __forceinline__ void partial_store(const f32x16_t (&acc)[MI][NI], __amdgpu_buffer_rsrc_t rp, int wid,
                                              int lane) {
    const int vo = lane * 16, wbase = wid * MI * NI * 4 * 1024;
    static_for<MI>([&](auto i) {
        static_for<NI>([&](auto j) {
            static_for<4>([&](auto c) {
                constexpr int cc = decltype(c)::value;
                constexpr int piece = (decltype(i)::value * NI + decltype(j)::value) * 4 + cc;
                const f32x16_t& v = acc[decltype(i)::value][decltype(j)::value];
                const i32x4_t w = __builtin_bit_cast(i32x4_t, f32x4_t{v[4 * cc], v[4 * cc + 1], v[4 * cc + 2], v[4 * cc + 3]});
                __builtin_amdgcn_raw_buffer_store_b128(w, rp, vo, wbase + piece * 1024, 1);
            });
        });
    });
    vm_wait<0>();
}
template <int MI, int NI>
__device__ __forceinline__ void partial_publish(const f32x16_t (&acc)[MI][NI], __amdgpu_buffer_rsrc_t rp,
                                                __amdgpu_buffer_rsrc_t rf, uint64_t epoch, int wid, int lane) {
    partial_store<MI, NI>(acc, rp, wid, lane);  // this wave's pieces are in L2
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint2 e = make_uint2((uint32_t)epoch, (uint32_t)(epoch >> 32));
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(__attribute__((ext_vector_type(2))) int, e), rf, 0, 0, 1);
    }
}
// Thread 0 polls the flag until it holds `expect` or `ticks` of the 100 MHz
// clock have passed; every thread gets the outcome (through `*okword`, one LDS
// word no wave is using).
__device__ __forceinline__ bool partial_wait(__amdgpu_buffer_rsrc_t rf, uint64_t expect, uint64_t ticks, int* okword) {
    if (threadIdx.x == 0) {
        const uint64_t t0 = wall_clock64();
        int good = 0;
        for (;;) {
            const auto v = __builtin_amdgcn_raw_buffer_load_b64(rf, 0, 0, 17);
            const uint64_t got = (uint64_t)(uint32_t)v[0] | ((uint64_t)(uint32_t)v[1] << 32);
            if (got == expect) { good = 1; break; }
            if (wall_clock64() - t0 > ticks) break;
            __builtin_amdgcn_s_sleep(2);
        }
        *okword = good;
    }
    __syncthreads();
    const bool ok = __builtin_amdgcn_readfirstlane(*okword) != 0;
    __syncthreads();  // the word may be overwritten after this
    return ok;
}
// acc += the partial-sum tile, element by element in register order: the 4 * NI
// pieces of one row of accumulator blocks are loaded together, then added.
template <int MI, int NI>
__device__ __forceinline__ void partial_add(f32x16_t (&acc)[MI][NI], __amdgpu_buffer_rsrc_t rp, int wid, int lane) {
    const int vo = lane * 16, wbase = wid * MI * NI * 4 * 1024;
    static_for<MI>([&](auto i) {
        constexpr int ii = decltype(i)::value;
        f32x4_t p[NI][4];
        static_for<NI>([&](auto j) {
            static_for<4>([&](auto c) {
                constexpr int piece = (ii * NI + decltype(j)::value) * 4 + decltype(c)::value;
                p[decltype(j)::value][decltype(c)::value] =
                    __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rp, vo, wbase + piece * 1024, 17));
            });
        });
        __builtin_amdgcn_sched_barrier(0);  // every load of the row issued before the first add
        static_for<NI>([&](auto j) {
            f32x16_t& v = acc[ii][decltype(j)::value];
            static_for<4>([&](auto c) {
                constexpr int cc = decltype(c)::value;
                const f32x4_t& q = p[decltype(j)::value][cc];
                v[4 * cc] = q[0] + v[4 * cc];
                v[4 * cc + 1] = q[1] + v[4 * cc + 1];
                v[4 * cc + 2] = q[2] + v[4 * cc + 2];
                v[4 * cc + 3] = q[3] + v[4 * cc + 3];
            });
        });
    });
}
// Stream-K partial sums in tile layout: slot s holds a BM x BN fp32 tile,
// row-major (tile-local row r, column c at byte (r * BN + c) * 4).  A
// workgroup writes its accumulators there through each wave's LDS staging
// rows (16-byte stores, workgroup-scope write-through of L1, so they sit in
// the XCD's L2), waits until every wave's stores are in L2 and raises its
// flag to `epoch`.
template <int BN, int MI, int NI, int WTM, int WTN, int NW>
__device__ __forceinline__ void sk_publish(f32x16_t (&acc)[MI][NI], char* smem, __amdgpu_buffer_rsrc_t rp,
                                           __amdgpu_buffer_rsrc_t rf, uint64_t epoch, int wm, int wn, int wid,
                                           int lane) {
    constexpr int EPI_LD = WTN * 4 + 16, Q = WTN / 4, RPI = 64 / Q, IT = 32 / RPI;
    char* epi = smem + wid * 32 * EPI_LD;
    const int rl = lane / Q, c4l = lane % Q;
    const int vo = (rl * BN + wn * WTN + 4 * c4l) * 4;
    static_for<MI>([&](auto i) {
        static_for<NI>([&](auto j) {
            static_for<16>([&](auto v) {
                constexpr int vv = decltype(v)::value;
                const int r = 8 * (vv >> 2) + 4 * (lane >> 5) + (vv & 3);
                *reinterpret_cast<float*>(epi + r * EPI_LD + (decltype(j)::value * 32 + (lane & 31)) * 4) =
                    acc[decltype(i)::value][decltype(j)::value][vv];
            });
        });
        // the staging rows belong to this wave; its LDS accesses are performed in order
        asm volatile("" : : : "memory");
        static_for<IT>([&](auto it_c) {
            constexpr int it = decltype(it_c)::value;
            const float4 v = *reinterpret_cast<const float4*>(epi + (rl + it * RPI) * EPI_LD + c4l * 16);
            const int so = (wm * WTM + decltype(i)::value * 32 + it * RPI) * BN * 4;
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4_t, v), rp, vo, so, 1);
        });
        asm volatile("" : : : "memory");
    });
    vm_wait<0>();  // this wave's stores are in L2
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint2 e = make_uint2((uint32_t)epoch, (uint32_t)(epoch >> 32));
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(__attribute__((ext_vector_type(2))) int, e), rf, 0, 0, 1);
    }
}

// Epilogue term of a stream-K owner: the partial sums of its contributors'
// slots (first_slot, first_slot + stride, ...; n of them), added in that order
// to every group of 4 accumulators, or NaN when a wait expired (ok == false).
template <int BN, int BM>
struct SkPartials {
    static constexpr bool kActive = true;
    float* partial;
    int first_slot, stride, n;
    bool ok;
    template <int IT>
    __device__ __forceinline__ void slab(float4 (&v)[IT], int r, int c, int step) const {
        for (int k = 0; k < n; ++k) {
            const __amdgpu_buffer_rsrc_t rp = partial_rsrc<BM, BN>(partial, first_slot + k * stride);
            f32x4_t p[IT];
            static_for<IT>([&](auto it_c) {
                constexpr int it = decltype(it_c)::value;
                p[it] = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rp, ((r + it * step) * BN + c) * 4, 0, 17));
            });
            __builtin_amdgcn_sched_barrier(0);  // every load of the slab issued before the first add
            static_for<IT>([&](auto it_c) {
                constexpr int it = decltype(it_c)::value;
                v[it].x += p[it][0]; v[it].y += p[it][1]; v[it].z += p[it][2]; v[it].w += p[it][3];
            });
        }
        if (!ok) static_for<IT>([&](auto it_c) { v[decltype(it_c)::value] = make_float4(__builtin_nanf(""), __builtin_nanf(""), __builtin_nanf(""), __builtin_nanf("")); });
    }
    __device__ __forceinline__ void one(float4& v, int r, int c) const {
        float4 w[1] = {v};
        for (int k = 0; k < n; ++k) {
            const f32x4_t p = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(
                partial_rsrc<BM, BN>(partial, first_slot + k * stride), (r * BN + c) * 4, 0, 17));
            w[0].x += p[0]; w[0].y += p[1]; w[0].z += p[2]; w[0].w += p[3];
        }
        if (!ok) w[0] = make_float4(__builtin_nanf(""), __builtin_nanf(""), __builtin_nanf(""), __builtin_nanf(""));
        v = w[0];
    }
};

template <int MI, int NI>
__device__ __forceinline__ void acc_fill_nan(f32x16_t (&acc)[MI][NI]) {
    static_for<MI>([&](auto i) {
        static_for<NI>([&](auto j) {
            static_for<16>([&](auto v) { acc[decltype(i)::value][decltype(j)::value][decltype(v)::value] = __builtin_nanf(""); });
        });
    });
}

// Two-stage kernel, any tile shape of the table.  Per K tile t (stage t & 1),
// four 16-deep K steps:
//   ks 0..2: MFMAs of step ks, reads of step ks+1 (alternating fragment sets)
//   wait for tile t+1's copies, barrier (every wave is done reading stage
//     t, so it may be overwritten)
//   ks 3:    MFMAs of step 3, reads of step 0 of tile t+1, copies of tile
//            t+2 into stage t & 1
// KFULL: every K slice is a whole number of 64-deep tiles, so the copies take
// their offsets as base + delta (one add per copy instead of the range checks).
//
// 256x256 and 256x128 tiles (8 or 4 waves) and 128x128 tiles (4 waves) use a
// different ring (RING3): two A stages and three B stages (2 x 32 + 3 x 32 KB,
// the whole LDS, for 256x256; 112 KB for 256x128; 80 KB, as before, for
// 128x128).  The
// copies of tile t+2 into a two-stage ring can only start once every wave is
// done with stage t, i.e. in step 3, so all 64 copies of the workgroup
// arrived as one burst: the CU accepts about 16-20 copies and then stalls
// further issue while it drains them at about 24 cycles per 1 KB, and a wave
// stalled on a copy issues no MFMAs.  With a third B stage the B copies of
// tile t+2 go to the stage of tile t-1 (free since the last barrier) and are
// issued in steps 0-2; only the A copies remain in step 3 (256x256 with 8
// waves and 128x128 with 4: 4 + 4 copies per wave; 256x256 with 4 waves
// issues twice as many):
//   ks 0: B copies q 0, 1   ks 1: B copy q 2   ks 2: B copy q 3
//   wait until at most those 4 are in flight (tile t+1 has landed), barrier
//   ks 3: A copies q 0-3 into A stage t & 1
// The last K tile runs without copies and without a barrier.
template <int BM, int BN, bool TB, int WM = 2, int WN = 2, bool KFULL = false, bool FIX = false>
__global__ __launch_bounds__(64 * WM * WN) void gemm_dma_kernel(GemmArgs a, TileMapArgs tmap) {
    gemm_batch_offset(a);
    constexpr int NW = WM * WN, STAGES = 2, BK = 64;
    constexpr int WTM = BM / WM, WTN = BN / WN, MI = WTM / 32, NI = WTN / 32;
    constexpr int A_BYTES = BM * 128, B_BYTES = BN * 128, STAGE = A_BYTES + B_BYTES;
    using Copier = DmaCopier<BM, BN, TB, NW>;
    constexpr int A_INSTR = Copier::A_INSTR, PER_TILE = Copier::A_INSTR + Copier::B_INSTR;
    static_assert(PER_TILE < 64, "vmcnt range");
    static_assert(NW * 32 * (WTN * 4 + 16) <= STAGES * STAGE, "epilogue staging must fit in LDS");
    // Two stages, then one idle block that copies of K tiles past the end
    // are sent to (see below).
    constexpr int SINK = 1024 * (A_INSTR > Copier::B_INSTR ? A_INSTR : Copier::B_INSTR) * NW;
    __shared__ __attribute__((aligned(1024))) char smem[STAGES * STAGE + SINK];

    const int tid = threadIdx.x, lane = tid & 63;
    // wave-uniform: the copies' LDS destinations are then scalar values
    const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wid / WN, wn = wid % WN;
    int tm, tn;
    map_tile(tmap, tm, tn);
    const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
    const int64_t kbeg = (int64_t)blockIdx.y * tmap.k_per_split;
    const int64_t kend = min(a.K, kbeg + tmap.k_per_split);
    const int nk = kend > kbeg ? (int)((kend - kbeg + BK - 1) / BK) : 0;
    const Copier cp(a, m0, n0, kend, wid, lane);

    // Copy instruction Q of K tile `tile` (A first, then B) into its stage.
    // Copies are issued without a branch: those of a K tile past the last one
    // read nothing (every offset is out of range, so no memory is touched) and
    // land in the idle sink block -- in the last iteration their stage may
    // still be being read.
    const uint32_t smem_base = lds_addr_of(smem);
    auto issue_part = [&](int tile, auto q_c) {
        constexpr int q = decltype(q_c)::value;
        const uint32_t sa = tile < nk ? smem_base + (uint32_t)((tile & 1) * STAGE) : smem_base + (uint32_t)(STAGES * STAGE);
        const int64_t k0 = kbeg + (int64_t)tile * BK;
        const uint32_t sb = tile < nk ? sa + (uint32_t)A_BYTES : sa;
        if constexpr (KFULL) {
            const bool live = tile < nk;
            if constexpr (q < A_INSTR) cp.template a_part_full<q>((uint32_t)(k0 * 2), sa, live);
            else cp.template b_part_full<q - A_INSTR>((uint32_t)(TB ? k0 * 2 : k0 * a.ldb * 2), sb, live);
        } else {
            if constexpr (q < A_INSTR) cp.template a_part<q>(k0, sa);
            else cp.template b_part<q - A_INSTR>(k0, sb);
        }
    };

    f32x16_t acc[MI][NI];
    static_for<MI>([&](auto i) {
        static_for<NI>([&](auto j) {
            static_for<16>([&](auto v) { acc[i][j][decltype(v)::value] = 0.0f; });
        });
    });

    using F = Frag<MI, NI>;
    constexpr int N_READS = MI + NI * (TB ? 1 : 2);  // LDS reads per fragment set
    auto read_part = [&](F& f, int stage, int ks, auto idx_c) {
        const char* sa = smem + stage * STAGE;
        read_frag_part<decltype(idx_c)::value, MI, NI, TB, BN>(f, sa, sa + A_BYTES, ks, wm * WTM, wn * WTN, lane);
    };
    // MI*NI MFMAs of fragment set f; after MFMA number k the side operation
    // side(k) is issued, so loads and copies go out while the matrix core is
    // busy instead of between MFMA groups.  sched_barrier pins the order.
    auto mfma_with = [&](const F& f, auto&& side) {
        static_for<MI * NI>([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            mfma32_bf16(acc[k / NI][k % NI], f.a[k / NI], f.b[k % NI]);
            side(kc);
            __builtin_amdgcn_sched_barrier(0);
        });
    };
    // MFMAs of f with the N_READS reads of (stage, ks) into g, plus (NC > 0)
    // the PER_TILE copies of tile ct, spread evenly over the MFMA slots
    // (slot k issues side ops [k*NOPS/S, (k+1)*NOPS/S), reads first).
    auto step = [&](const F& f, F& g, int stage, int ks, auto nc_c, int ct) {
        constexpr int NC = decltype(nc_c)::value;
        mfma_with(f, [&](auto kc) {
            constexpr int k = decltype(kc)::value;
            constexpr int S = MI * NI, NOPS = N_READS + NC;
            constexpr int lo = (k * NOPS + S - 1) / S, hi = ((k + 1) * NOPS + S - 1) / S;
            static_for<hi - lo>([&](auto d) {
                constexpr int o = lo + decltype(d)::value;
                if constexpr (o < N_READS) read_part(g, stage, ks, std::integral_constant<int, o>{});
                else if constexpr (NC > 0) issue_part(ct, std::integral_constant<int, o - N_READS>{});
            });
        });
    };
    using None = std::integral_constant<int, 0>;

    constexpr bool RING3 = (BM == 256 && (BN == 256 || BN == 128) && (NW == 8 || NW == 4)) || (BM == 128 && BN == 128 && NW == 4);
    if constexpr (RING3) {
        static_assert(2 * A_BYTES + 3 * B_BYTES <= STAGES * STAGE + SINK, "three-stage B ring layout");
        // three B stages (three A stages measured the same on the 8192^3, 8192x1024x16384,
        // 2048x3072x1024 and 32768x512x2560 products)
        if (nk > 0) ring3_main_loop<BM, BN, TB, WM, WN, KFULL, false>(acc, smem, smem_base, cp, a, kbeg, nk, wm, wn, lane);
    } else if (nk > 0) {
        static_for<PER_TILE>([&](auto q) { issue_part(0, q); });
        if (nk > 1) {
            static_for<PER_TILE>([&](auto q) { issue_part(1, q); });
            vm_wait<PER_TILE>();
        } else {
            vm_wait<0>();
        }
        block_sync();
        F f0, f1;
        static_for<N_READS>([&](auto idx) { read_part(f0, 0, 0, idx); });
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): nothing pending at the loop head
        for (int t = 0; t < nk; ++t) {
            const int st = t & 1;
            __builtin_amdgcn_sched_barrier(0);
            step(f0, f1, st, 1, None{}, 0);
            __builtin_amdgcn_s_waitcnt(0xc07f);
            step(f1, f0, st, 2, None{}, 0);
            __builtin_amdgcn_s_waitcnt(0xc07f);
            step(f0, f1, st, 3, None{}, 0);
            __builtin_amdgcn_s_waitcnt(0xc07f);
            if (t + 1 < nk) {
                vm_wait<0>();  // only tile t+1's copies are in flight here
                block_sync();
            }
            // Reads of step 0 of tile t+1 are unconditional (after the last
            // tile they read an idle stage and are unused) so every path
            // reaching the MFMAs has the same LDS requests in flight.
            step(f1, f0, st ^ 1, 0, std::integral_constant<int, PER_TILE>{}, t + 2);
            // The next K step's fragments were requested during these MFMAs;
            // waiting here tells the compiler nothing is pending at the loop
            // head, which keeps it from draining reads it does not need.
            __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
        }
    }
    if constexpr (RING3) vm_wait<0>();  // copies of tiles past the end still write (zeros) into LDS
    if constexpr (FIX) {
        // In-kernel sum of two K slices (tmap.fixup is set for this instance).
        // Both slices of a tile run on one XCD (the host enables this only
        // when they do), so the exchange goes through that XCD's L2.
        const __amdgpu_buffer_rsrc_t rp = partial_rsrc<BM, BN>(a.partial, blockIdx.x);
        if (tmap.fixup == 2) {
            // Each slice finishes the rows of one wave row (slice s: wave row
            // s); its other waves publish their partial sums for the other
            // slice.  a + b = b + a in fp32, so every output is the same sum
            // as in the one-way form.
            static_assert(WM == 2, "the two slices split the tile by wave rows");
            const int y = blockIdx.y;
            const bool mine = wm == y;
            uint64_t* line = tmap.flags + (size_t)blockIdx.x * 16;
            const __amdgpu_buffer_rsrc_t rf_own = make_rsrc(line + 8 * y, 64), rf_other = make_rsrc(line + 8 * (1 - y), 64);
            if (!mine) partial_store<MI, NI>(acc, rp, wid, lane);  // waits for its stores
            __syncthreads();  // every wave is done with the stages and its stores are in L2
            if (threadIdx.x == 0) {
                const uint2 e = make_uint2((uint32_t)tmap.epoch, (uint32_t)(tmap.epoch >> 32));
                __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(__attribute__((ext_vector_type(2))) int, e),
                                                      rf_own, 0, 0, 1);
            }
            const bool ok = partial_wait(rf_other, tmap.expect, tmap.wait_ticks, reinterpret_cast<int*>(smem));
            if (!mine) return;
            if (ok) partial_add<MI, NI>(acc, rp, wid, lane);
            else acc_fill_nan<MI, NI>(acc);
            store_acc_tile<MI, NI, WTM, WTN, NW>(a, acc, smem, m0, n0, wm, wn, wid, lane, FIX);
            return;
        }
        const __amdgpu_buffer_rsrc_t rf = make_rsrc(tmap.flags + (size_t)blockIdx.x * 16, 128);
        if (blockIdx.y == 0) {
            partial_publish<MI, NI>(acc, rp, rf, tmap.epoch, wid, lane);
            return;
        }
        // slice 1: wait for slice 0's flag (bounded; on timeout the tile becomes NaN)
        __syncthreads();  // every wave is done with the stages
        if (partial_wait(rf, tmap.expect, tmap.wait_ticks, reinterpret_cast<int*>(smem))) partial_add<MI, NI>(acc, rp, wid, lane);
        else acc_fill_nan<MI, NI>(acc);
    }
    __syncthreads();
    store_acc_tile<MI, NI, WTM, WTN, NW>(a, acc, smem, m0, n0, wm, wn, wid, lane, FIX);
}


// Stream-K schedule of the three-stage-ring kernel, for products whose tile
// count leaves most compute units idle in a last partial round (the paper's
// allocation of work to processing units, Section 3.4, with the partial
// products of one output tile summed as in its Fig. 2).  One workgroup per
// CU (two for 128x128 tiles, whose ring takes half the LDS), persistent.
// The tiles are cut into sk_parts contiguous ranges, one per XCD (workgroup b
// runs on XCD b % sk_parts under the round-robin dispatch).  The whole rounds
// the range fills go first (all but the last when sk_keep = 1), one whole
// tile per workgroup and round (so the workgroups of an XCD walk K together
// and share their A and B slices in L2); the (tile, 64-deep K tile) units of
// the remaining tiles are then dealt to the XCD's workgroups in equal
// contiguous runs, so each workgroup computes about the same number of MFMAs.  A run is a sequence of
// segments, each one tile's K range [kt0, kt1):
//   * kt0 > 0 (only a run's first segment can start inside a tile): the
//     workgroup leaves its sums in its partial-sum slot (tile layout) and
//     raises its flag;
//   * kt0 == 0: the workgroup owns the tile.  If the tile continues past its
//     run, the continuation belongs to the next workgroups of the XCD, which
//     compute it first thing; the owner computes its own K range, waits for
//     their flags, and its epilogue adds their partial sums in workgroup
//     order (a fixed order, so the result does not depend on timing) before
//     writing C.
// A workgroup's first segment never waits, so every wait ends; each is
// bounded all the same (on timeout the tile becomes NaN).  Exchanges stay
// inside one XCD's L2.
template <int BM, int BN, bool TB, int WM, int WN, bool KFULL>
__global__ __launch_bounds__(64 * WM * WN, BM == 128 ? 2 : 1) void gemm_dma_sk_kernel(GemmArgs a, TileMapArgs tmap) {
    constexpr int NW = WM * WN, BK = 64;
    constexpr int WTM = BM / WM, WTN = BN / WN, MI = WTM / 32, NI = WTN / 32;
    constexpr int A_BYTES = BM * 128, B_BYTES = BN * 128;
    using Copier = DmaCopier<BM, BN, TB, NW>;
    static_assert(Copier::A_INSTR + Copier::B_INSTR < 64, "vmcnt range");
    constexpr int LDS = 2 * A_BYTES + 3 * B_BYTES;
    static_assert(NW * 32 * (WTN * 4 + 16) <= LDS, "epilogue staging must fit in LDS");
    __shared__ __attribute__((aligned(1024))) char smem[LDS];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wid / WN, wn = wid % WN;
    const uint32_t smem_base = lds_addr_of(smem);

    const int parts = tmap.sk_parts, nkt = tmap.sk_nkt;
    const int x = (int)blockIdx.x % parts, li = (int)blockIdx.x / parts, gx = (int)gridDim.x / parts;
    const int tiles = tmap.tiles_m * tmap.tiles_n;
    const int t_lo = x * tiles / parts, t_hi = (x + 1) * tiles / parts;
    // Whole rounds first (every workgroup one whole tile per round, all of
    // them walking K together), then the remaining tiles' units in runs; with
    // sk_keep = 1 the last whole round joins the runs, so a small remainder is
    // not cut into many short shares.  (The host keeps tiles * K tiles below
    // 2^31.  With fewer remaining units than workgroups the last workgroups'
    // runs are empty and start at the end of the last tile, so no owner counts
    // them as contributors.)
    const int full = max(0, (t_hi - t_lo) / gx - tmap.sk_keep), s_lo = t_lo + full * gx;
    const int units = (t_hi - s_lo) * nkt, base = units / gx, rem = units - base * gx;
    auto run_begin = [&](int i) { return i * base + min(i, rem); };

    f32x16_t acc[MI][NI];
    int u = run_begin(li);
    const int u_end = run_begin(li + 1);
    for (int r = 0; r < full || u < u_end;) {
        int tile, tl = 0, kt0 = 0, kt1 = nkt;
        if (r < full) {
            tile = t_lo + r * gx + li;
            ++r;
        } else {
            tl = u / nkt;
            kt0 = u - tl * nkt;
            kt1 = min(nkt, kt0 + (u_end - u));
            tile = s_lo + tl;
            u += kt1 - kt0;
        }
        int tm, tn;
        tile_coords(tmap, tile, tm, tn);
        const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
        const int64_t kbeg = (int64_t)kt0 * BK, kend = min(a.K, (int64_t)kt1 * BK);
        // The lane index goes through an empty asm each segment, so the
        // compiler recomputes the per-lane LDS, copy and store offsets in
        // each segment instead of hoisting them out of the segment loop and
        // holding them in registers across the main loop.
        int ln = lane;
        asm volatile("" : "+v"(ln));
        static_for<MI>([&](auto i) {
            static_for<NI>([&](auto j) {
                static_for<16>([&](auto v) { acc[i][j][decltype(v)::value] = 0.0f; });
            });
        });
        const Copier cp(a, m0, n0, kend, wid, ln);
        ring3_main_loop<BM, BN, TB, WM, WN, KFULL, false>(acc, smem, smem_base, cp, a, kbeg, kt1 - kt0, wm, wn, ln);
        vm_wait<0>();     // copies of K tiles past the segment still write (zeros) into LDS
        __syncthreads();  // every wave is done with the stages the staging rows overlap
        if (kt0 > 0) {
            sk_publish<BN, MI, NI, WTM, WTN, NW>(acc, smem, partial_rsrc<BM, BN>(a.partial, blockIdx.x),
                                                 make_rsrc(tmap.flags + (size_t)blockIdx.x * 16, 128), tmap.epoch, wm,
                                                 wn, wid, ln);
        } else {
            // the tile's later K tiles: runs of workgroups li+1, li+2, ... of this XCD
            SkPartials<BN, BM> ex{a.partial, (li + 1) * parts + x, parts, 0, true};
            const int tile_end = (tl + 1) * nkt;
            for (int j = li + 1; kt1 < nkt && j < gx && run_begin(j) < tile_end; ++j) {
                const int slot = j * parts + x;
                ex.ok = partial_wait(make_rsrc(tmap.flags + (size_t)slot * 16, 128), tmap.expect, tmap.wait_ticks,
                                     reinterpret_cast<int*>(smem)) && ex.ok;
                ++ex.n;
            }
            store_acc_tile<MI, NI, WTM, WTN, NW>(a, acc, smem, m0, n0, wm, wn, wid, ln, true, ex);
        }
        __syncthreads();  // the next segment's copies overwrite the stages / staging rows
    }
}

}  // namespace isam
