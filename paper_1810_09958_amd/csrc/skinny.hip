// Skinny GEMM, C[M][N] = A[M][K] . B[K][N] with N <= 32: the RNN-batch form of
// the paper's first listing (GRU-shaped products, Section 6.2.2).  The
// product is bound by streaming A from HBM once, so the kernel is built
// around that stream:
//   * A never touches LDS: each lane loads 64 contiguous bytes of one row per
//     K group straight into registers in MFMA operand order, and every load
//     of a wave is issued before its first MFMA (16 x 16 bytes per lane in
//     flight);
//   * B's K slice for the workgroup (zero-padded to 32 columns) is copied to
//     LDS with buffer_load ... lds and read as MFMA B fragments: bf16 with
//     ds_read_b64_tr_b16 (N-contiguous rows give K-contiguous fragments), fp32
//     with ds_read_b32;
//   * 8 waves split the workgroup's K slice; their 32-row partial tiles are
//     summed through LDS in wave order, and K slices of different
//     workgroups (split-K) are summed by a separate pass in slice order, so
//     results are deterministic.
// Lane l of a wave handles row (l % 32) and K half g = l / 32.  Within a K
// group of 2*CK values (CK = 32 bf16 or 16 fp32) half g owns
// [g*CK, g*CK + CK); MFMA number s of the group takes the s-th 16-byte piece
// (bf16, 8 K values) or, for fp32, piece s/4 element s%4 -- A and B use the
// same assignment.
#include "common.hpp"
#include "kernels.hpp"

namespace isam {
namespace {

typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16_t lds_v4i16_t;

constexpr int kSkWaves = 8;

__device__ __forceinline__ void sk_dma16(__amdgpu_buffer_rsrc_t rs, uint32_t lds_addr, uint32_t voff) {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %1, %2, 0 offen lds"
        :
        : "s"(lds_addr), "v"(voff), "s"(rs)
        : "memory", "m0");
}

__device__ __forceinline__ uint32_t sk_lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}

// bf16 B rows are 64 bytes (two 32-byte blocks); block b of K row k sits at
// block b ^ ((k >> 1) & 1) so a transpose read of 4 consecutive rows hits 4
// different bank groups.
__device__ __forceinline__ uint32_t sk_b16_off(int k, int col) {
    return (uint32_t)(k * 64 + ((((col >> 4) ^ ((k >> 1) & 1))) << 5) + (col & 15) * 2);
}

template <typename T, int RT, int KC>
__global__ __launch_bounds__(64 * kSkWaves) void skinny_kernel(GemmArgs a) {
    constexpr bool BF = sizeof(T) == 2;
    constexpr int E = 16 / (int)sizeof(T);    // elements per 16 bytes
    constexpr int CK = 64 / (int)sizeof(T);   // K values per lane per group
    constexpr int GK = 2 * CK;                // K values per group
    constexpr int KW = KC / kSkWaves;         // K values per wave
    constexpr int NG = KW / GK;               // groups per wave
    constexpr int ROWB = 32 * (int)sizeof(T); // bytes of one padded B row in LDS
    constexpr int B_BYTES = KC * ROWB;
    static_assert(NG >= 1 && KW % GK == 0, "K slice must split into whole groups");
    static_assert(B_BYTES % (1024 * kSkWaves) == 0, "B slice copy must split evenly");
    __shared__ __attribute__((aligned(1024))) char smem[B_BYTES];

    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int g = lane >> 5, r = lane & 31;
    const int64_t m0 = (int64_t)blockIdx.x * (32 * RT);
    const int split = blockIdx.y;
    const int64_t ks0 = (int64_t)split * KC;  // first K of this workgroup

    const __amdgpu_buffer_rsrc_t rsA = make_rsrc(a.A, (uint32_t)(((a.M - 1) * a.lda + a.K) * (int64_t)sizeof(T)));
    const __amdgpu_buffer_rsrc_t rsB = make_rsrc(a.B, (uint32_t)(((a.K - 1) * a.ldb + a.N) * (int64_t)sizeof(T)));

    // 1. Copy B[ks0 .. ks0+KC)[0 .. 32) into LDS (columns >= N and rows >= K read as zero).
    {
        constexpr int UNITS_PER_ROW = ROWB / 16;
        constexpr int INSTR = B_BYTES / 1024 / kSkWaves;
#pragma unroll
        for (int q = 0; q < INSTR; ++q) {
            const int unit = (wid * INSTR + q) * 64 + lane;
            const int k = unit / UNITS_PER_ROW, pu = unit % UNITS_PER_ROW;
            int col;
            if constexpr (BF) {
                const int pb = pu >> 1;  // physical 32-byte block
                col = ((pb ^ ((k >> 1) & 1)) << 4) + (pu & 1) * 8;
            } else {
                col = pu * 4;
            }
            const int64_t kk = ks0 + k;
            const uint32_t off = (kk < a.K && col < a.N) ? (uint32_t)((kk * a.ldb + col) * (int64_t)sizeof(T)) : kOob;
            sk_dma16(rsB, __builtin_amdgcn_readfirstlane(sk_lds_addr(smem + (wid * INSTR + q) * 1024)), off);
        }
    }

    // 2. Issue every A load of this wave: RT row tiles x NG groups x 4 pieces.
    uint4 av[RT][NG][4];
    const int64_t kw0 = ks0 + (int64_t)wid * KW;
#pragma unroll
    for (int t = 0; t < RT; ++t) {
        const int64_t row = m0 + t * 32 + r;
#pragma unroll
        for (int q = 0; q < NG; ++q)
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                const int64_t k = kw0 + q * GK + g * CK + p * E;
                const uint32_t off = (row < a.M && k < a.K) ? (uint32_t)((row * a.lda + k) * (int64_t)sizeof(T)) : kOob;
                av[t][q][p] = buf_load16(rsA, off);
            }
    }

    // 3. Wait for this wave's copies (issued before the A loads) and for
    //    everyone's, then run the MFMAs.
    {
        constexpr int N_A = RT * NG * 4;
        static_assert(N_A < 64, "vmcnt range");
        asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N_A) : "memory");
    }
    // Barrier without a memory fence: the A loads stay in flight (the
    // compiler waits for each before its first MFMA use).
    asm volatile("" : : : "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" : : : "memory");

    f32x16_t acc[RT];
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[t][v] = 0.0f;

    const int kl0 = wid * KW;  // wave's first K row inside the LDS slice
#pragma unroll
    for (int q = 0; q < NG; ++q) {
        if constexpr (BF) {
            // 4 MFMAs per group; B fragment of MFMA s = K rows kb+s*8 .. +8 of column (lane % 32)
            const int gq = lane >> 4, li = lane & 15;
            const int col = (gq & 1) * 16 + 4 * (li & 3);
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const int kb = kl0 + q * GK + (gq >> 1) * CK + s * 8;
                uint32_t w[4];
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int k = kb + h * 4 + (li >> 2);
                    v4i16_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(smem + sk_b16_off(k, col)));
                    const uint2 u = __builtin_bit_cast(uint2, v);
                    w[2 * h] = u.x;
                    w[2 * h + 1] = u.y;
                }
                const uint4 bfrag = make_uint4(w[0], w[1], w[2], w[3]);
#pragma unroll
                for (int t = 0; t < RT; ++t) mfma32_bf16(acc[t], av[t][q][s], bfrag);
            }
        } else {
            // 16 MFMAs per group; MFMA (p, e) takes K = kb + p*4 + e, one value per lane
#pragma unroll
            for (int p = 0; p < 4; ++p)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int k = kl0 + q * GK + g * CK + p * 4 + e;
                    const float bv = *reinterpret_cast<const float*>(smem + k * ROWB + r * 4);
#pragma unroll
                    for (int t = 0; t < RT; ++t) {
                        const uint4 x = av[t][q][p];
                        const uint32_t xe = e == 0 ? x.x : e == 1 ? x.y : e == 2 ? x.z : x.w;
                        acc[t] = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(xe), bv, acc[t], 0, 0, 0);
                    }
                }
        }
    }

    // 4. Sum the 8 waves' tiles through LDS (B slice no longer needed).
    __syncthreads();
    float* red = reinterpret_cast<float*>(smem);  // [wave][RT*32][32]
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int row = t * 32 + 8 * (v >> 2) + 4 * g + (v & 3);
            red[(wid * RT * 32 + row) * 32 + r] = acc[t][v];
        }
    __syncthreads();
    const bool split_out = gridDim.y > 1;
    for (int o = tid; o < RT * 32 * 32; o += 64 * kSkWaves) {
        const int row = o >> 5, col = o & 31;
        float sum = 0.0f;
#pragma unroll
        for (int w = 0; w < kSkWaves; ++w) sum += red[(w * RT * 32 + row) * 32 + col];
        const int64_t gr = m0 + row;
        if (gr >= a.M || col >= a.N) continue;
        if (split_out) {
            a.partial[((int64_t)split * a.M + gr) * a.N + col] = sum;
        } else {
            const int64_t idx = gr * a.ldc + col;
            if (a.bias) sum += a.bias[col];
            if (a.c_type == kF32) {
                float* C = static_cast<float*>(a.C);
                C[idx] = a.accumulate ? C[idx] + sum : sum;
            } else {
                uint16_t* C = static_cast<uint16_t*>(a.C);
                C[idx] = (uint16_t)f32_to_bf16(a.accumulate ? bf16_to_f32(C[idx]) + sum : sum);
            }
        }
    }
}

// Row-streaming variant (bf16, N <= 32, one pass, no split): a workgroup
// owns 16 rows of C and the whole K range; its 8 waves split K and each runs
// a private 3-stage pipeline of direct-to-LDS copies (64-deep K chunks: A
// 16 rows x 128 bytes, B 64 rows x 64 bytes -- whole cache lines), so no
// workgroup barrier is needed until the final cross-wave sum.  A streams
// from HBM once in 1 KB contiguous copies; 16x16x32 MFMAs take A fragments
// with ds_read_b128 and B fragments with ds_read_b64_tr_b16.
// LDS layouts per stage: A row r (128 bytes) chunk c at c ^ ((r >> 1) & 7);
// B K row k (64 bytes) 32-byte block b at b ^ ((k >> 3) & 1) -- both
// conflict-free for the reads below.
constexpr int kRowsPerWg = 16;
constexpr int kStreamStages = 3;
constexpr int kStageA = kRowsPerWg * 128;   // 2 KB
constexpr int kStageB = 64 * 64;            // 4 KB
constexpr int kStage = kStageA + kStageB;

__device__ __forceinline__ int sr_a_swz(int r) { return (r >> 1) & 7; }
__device__ __forceinline__ uint32_t sr_a_off(int r, int c) { return (uint32_t)(r * 128 + ((c ^ sr_a_swz(r)) << 4)); }
__device__ __forceinline__ uint32_t sr_b_off(int k, int n) {
    return (uint32_t)(k * 64 + ((((n >> 4) ^ ((k >> 3) & 1))) << 5) + (n & 15) * 2);
}

__global__ __launch_bounds__(64 * kSkWaves) void skinny_rows_kernel(GemmArgs a) {
    __shared__ __attribute__((aligned(1024))) char smem[kSkWaves * kStreamStages * kStage];
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int64_t m0 = (int64_t)blockIdx.x * kRowsPerWg;
    const __amdgpu_buffer_rsrc_t rsA = make_rsrc(a.A, (uint32_t)(((a.M - 1) * a.lda + a.K) * 2));
    const __amdgpu_buffer_rsrc_t rsB = make_rsrc(a.B, (uint32_t)(((a.K - 1) * a.ldb + a.N) * 2));
    char* ws = smem + wid * kStreamStages * kStage;  // this wave's stages

    // This wave's K range, in 64-deep chunks.
    const int64_t nchunk_all = (a.K + 63) / 64;
    const int64_t c_lo = nchunk_all * wid / kSkWaves, c_hi = nchunk_all * (wid + 1) / kSkWaves;
    const int nc = (int)(c_hi - c_lo);

    // Copy plan: A copy q (0..1) fills rows 8q .. 8q+7 (lane -> row 8q + lane/8,
    // physical chunk lane%8); B copy q (0..3) fills K rows 16q .. 16q+15 (lane
    // -> row 16q + lane/4, physical 16-byte unit lane%4).
    int64_t a_row_off[2];
    int a_k[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int r = 8 * q + (lane >> 3), pc = lane & 7;
        a_k[q] = (pc ^ sr_a_swz(r)) * 8;
        a_row_off[q] = (m0 + r < a.M) ? (m0 + r) * a.lda : -1;
    }
    int b_kr[4], b_n[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int k = 16 * q + (lane >> 2), pu = lane & 3;  // physical 16-byte unit in the 64-byte row
        const int blk = (pu >> 1) ^ ((k >> 3) & 1);         // logical 32-byte block held there
        b_kr[q] = k;
        b_n[q] = blk * 16 + (pu & 1) * 8;
    }
    // Workgroups start their walk over the wave's chunks at different
    // positions (rotation by workgroup index), so the 32 workgroups of an XCD
    // do not all read the same lines of B from its L2 at the same moment.
    const int rot = nc > 0 ? (int)((blockIdx.x >> 3) % (unsigned)nc) : 0;  // workgroups are dealt to 8 XCDs in turn
    auto issue = [&](int c) {  // position c in this wave's walk
        char* st = ws + (c % kStreamStages) * kStage;
        const int cc = c + rot < nc ? c + rot : c + rot - nc;
        const int64_t k0 = (c_lo + cc) * 64;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int64_t k = k0 + a_k[q];
            const uint32_t off = (a_row_off[q] >= 0 && k < a.K) ? (uint32_t)((a_row_off[q] + k) * 2) : kOob;
            sk_dma16(rsA, __builtin_amdgcn_readfirstlane(sk_lds_addr(st + q * 1024)), off);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int64_t k = k0 + b_kr[q];
            const uint32_t off = (k < a.K && b_n[q] < a.N) ? (uint32_t)((k * a.ldb + b_n[q]) * 2) : kOob;
            sk_dma16(rsB, __builtin_amdgcn_readfirstlane(sk_lds_addr(st + kStageA + q * 1024)), off);
        }
    };

    f32x4_t acc[2];
    acc[0] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    acc[1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const int g = lane >> 4, li = lane & 15;
    if (nc > 0) issue(0);
    if (nc > 1) issue(1);
    for (int c = 0; c < nc; ++c) {
        // Chunk c has landed once at most the copies of chunk c+1 are in flight.
        if (c + 1 < nc) asm volatile("s_waitcnt vmcnt(6)" ::: "memory");
        else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        // Stage (c+2) % 3 was last read for chunk c-1, whose reads completed
        // before its MFMAs: refill it now.
        if (c + 2 < nc) issue(c + 2);
        const char* st = ws + (c % kStreamStages) * kStage;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {  // two 32-deep MFMA steps per chunk
            // A fragment: row li, K chunk ks*4 + g (8 values).
            const uint4 af = *reinterpret_cast<const uint4*>(st + sr_a_off(li, ks * 4 + g));
#pragma unroll
            for (int nt = 0; nt < 2; ++nt) {
                uint32_t w[4];
#pragma unroll
                for (int rr = 0; rr < 2; ++rr) {
                    const int k = ks * 32 + g * 8 + rr * 4 + (li >> 2);
                    const int n = nt * 16 + 4 * (li & 3);
                    v4i16_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(st + kStageA + sr_b_off(k, n)));
                    const uint2 u = __builtin_bit_cast(uint2, v);
                    w[2 * rr] = u.x;
                    w[2 * rr + 1] = u.y;
                }
                mfma16_bf16(acc[nt], af, make_uint4(w[0], w[1], w[2], w[3]));
            }
        }
    }

    // Sum the 8 waves' 16x32 tiles in wave order (stages no longer needed).
    __syncthreads();
    float* red = reinterpret_cast<float*>(smem);  // [wave][16][32]
    // acc[nt] element v of lane l: row 4*(l/16) + v, column nt*16 + l%16
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int v = 0; v < 4; ++v) red[(wid * 16 + 4 * g + v) * 32 + nt * 16 + li] = acc[nt][v];
    __syncthreads();
    for (int o = tid; o < kRowsPerWg * 32; o += 64 * kSkWaves) {
        const int row = o >> 5, col = o & 31;
        float sum = 0.0f;
#pragma unroll
        for (int w = 0; w < kSkWaves; ++w) sum += red[(w * 16 + row) * 32 + col];
        const int64_t gr = m0 + row;
        if (gr >= a.M || col >= a.N) continue;
        const int64_t idx = gr * a.ldc + col;
        if (a.bias) sum += a.bias[col];
        if (a.c_type == kF32) {
            float* C = static_cast<float*>(a.C);
            C[idx] = a.accumulate ? C[idx] + sum : sum;
        } else {
            uint16_t* C = static_cast<uint16_t*>(a.C);
            C[idx] = (uint16_t)f32_to_bf16(a.accumulate ? bf16_to_f32(C[idx]) + sum : sum);
        }
    }
}

// fp32 row-streaming variant: the same one-pass structure (16 rows per
// workgroup, 8 waves splitting K, a private 3-stage pipeline of direct-to-LDS
// copies per wave, fixed-order cross-wave sum), with 32-deep K chunks (A rows
// of 128 bytes -- whole lines; B 32 K rows x 32 columns, 128-byte rows) and
// 16x16x4 fp32 MFMAs fed one value per lane by ds_read_b32: MFMA s of a
// chunk takes K = 4s + q from lane quarter q for both operands.  LDS layouts
// per stage: A row r chunk c at c ^ ((r >> 1) & 7); B K row k 16-byte unit u
// at u ^ (4 * ((k >> 1) & 1)) -- the 64 lanes of every read then fall on 64
// different banks.  Measured against two other schedules (reads of chunk
// c+1 issued during chunk c's MFMAs, with 8 waves x 3 stages or 4 waves x 6
// stages): this one is the fastest (4096x32x4096: 23-25 us against 27-36).
constexpr int kF32Waves = kSkWaves;
constexpr int kF32Stages = kStreamStages;
constexpr int kF32StageA = kRowsPerWg * 128;  // 2 KB
constexpr int kF32StageB = 32 * 128;          // 4 KB
constexpr int kF32Stage = kF32StageA + kF32StageB;
constexpr int kF32CopiesPerChunk = 6;          // 2 A + 4 B copies of 1 KB

__device__ __forceinline__ uint32_t srf_a_off(int r, int k) {
    return (uint32_t)(r * 128 + ((((k >> 2) ^ sr_a_swz(r))) << 4) + (k & 3) * 4);
}
__device__ __forceinline__ uint32_t srf_b_off(int k, int n) {
    return (uint32_t)(k * 128 + ((((n >> 2) ^ (4 * ((k >> 1) & 1)))) << 4) + (n & 3) * 4);
}

__global__ __launch_bounds__(64 * kF32Waves) void skinny_rows_f32_kernel(GemmArgs a) {
    __shared__ __attribute__((aligned(1024))) char smem[kF32Waves * kF32Stages * kF32Stage];
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int64_t m0 = (int64_t)blockIdx.x * kRowsPerWg;
    const __amdgpu_buffer_rsrc_t rsA = make_rsrc(a.A, (uint32_t)(((a.M - 1) * a.lda + a.K) * 4));
    const __amdgpu_buffer_rsrc_t rsB = make_rsrc(a.B, (uint32_t)(((a.K - 1) * a.ldb + a.N) * 4));
    char* ws = smem + wid * kF32Stages * kF32Stage;  // this wave's stages

    // This wave's K range, in 32-deep chunks.
    const int64_t nchunk_all = (a.K + 31) / 32;
    const int64_t c_lo = nchunk_all * wid / kF32Waves, c_hi = nchunk_all * (wid + 1) / kF32Waves;
    const int nc = (int)(c_hi - c_lo);

    // Copy plan: A copy q (0..1) fills rows 8q .. 8q+7 (lane -> row 8q + lane/8,
    // physical chunk lane%8); B copy q (0..3) fills K rows 8q .. 8q+7 (lane ->
    // row 8q + lane/8, physical unit lane%8).
    int64_t a_row_off[2];
    int a_k[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int r = 8 * q + (lane >> 3), pc = lane & 7;
        a_k[q] = (pc ^ sr_a_swz(r)) * 4;
        a_row_off[q] = (m0 + r < a.M) ? (m0 + r) * a.lda : -1;
    }
    int b_kr[4], b_n[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int k = 8 * q + (lane >> 3), pu = lane & 7;
        b_kr[q] = k;
        b_n[q] = (pu ^ (4 * ((k >> 1) & 1))) * 4;
    }
    auto issue = [&](int c) {  // chunk index relative to this wave
        char* st = ws + (c % kF32Stages) * kF32Stage;
        const int64_t k0 = (c_lo + c) * 32;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int64_t k = k0 + a_k[q];
            const uint32_t off = (a_row_off[q] >= 0 && k < a.K) ? (uint32_t)((a_row_off[q] + k) * 4) : kOob;
            sk_dma16(rsA, __builtin_amdgcn_readfirstlane(sk_lds_addr(st + q * 1024)), off);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int64_t k = k0 + b_kr[q];
            const uint32_t off = (k < a.K && b_n[q] < a.N) ? (uint32_t)((k * a.ldb + b_n[q]) * 4) : kOob;
            sk_dma16(rsB, __builtin_amdgcn_readfirstlane(sk_lds_addr(st + kF32StageA + q * 1024)), off);
        }
    };
    const int g = lane >> 4, li = lane & 15;
    // Operands of one chunk: A value and two B values for each of its 8 MFMA K steps.
    struct Frags {
        float av[8], bv[2][8];
    };
    auto read_chunk = [&](int c, Frags& f) {
        const char* st = ws + (c % kF32Stages) * kF32Stage;
#pragma unroll
        for (int s8 = 0; s8 < 8; ++s8) {
            const int k = 4 * s8 + g;
            f.av[s8] = *reinterpret_cast<const float*>(st + srf_a_off(li, k));
#pragma unroll
            for (int nt = 0; nt < 2; ++nt)
                f.bv[nt][s8] = *reinterpret_cast<const float*>(st + kF32StageA + srf_b_off(k, nt * 16 + li));
        }
    };

    f32x4_t acc[2];
    acc[0] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    acc[1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    // chunk c is waited for LEAD-1 chunks after its copies were issued
    constexpr int LEAD = kF32Stages - 1;
    for (int c = 0; c < LEAD && c < nc; ++c) issue(c);
    for (int c = 0; c < nc; ++c) {
        if (c + LEAD - 1 < nc) asm volatile("s_waitcnt vmcnt(%0)" ::"n"((LEAD - 1) * kF32CopiesPerChunk) : "memory");
        else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        Frags cur;
        read_chunk(c, cur);
#pragma unroll
        for (int s8 = 0; s8 < 8; ++s8)
#pragma unroll
            for (int nt = 0; nt < 2; ++nt)
                acc[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(cur.av[s8], cur.bv[nt][s8], acc[nt], 0, 0, 0);
        // the stage of chunk c-1 (read in the previous iteration) takes chunk c + LEAD
        if (c + LEAD < nc) issue(c + LEAD);
    }

    // Sum the waves' 16x32 tiles in wave order (stages no longer needed).
    __syncthreads();
    float* red = reinterpret_cast<float*>(smem);  // [wave][16][32]
    // acc[nt] element v of lane l: row 4*(l/16) + v, column nt*16 + l%16
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int v = 0; v < 4; ++v) red[(wid * 16 + 4 * g + v) * 32 + nt * 16 + li] = acc[nt][v];
    __syncthreads();
    for (int o = tid; o < kRowsPerWg * 32; o += 64 * kF32Waves) {
        const int row = o >> 5, col = o & 31;
        float sum = 0.0f;
#pragma unroll
        for (int w = 0; w < kF32Waves; ++w) sum += red[(w * 16 + row) * 32 + col];
        const int64_t gr = m0 + row;
        if (gr >= a.M || col >= a.N) continue;
        const int64_t idx = gr * a.ldc + col;
        if (a.bias) sum += a.bias[col];
        if (a.c_type == kF32) {
            float* C = static_cast<float*>(a.C);
            C[idx] = a.accumulate ? C[idx] + sum : sum;
        } else {
            uint16_t* C = static_cast<uint16_t*>(a.C);
            C[idx] = (uint16_t)f32_to_bf16(a.accumulate ? bf16_to_f32(C[idx]) + sum : sum);
        }
    }
}

// Narrow product (N < 8, any ldb): the batch-1..7 matrix-vector form, where
// the paper's mapper would pick a dot-product instruction rather than a
// matrix one (Section 4).  Bound by streaming A once.  A workgroup owns 8
// rows; in each wave eight lanes share a row, and the 4 waves split K: wave
// w takes the 64-value K blocks w, w+4, w+8, ... of the current slice, lane j
// of a row the 16-byte piece j of each block (8 lanes read 128 contiguous
// bytes), 16 (bf16) or 8 (fp32) blocks per batch.  Each piece is dotted with the
// matching K values of the N columns of B, which sit transposed in LDS
// (B^T[n][k], zero past K; all lanes with the same j read the same
// address): v_dot2_f32_bf16 for bf16, FMAs for fp32.  K runs in LDS-sized
// slices; the next batch of A loads is always in flight during the
// arithmetic.  At the end the 8 lanes of a row are summed (butterfly), then the
// 4 waves in wave order through LDS, and C is written.
constexpr int kNarrowRows = 8;
constexpr int kNarrowWaves = 4;
constexpr int kNarrowSliceBytes = 64 * 1024;  // B^T slice in LDS

typedef __bf16 nbf16x2_t __attribute__((ext_vector_type(2)));

template <typename T>
__global__ __launch_bounds__(64 * kNarrowWaves) void narrow_kernel(GemmArgs a, int ks_len) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    constexpr bool BF = sizeof(T) == 2;
    constexpr int PIECES = BF ? 1 : 2;  // 16-byte loads per 8 K values
    constexpr int kNarrowUnroll = BF ? 16 : 8;  // blocks per batch and lane
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int N = (int)a.N;
    const int r = lane >> 3, j = lane & 7;
    const int64_t row = (int64_t)blockIdx.x * kNarrowRows + r;
    const bool row_ok = row < a.M;
    const T* B = static_cast<const T*>(a.B);
    T* bt = reinterpret_cast<T*>(smem);  // [N][ks_len]
    const __amdgpu_buffer_rsrc_t rsA = make_rsrc(a.A, (uint32_t)(((a.M - 1) * a.lda + a.K) * sizeof(T)));
    const uint32_t a_row = row_ok ? (uint32_t)(row * a.lda * sizeof(T)) : 0u;
    float acc[7];
#pragma unroll
    for (int n = 0; n < 7; ++n) acc[n] = 0.0f;

    // Batch b of a slice: this wave's blocks wid + 4*(b*U + u), u < U.  The
    // loads of batch b+1 are issued before the arithmetic of batch b, and the
    // first batch of a slice before its B^T is staged.
    uint4 av[kNarrowUnroll][PIECES], nx[kNarrowUnroll][PIECES];
    auto load_batch = [&](uint4 (&dst)[kNarrowUnroll][PIECES], int64_t k0, int blocks, int b) {
#pragma unroll
        for (int u = 0; u < kNarrowUnroll; ++u) {
            const int blk = wid + kNarrowWaves * (b * kNarrowUnroll + u);
            const int kk = blk * 64 + j * 8;
            const bool ok = row_ok && blk < blocks;
#pragma unroll
            for (int p = 0; p < PIECES; ++p)
                dst[u][p] = buf_load16(rsA, ok ? a_row + (uint32_t)((k0 + kk) * sizeof(T)) + p * 16 : kOob);
        }
    };
    for (int64_t k0 = 0; k0 < a.K; k0 += ks_len) {
        const int len = (int)min((int64_t)ks_len, a.K - k0);
        const int blocks = (len + 63) / 64;
        const int batches = (blocks + kNarrowWaves * kNarrowUnroll - 1) / (kNarrowWaves * kNarrowUnroll);
        __syncthreads();  // the previous slice's reads are done
        // Stage B^T: a thread takes 8 consecutive K values of one column per
        // step, its 8 element loads issued together, then the LDS stores.
        for (int g0 = tid; g0 < (ks_len / 8) * N; g0 += 64 * kNarrowWaves) {
            const int n = g0 / (ks_len / 8), kk = (g0 - n * (ks_len / 8)) * 8;
            T v[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = kk + e < len ? B[(k0 + kk + e) * a.ldb + n] : T(0);
            T* d = bt + n * ks_len + kk;
#pragma unroll
            for (int e = 0; e < 8; ++e) d[e] = v[e];
        }
        load_batch(nx, k0, blocks, 0);
        __syncthreads();
        for (int bb = 0; bb < batches; ++bb) {
#pragma unroll
            for (int u = 0; u < kNarrowUnroll; ++u)
#pragma unroll
                for (int p = 0; p < PIECES; ++p) av[u][p] = nx[u][p];
            if (bb + 1 < batches) load_batch(nx, k0, blocks, bb + 1);
#pragma unroll
            for (int u = 0; u < kNarrowUnroll; ++u) {
                const int blk = wid + kNarrowWaves * (bb * kNarrowUnroll + u);
                if (blk >= blocks) break;
                const int kk = blk * 64 + j * 8;
#pragma unroll
                for (int n = 0; n < 7; ++n) {
                    if (n >= N) break;
                    const T* bp = bt + n * ks_len + kk;
                    if constexpr (BF) {
                        const uint4 bv = *reinterpret_cast<const uint4*>(bp);
                        const uint32_t aw[4] = {av[u][0].x, av[u][0].y, av[u][0].z, av[u][0].w};
                        const uint32_t bw[4] = {bv.x, bv.y, bv.z, bv.w};
                        float t = acc[n];
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            t = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(nbf16x2_t, aw[q]),
                                                                __builtin_bit_cast(nbf16x2_t, bw[q]), t, false);
                        acc[n] = t;
                    } else {
                        const float4 b0v = *reinterpret_cast<const float4*>(bp);
                        const float4 b1v = *reinterpret_cast<const float4*>(bp + 4);
                        const float4 a0 = __builtin_bit_cast(float4, av[u][0]);
                        const float4 a1 = __builtin_bit_cast(float4, av[u][PIECES - 1]);
                        float t = acc[n];
                        t = fmaf(a0.x, b0v.x, t); t = fmaf(a0.y, b0v.y, t); t = fmaf(a0.z, b0v.z, t); t = fmaf(a0.w, b0v.w, t);
                        t = fmaf(a1.x, b1v.x, t); t = fmaf(a1.y, b1v.y, t); t = fmaf(a1.z, b1v.z, t); t = fmaf(a1.w, b1v.w, t);
                        acc[n] = t;
                    }
                }
            }
        }
    }
    // Sum the 8 lanes of each row (lane j += lane j^1, then ^2, then ^4),
    // then the 4 waves in wave order.
#pragma unroll
    for (int n = 0; n < 7; ++n) {
        float v = acc[n];
        v += __shfl_xor(v, 1, 64);
        v += __shfl_xor(v, 2, 64);
        v += __shfl_xor(v, 4, 64);
        acc[n] = v;
    }
    __syncthreads();  // B^T reads are done: reuse LDS
    float* red = reinterpret_cast<float*>(smem);  // [wave][row][7]
    if (j == 0) {
#pragma unroll
        for (int n = 0; n < 7; ++n) red[(wid * kNarrowRows + r) * 7 + n] = acc[n];
    }
    __syncthreads();
    if (wid != 0 || j != 0 || !row_ok) return;
#pragma unroll
    for (int n = 0; n < 7; ++n) {
        if (n >= N) break;
        float v = 0.0f;
#pragma unroll
        for (int w = 0; w < kNarrowWaves; ++w) v += red[(w * kNarrowRows + r) * 7 + n];
        if (a.bias) v += a.bias[n];
        const int64_t idx = row * a.ldc + n;
        if (a.c_type == kF32) {
            float* C = static_cast<float*>(a.C);
            C[idx] = a.accumulate ? C[idx] + v : v;
        } else {
            uint16_t* C = static_cast<uint16_t*>(a.C);
            C[idx] = (uint16_t)f32_to_bf16(a.accumulate ? bf16_to_f32(C[idx]) + v : v);
        }
    }
}

}  // namespace

// K depth of one workgroup's slice (the split-K unit) for the skinny kernel.
int64_t skinny_k_slice(int ab_type) { return ab_type == kBF16 ? 2048 : 1024; }
int skinny_rows_per_wg(int ab_type) { return ab_type == kBF16 ? 32 : 64; }

int skinny_stream_rows() { return kRowsPerWg; }

hipError_t launch_narrow(const GemmArgs& a, hipStream_t s) {
    if (a.N < 1 || a.N > 7) return hipErrorInvalidValue;
    const size_t es = a.ab_type == kBF16 ? 2 : 4;
    // K slice: a multiple of 64 whose N x slice B^T fits the LDS budget
    int64_t ks = (int64_t)(kNarrowSliceBytes / (a.N * es)) / 64 * 64;
    if (ks > ((a.K + 63) / 64) * 64) ks = ((a.K + 63) / 64) * 64;
    if (ks < 64) ks = 64;
    // (at least room for the cross-wave sums)
    const size_t lds = std::max<size_t>((size_t)ks * a.N * es, kNarrowWaves * kNarrowRows * 7 * sizeof(float));
    const void* fn = a.ab_type == kBF16 ? reinterpret_cast<const void*>(narrow_kernel<uint16_t>)
                                        : reinterpret_cast<const void*>(narrow_kernel<float>);
    hipError_t e = ensure_dynamic_lds(fn, lds);
    if (e != hipSuccess) return e;
    const dim3 grid((unsigned)((a.M + kNarrowRows - 1) / kNarrowRows)), block(64 * kNarrowWaves);
    if (a.ab_type == kBF16) hipLaunchKernelGGL(narrow_kernel<uint16_t>, grid, block, lds, s, a, (int)ks);
    else hipLaunchKernelGGL(narrow_kernel<float>, grid, block, lds, s, a, (int)ks);
    return hipGetLastError();
}

hipError_t launch_skinny_rows(const GemmArgs& a, hipStream_t s) {
    const dim3 grid((unsigned)((a.M + kRowsPerWg - 1) / kRowsPerWg)), block(64 * kSkWaves);
    if (a.ab_type == kBF16) hipLaunchKernelGGL(skinny_rows_kernel, grid, block, 0, s, a);
    else hipLaunchKernelGGL(skinny_rows_f32_kernel, grid, dim3(64 * kF32Waves), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_skinny(const GemmArgs& a, int splits, hipStream_t s) {
    const int R = skinny_rows_per_wg(a.ab_type);
    const dim3 grid((unsigned)((a.M + R - 1) / R), (unsigned)splits), block(64 * kSkWaves);
    if (a.ab_type == kBF16) hipLaunchKernelGGL((skinny_kernel<bf16_t, 1, 2048>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((skinny_kernel<float, 2, 1024>), grid, block, 0, s, a);
    return hipGetLastError();
}

}  // namespace isam
