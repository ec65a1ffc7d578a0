// GRU recurrence as one persistent kernel.
//
// The paper schedules a recurrent loop body three times -- a priming
// iteration that leaves buffers next to the compute units, a recursive
// iteration run as often as needed with weights persistent, and a finish
// iteration that puts the results where the next consumer wants them
// (Section 3.6) -- and credits its GRU results to fusing the cell's
// element-wise work with the matrix products and keeping reused data on-chip
// (Section 6.2.2).  On gfx950 that becomes:
//   priming   : every workgroup copies its slice of U (the rows of all three
//               gates for its hidden units) into LDS once;
//   recursive : per step, a 16x16 MFMA contraction of that U slice with the
//               bf16 (or fp32) copy of h_{t-1}, split over 4 waves along K
//               and reduced through LDS, then the r/z/n gate math fused in
//               the epilogue, then a grid-wide barrier;
//   finish    : h_T written to its output.
// The input projection x_t W^T for all t is one GEMM launched before this
// kernel (it does not depend on h).
//
// Cell (gate rows of W and U stacked r, z, n):
//   r = sigmoid(Gx_r + b_r + (U_r h)),  z = sigmoid(Gx_z + b_z + (U_z h)),
//   n = tanh(Gx_n + b_n + r * ((U_n h) + b_hn)),  h' = (1 - z) n + z h.
// The U_n h product is complete before it is scaled by r.
//
// All workgroups must be co-resident.  The host launches no more of them
// than the device holds at once (occupancy query), as an ordinary kernel: on
// a device with nothing else running every workgroup is then resident from
// the start (a cooperative launch would guarantee it even beside other work,
// but costs about 17 us of extra gaps around the kernel).  Every barrier
// wait is bounded and raises an error flag instead of spinning forever, so a
// launch that shares the device with work that holds CUs for longer ends
// with NaN outputs rather than a hang.
#include <algorithm>
#include <cstdlib>
#include <mutex>

#include "common.hpp"
#include "kernels.hpp"

namespace isam {
namespace {

constexpr int kWaves = 4;
constexpr int kSyncWords = kGruSyncBytes / 4;
constexpr int kRedLd = 20;  // floats per row of the cross-wave sums (20: the 4 row groups written by
                            // one store instruction fall on different banks)

__host__ __device__ __forceinline__ int gru_rows(int J) { return ((3 * J + 15) / 16) * 16; }
// U rows in LDS: a multiple of 256 bytes, so the chunk swizzle below stays
// inside the row.
__host__ __device__ __forceinline__ int64_t gru_row_bytes(int64_t H, int64_t es) { return (H * es + 255) / 256 * 256; }
// 16-byte chunk c of U row r sits at chunk c ^ (2 * (r & 7)): the 16 lanes of
// every ds_read_b128 phase (rows r = lane % 16, chunk offsets lane / 16) then
// fall on 16 different bank groups.
__device__ __forceinline__ int u_chunk(int r, int c) { return c ^ (2 * (r & 7)); }

// Cross-workgroup exchange of h and the step barrier.
//
// h_{t-1} travels between workgroups (and XCDs, whose L2 caches are not
// coherent with each other) through a ring of T+1 slots, one per step: h_t is
// written to slot t+1 with device-scope (sc1) stores, which write through to
// the device coherence point.  A store counts as complete (vmcnt) only once
// that write is acknowledged, and s_barrier does not wait for the stores of
// the other waves, so every wave waits for vmcnt(0) itself before the
// workgroup barrier that precedes the arrival atomic: no workgroup signals
// arrival while any of its h stores is still in flight.
//
// After the barrier, slot t+1 is read with ordinary (L2-cached) loads.  No
// workgroup reads any line of slot t+1 before barrier t: slots are padded to
// whole 256-byte blocks, so the lines of slot t (read during step t) never hold
// bytes of slot t+1, and a line of slot t+1 enters an XCD's L2 only through
// the write-through stores of that XCD's own workgroups, which carry no stale
// bytes.  The first reader on each XCD then brings the slot into that XCD's L2
// for the other workgroups there -- each step's state leaves memory once per
// XCD instead of once per workgroup.  The kernel boundary (whose acquire
// invalidates the caches) separates launches that reuse the ring.
//
// The barrier is two-level to limit serialised atomics on one address:
// workgroups arrive on a counter of their group (a.barrier_group members:
// 8, or more when a domain would need more than 31 groups), the last arrival
// of a group bumps the domain counter, and every workgroup polls the domain
// counter.  All counters are monotonic over the steps of one launch (zeroed
// by the init kernel).  Each wait is bounded in time; a timeout sets the
// sticky error word, after which every wait returns at once, and the check
// kernel launched behind the recurrence then fills h_seq and h_T with NaN.

constexpr int kSyncError = 0;           // word offsets; counters sit 64 bytes apart
constexpr int kSyncDomainWords = 512;   // per batch group: global counter + group counters
constexpr int kCpolDevice = 16;         // sc1: device-scope coherence

// Workgroups of one batch group form a barrier domain: batch groups are
// independent sequences, so they never wait for each other.
__device__ __forceinline__ void grid_barrier(const GruArgs& a, int64_t step, int domain, int member, int n_members) {
    // Every wave's h stores must be complete before the workgroup can arrive.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned* sync = a.sync;
        const int kGroup = a.barrier_group;
        unsigned* dom = sync + kSyncDomainWords * (1 + domain);
        const int g = member / kGroup;
        const int n_groups = (n_members + kGroup - 1) / kGroup;
        const unsigned gsize = (unsigned)min(kGroup, n_members - g * kGroup);
        const unsigned old = __hip_atomic_fetch_add(dom + 16 * (1 + g), 1u, __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT);
        if (old + 1 == (unsigned)(step + 1) * gsize)
            __hip_atomic_fetch_add(dom, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const unsigned target = (unsigned)(step + 1) * (unsigned)n_groups + (unsigned)a.stall;
        const uint64_t start = wall_clock64();
        while (__hip_atomic_load(dom, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target &&
               __hip_atomic_load(sync + kSyncError, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u) {
            __builtin_amdgcn_s_sleep(2);
            if (wall_clock64() - start > a.timeout_ticks) {
                __hip_atomic_fetch_or(sync + kSyncError, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                break;
            }
        }
    }
    __syncthreads();
}

// Gate nonlinearities on the hardware base-2 exponential and reciprocal (about
// one ulp each, against a dozen dependent instructions for expf and a branch for
// tanhf).  The state is a convex blend of values in [-1, 1], so the absolute
// error these leave in h stays near 1e-7.  exp2 overflows to +inf for very
// negative v, whose reciprocal is 0: both limits come out exact.
__device__ __forceinline__ float gate_sigmoid(float v) {
    return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(v * -1.44269504088896341f));
}
__device__ __forceinline__ float gate_tanh(float v) { return 2.0f * gate_sigmoid(2.0f * v) - 1.0f; }

template <typename T>
__global__ void gru_init_kernel(GruArgs a) {
    const int64_t n = a.batch * a.H;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {  // slot 0 of the ring: h0 in the operand type
        const float v = a.h0 ? a.h0[i] : 0.0f;
        if constexpr (sizeof(T) == 2) static_cast<uint16_t*>(a.hbuf)[i] = (uint16_t)f32_to_bf16(v);
        else static_cast<float*>(a.hbuf)[i] = v;
    }
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i < kSyncWords; i += blockDim.x) a.sync[i] = 0u;
}

template <typename T>
__global__ __launch_bounds__(64 * kWaves) void gru_recurrent_kernel(GruArgs a) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    constexpr int E = 16 / (int)sizeof(T);
    const int J = a.units_per_wg, BB = a.batch_per_wg;
    const int64_t H = a.H, B = a.batch;
    const int RT = gru_rows(J), MT = RT / 16;
    const int row_bytes = (int)gru_row_bytes(H, sizeof(T));
    const int n_ug = (int)(H / J);
    const int ug = blockIdx.x % n_ug, bg = blockIdx.x / n_ug;
    const int64_t j0 = (int64_t)ug * J, b0 = (int64_t)bg * BB;
    const int nb = (int)min((int64_t)BB, B - b0);
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;

    char* u_lds = smem;
    float* red = reinterpret_cast<float*>(smem + RT * row_bytes);  // [kWaves][RT][kRedLd]

    // Priming: U rows (g*H + j0 + jj) for local row g*J + jj; padding rows are zero.
    {
        const int chunks_per_row = (int)(H / E);
        const T* U = static_cast<const T*>(a.U);
        for (int q = tid; q < RT * chunks_per_row; q += 64 * kWaves) {
            const int lr = q / chunks_per_row, c = q - lr * chunks_per_row;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (lr < 3 * J) {
                const int g = lr / J, jj = lr - g * J;
                v = *reinterpret_cast<const uint4*>(U + (g * H + j0 + jj) * H + (int64_t)c * E);
            }
            *reinterpret_cast<uint4*>(u_lds + lr * row_bytes + u_chunk(lr, c) * 16) = v;
        }
    }

    // Owned outputs: thread p < J * nb handles (jj, n) = (p % J, p / J).
    const int p = tid;
    const bool owner = p < J * nb;
    const int jj = owner ? p % J : 0, nn = owner ? p / J : 0;
    const int64_t j = j0 + jj, bb = b0 + nn;
    float h_prev = 0.0f;
    float bias_r = 0.f, bias_z = 0.f, bias_n = 0.f, bias_hn = 0.f;
    if (owner) {
        if (a.h0) h_prev = a.h0[bb * H + j];
        if (a.bias) { bias_r = a.bias[j]; bias_z = a.bias[H + j]; bias_n = a.bias[2 * H + j]; }
        if (a.bias_hn) bias_hn = a.bias_hn[j];
    }
    __syncthreads();

    const int KG = (int)((H * (int64_t)sizeof(T) + 63) / 64);  // 64-byte K groups
    // Wave w owns the contiguous K groups [kg_lo, kg_hi).
    const int kg_lo = (KG * wid) / kWaves, kg_hi = (KG * (wid + 1)) / kWaves;
    const int n_col = lane & 15, quarter = lane >> 4;
    const bool col_ok = n_col < nb;
    const int64_t hb_row = b0 + n_col;

    // Input-projection values of the owned (b, j) for the next step, fetched
    // one step ahead so their latency hides behind the barrier.
    float gx_r = 0.f, gx_z = 0.f, gx_n = 0.f;
    auto fetch_gx = [&](int64_t t) {
        if (owner && t < a.T) {
            const float* gx = a.gx + (t * B + bb) * 3 * H;
            gx_r = gx[j];
            gx_z = gx[H + j];
            gx_n = gx[2 * H + j];
        }
    };
    fetch_gx(0);

    constexpr int kBatch = 8;  // h chunks requested together per lane
    const __amdgpu_buffer_rsrc_t rs_h = make_rsrc(a.hbuf, (uint32_t)((a.T + 1) * a.slot * (int64_t)sizeof(T)));
    for (int64_t t = 0; t < a.T; ++t) {
        const int64_t hcur_off = t * a.slot;  // element offset of h_{t-1}: ring slot t
        f32x4_t acc[4];
#pragma unroll
        for (int m = 0; m < 4; ++m) acc[m] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        for (int kg0 = kg_lo; kg0 < kg_hi; kg0 += kBatch) {
            // Issue every h load of the batch, then the U fragment reads (they
            // do not depend on h), before the first MFMA needs either.
            uint4 hv[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int kg = kg0 + u;
                const int64_t k = (int64_t)(kg * 4 + quarter) * E;
                const bool ok = kg < kg_hi && col_ok && k < H;
                const uint32_t off = ok ? (uint32_t)((hcur_off + hb_row * H + k) * (int64_t)sizeof(T)) : kOob;
                hv[u] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs_h, (int)off, 0, 0));
            }
            uint4 uf[kBatch][3];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int chunk = (kg0 + u) * 4 + quarter;
                const bool kok = kg0 + u < kg_hi && (int64_t)chunk * E < H;
#pragma unroll
                for (int m = 0; m < 3; ++m) {
                    const int r = m * 16 + n_col;
                    uf[u][m] = (m < MT && kok) ? *reinterpret_cast<const uint4*>(u_lds + r * row_bytes + u_chunk(r, chunk) * 16)
                                               : make_uint4(0, 0, 0, 0);
                }
            }
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                if (kg0 + u >= kg_hi) break;
#pragma unroll
                for (int m = 0; m < 3; ++m) {
                    if (m >= MT) break;
                    if constexpr (sizeof(T) == 2) mfma16_bf16(acc[m], uf[u][m], hv[u]);
                    else mfma16_f32x4(acc[m], uf[u][m], hv[u]);
                }
            }
        }
        // acc[m] element v of lane l: local row m*16 + 4*(l/16) + v, batch column l%16
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            if (m >= MT) break;
#pragma unroll
            for (int v = 0; v < 4; ++v)
                red[(wid * RT + m * 16 + 4 * quarter + v) * kRedLd + n_col] = acc[m][v];
        }
        __syncthreads();
        if (owner) {
            float gh[3];
#pragma unroll
            for (int g = 0; g < 3; ++g) {
                float s = 0.0f;
#pragma unroll
                for (int w = 0; w < kWaves; ++w) s += red[(w * RT + g * J + jj) * kRedLd + nn];
                gh[g] = s;
            }
            const float r = gate_sigmoid(gx_r + bias_r + gh[0]);
            const float z = gate_sigmoid(gx_z + bias_z + gh[1]);
            const float n = gate_tanh(gx_n + bias_n + r * (gh[2] + bias_hn));
            const float h = (1.0f - z) * n + z * h_prev;
            h_prev = h;
            if (a.h_seq) a.h_seq[(t * B + bb) * H + j] = h;
            const int64_t hn = (t + 1) * a.slot + bb * H + j;  // ring slot t+1
            if constexpr (sizeof(T) == 2)
                __builtin_amdgcn_raw_buffer_store_b16((unsigned short)f32_to_bf16(h), rs_h, (int)(hn * 2), 0, kCpolDevice);
            else
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(h), rs_h, (int)(hn * 4), 0, kCpolDevice);
        }
        fetch_gx(t + 1);
        if (t + 1 < a.T) grid_barrier(a, t, bg, ug, n_ug);
    }
    if (owner && a.h_T) a.h_T[bb * H + j] = h_prev;
}

// Batch-group form of the persistent recurrence (bf16 weights).  The batch
// columns are independent sequences, so the grid is split into `groups`
// barrier domains: domain g owns a contiguous slice of at most 16 columns and
// runs on P = n_wg / groups workgroups, each owning 32 hidden units (the 96 rows
// of U of their three gates).  Against one domain per 16 columns spread over
// the whole chip this trades more matrix-core work per workgroup (cheap at
// these sizes) for a barrier among P workgroups instead of 128 and an h
// exchange of the domain's own columns only (8 KiB per workgroup and step at
// 4 columns and hidden 1024, instead of 32 KiB).  Workgroup g + groups * r is
// member r of domain g, so under the round-robin dispatch of workgroups to XCDs
// a domain sits on one XCD.
//
// Exchange.  At launch every workgroup publishes its XCC id (device scope) and
// the domain passes one device-scope barrier; then each member reads the ids of
// its domain.  If all members share one XCD (the normal case), h and the step
// flags travel through that XCD's L2: stores with workgroup scope (sc0) reach
// the L2, and loads with system scope (sc0 sc1) miss the per-CU L1 and return
// the L2's copy; the step barrier is one flag word per member (no atomics,
// which are performed beyond the L2) -- member r stores t+1 into word r after
// every wave's stores have completed, and one wave polls the P words.  If the
// members are spread over XCDs, everything goes through device-scope stores,
// loads and the atomic barrier instead.  The choice is made per domain from
// data every member reads alike, so it is uniform within the domain.
//
// Priming: each of the 8 waves loads its K range (H / 8 values) of all 96 rows
// of U into registers, where it stays for the whole launch -- the weights live
// on the register files between steps, as in the paper's recurrent schedule.
// Recursive step: every wave reads the domain's h_{t-1} for its K range from
// ring slot t, runs 6 x KS MFMAs of 16x16x32, and the 8 partial tiles are
// summed through LDS in wave order; the owner threads (unit, column) apply the
// gates, write h_seq (fp32) and ring slot t+1 (bf16), then the domain barrier.
// Finish: h_T.
constexpr int kGWaves = 8;
constexpr int kGRows = 3 * kGruGroupUnits;  // 96 rows of U per workgroup
constexpr int kGMT = kGRows / 16;           // 6 row tiles of 16
constexpr int kCpolGroup = 1;               // sc0: workgroup scope
constexpr int kCpolSystem = 17;             // sc0 sc1: system scope

// Poll the P flag words of a domain (one wave) until each holds at least
// `target`; bounded like the grid barrier, and stops early on the error word.
__device__ __forceinline__ void flag_wait(const GruArgs& a, __amdgpu_buffer_rsrc_t rs_sync, uint32_t flag_off,
                                          int P, unsigned target) {
    const int l = threadIdx.x;  // wave 0
    const uint64_t start = wall_clock64();
    for (unsigned it = 1;; ++it) {
        const unsigned v = (unsigned)__builtin_amdgcn_raw_buffer_load_b32(rs_sync, (int)(flag_off + 4u * (unsigned)(l % P)), 0,
                                                                        kCpolSystem);
        if (__builtin_amdgcn_ballot_w64(l < P && v < target) == 0) break;
        // the sticky error word lives beyond the L2: look at it now and then only
        if ((it & 255u) == 0 && __hip_atomic_load(a.sync + kSyncError, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u)
            break;
        if (wall_clock64() - start > a.timeout_ticks) {
            if (l == 0) __hip_atomic_fetch_or(a.sync + kSyncError, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            break;
        }
    }
}

template <int KS, bool LOCAL>
__device__ __forceinline__ void group_steps(const GruArgs& a, const uint4 (&uf)[kGMT][KS], float* red, int g, int rank,
                                            int P, int64_t c0, int nb, float h_prev, float bias_r, float bias_z,
                                            float bias_n, float bias_hn) {
    constexpr int cp_st = LOCAL ? kCpolGroup : kCpolDevice;
    constexpr int cp_ld = LOCAL ? kCpolSystem : kCpolDevice;
    const int64_t H = a.H, B = a.batch;
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int n_col = lane & 15, quarter = lane >> 4;
    const bool owner = tid < kGruGroupUnits * nb;
    const int jj = owner ? tid % kGruGroupUnits : 0, nn = owner ? tid / kGruGroupUnits : 0;
    const int64_t j = (int64_t)rank * kGruGroupUnits + jj, bb = c0 + nn;
    float gx_r = 0.f, gx_z = 0.f, gx_n = 0.f;
    auto fetch_gx = [&](int64_t t) {
        if (owner && t < a.T) {
            const float* gx = a.gx + (t * B + bb) * 3 * H;
            gx_r = gx[j];
            gx_z = gx[H + j];
            gx_n = gx[2 * H + j];
        }
    };
    fetch_gx(0);
    const bool col_ok = n_col < nb;
    const int64_t h_row = (c0 + n_col) * H;
    const __amdgpu_buffer_rsrc_t rs_h = make_rsrc(a.hbuf, (uint32_t)((a.T + 1) * a.slot * 2));
    const __amdgpu_buffer_rsrc_t rs_sync = make_rsrc(a.sync, (uint32_t)kGruSyncBytes);
    const uint32_t flag_off = (uint32_t)(kGruFlagWord + 64 * g) * 4u;
    for (int64_t t = 0; t < a.T; ++t) {
        uint4 hv[KS];
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            const int64_t k = (int64_t)(wid * KS + s) * 32 + quarter * 8;
            const uint32_t off = col_ok ? (uint32_t)((t * a.slot + h_row + k) * 2) : kOob;
            hv[s] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs_h, (int)off, 0, cp_ld));
        }
        // every h load of the step in flight before the first wait
        __builtin_amdgcn_sched_barrier(0);
        f32x4_t acc[kGMT];
#pragma unroll
        for (int m = 0; m < kGMT; ++m) acc[m] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KS; ++s) {
#pragma unroll
            for (int m = 0; m < kGMT; ++m) mfma16_bf16(acc[m], uf[m][s], hv[s]);
        }
        // acc[m] element v of lane l: local row m*16 + 4*(l/16) + v, column l%16
#pragma unroll
        for (int m = 0; m < kGMT; ++m) {
#pragma unroll
            for (int v = 0; v < 4; ++v) red[(wid * kGRows + m * 16 + 4 * quarter + v) * kRedLd + n_col] = acc[m][v];
        }
        __syncthreads();
        if (owner) {
            float gh[3];
#pragma unroll
            for (int q = 0; q < 3; ++q) {
                float sum = 0.0f;
#pragma unroll
                for (int w = 0; w < kGWaves; ++w) sum += red[(w * kGRows + q * kGruGroupUnits + jj) * kRedLd + nn];
                gh[q] = sum;
            }
            const float r = gate_sigmoid(gx_r + bias_r + gh[0]);
            const float z = gate_sigmoid(gx_z + bias_z + gh[1]);
            const float n = gate_tanh(gx_n + bias_n + r * (gh[2] + bias_hn));
            const float h = (1.0f - z) * n + z * h_prev;
            h_prev = h;
            if (a.h_seq) a.h_seq[(t * B + bb) * H + j] = h;
            const int64_t hn = (t + 1) * a.slot + bb * H + j;  // ring slot t+1
            __builtin_amdgcn_raw_buffer_store_b16((unsigned short)f32_to_bf16(h), rs_h, (int)(hn * 2), 0, cp_st);
        }
        fetch_gx(t + 1);
        if (t + 1 < a.T) {
            if constexpr (LOCAL) {
                // every wave's slot stores complete (in the L2) before the flag
                asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
                __syncthreads();
                if (tid == 0)
                    __builtin_amdgcn_raw_buffer_store_b32((unsigned)(t + 1), rs_sync, (int)(flag_off + 4u * (uint32_t)rank), 0,
                                                          kCpolGroup);
                if (wid == 0) flag_wait(a, rs_sync, flag_off, P, (unsigned)(t + 1) + (unsigned)a.stall);
                __syncthreads();
            } else {
                grid_barrier(a, t + 1, g, rank, P);  // round 0 was the placement check
            }
        } else {
            __syncthreads();
        }
    }
    if (owner && a.h_T) a.h_T[bb * H + j] = h_prev;
}

template <int KS>
__global__ __launch_bounds__(64 * kGWaves) void gru_group_kernel(GruArgs a) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    float* red = reinterpret_cast<float*>(smem);  // [kGWaves][kGRows][kRedLd]
    __shared__ int s_local;
    const int64_t H = a.H, B = a.batch;
    // Workgroup b is slot i = b / X of XCD lane x = b % X (X = a.xcds, the
    // round-robin width of the dispatcher); slots are cut into layers of P,
    // and domain g = x + X * layer takes rank i % P.  Slots of domains past
    // the last one have no work.
    const int G = a.groups, P = (int)(H / kGruGroupUnits), X = a.xcds;
    const int xl = (int)(blockIdx.x % (unsigned)X), slot = (int)(blockIdx.x / (unsigned)X);
    const int layer = slot / P, rank = slot % P;
    const int g = xl + X * layer;
    if (g >= G) return;
    const int64_t c0 = (B * g) / G, c1 = (B * (g + 1)) / G;
    const int nb = (int)(c1 - c0);
    const int64_t j0 = (int64_t)rank * kGruGroupUnits;
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int n_col = lane & 15, quarter = lane >> 4;

    // Placement: publish this workgroup's XCC id, one device-scope barrier of
    // the domain, then compare the ids of all members.
    const __amdgpu_buffer_rsrc_t rs_sync = make_rsrc(a.sync, (uint32_t)kGruSyncBytes);
    if (tid == 0) {
        const unsigned xcc = __builtin_amdgcn_s_getreg((20) | (0 << 6) | (31 << 11)) & 0xfu;  // HW_REG_XCC_ID
        __builtin_amdgcn_raw_buffer_store_b32(xcc, rs_sync, (int)((kGruXccWord + blockIdx.x) * 4u), 0, kCpolDevice);
    }
    grid_barrier(a, 0, g, rank, P);
    if (wid == 0) {
        unsigned id = 0, id0 = 0;
        for (int r0 = 0; r0 < P; r0 += 64) {
            const int r = r0 + lane;
            const unsigned v = r < P ? (unsigned)__builtin_amdgcn_raw_buffer_load_b32(
                                           rs_sync, (int)((kGruXccWord + xl + X * (layer * P + r)) * 4u), 0, kCpolDevice)
                                     : 0u;
            if (r0 == 0) id0 = __builtin_amdgcn_readfirstlane(v);
            id |= (r < P && v != id0) ? 1u : 0u;
        }
        const bool same = __builtin_amdgcn_ballot_w64(id != 0) == 0;
        if (lane == 0) s_local = (same && !a.device_scope) ? 1 : 0;
    }

    // Priming: U fragments of this wave.  Local row lr = m*16 + n_col is unit
    // lr % 32 of gate lr / 32; K-step s of wave w covers K [(w*KS + s)*32, +32),
    // of which this lane carries the 8 values at quarter*8.
    uint4 uf[kGMT][KS];
    {
        const __amdgpu_buffer_rsrc_t rs_u = make_rsrc(a.U, (uint32_t)(3 * H * H * 2));
#pragma unroll
        for (int m = 0; m < kGMT; ++m) {
            const int lr = m * 16 + n_col;
            const int64_t row = (int64_t)(lr / kGruGroupUnits) * H + j0 + lr % kGruGroupUnits;
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                const int64_t k = (int64_t)(wid * KS + s) * 32 + quarter * 8;
                uf[m][s] = buf_load16(rs_u, (uint32_t)((row * H + k) * 2));
            }
        }
    }
    const bool owner = tid < kGruGroupUnits * nb;
    const int jj = owner ? tid % kGruGroupUnits : 0, nn = owner ? tid / kGruGroupUnits : 0;
    const int64_t j = j0 + jj, bb = c0 + nn;
    float h_prev = 0.0f;
    float bias_r = 0.f, bias_z = 0.f, bias_n = 0.f, bias_hn = 0.f;
    if (owner) {
        if (a.h0) h_prev = a.h0[bb * H + j];
        if (a.bias) { bias_r = a.bias[j]; bias_z = a.bias[H + j]; bias_n = a.bias[2 * H + j]; }
        if (a.bias_hn) bias_hn = a.bias_hn[j];
    }
    __syncthreads();
    if (s_local)
        group_steps<KS, true>(a, uf, red, g, rank, P, c0, nb, h_prev, bias_r, bias_z, bias_n, bias_hn);
    else
        group_steps<KS, false>(a, uf, red, g, rank, P, c0, nb, h_prev, bias_r, bias_z, bias_n, bias_hn);
}

// Stepwise form of the same recurrence: the priming, recursive and finish
// iterations as separate kernels launched in order by the host (Section 3.6's
// schedule with T fixed per call).  One launch per step t: every
// workgroup reads its rows of U straight from global memory (they stay in
// the L2 of its XCD from step to step), h_{t-1} in the operand type from ring
// slot t and the fp32 state from hstate[t & 1]; it writes h_t to h_seq[t],
// ring slot t+1, hstate[(t+1) & 1] and, at the last step, h_T.  Kernel
// boundaries order the steps, so there is no grid barrier and no
// co-residency requirement; the arithmetic is that of the persistent kernel.
template <typename T>
__global__ void gru_step_init_kernel(GruArgs a, float* hstate) {
    const int64_t n = a.batch * a.H;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {  // ring slot 0 and state 0: h0
        const float v = a.h0 ? a.h0[i] : 0.0f;
        hstate[i] = v;
        if constexpr (sizeof(T) == 2) static_cast<uint16_t*>(a.hbuf)[i] = (uint16_t)f32_to_bf16(v);
        else static_cast<float*>(a.hbuf)[i] = v;
    }
}

// MT (row tiles of 16 U rows: gru_rows(J) / 16) is a template argument so that
// every load of the step is unconditional: a load whose operand lies outside
// the matrix reads the buffer's out-of-range offset and returns zeros.  With
// MT known only at run time, the loads sit behind branches whose joins make
// the compiler wait for the loads already in flight, one memory round trip
// per K batch instead of one per step.
template <typename T, int MT>
__global__ __launch_bounds__(64 * kWaves) void gru_step_kernel(GruArgs a, float* hstate, int64_t t) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    constexpr int E = 16 / (int)sizeof(T);
    const int J = a.units_per_wg, BB = a.batch_per_wg;
    const int64_t H = a.H, B = a.batch;
    constexpr int RT = MT * 16;
    const int n_ug = (int)(H / J);
    const int ug = blockIdx.x % n_ug, bg = blockIdx.x / n_ug;
    const int64_t j0 = (int64_t)ug * J, b0 = (int64_t)bg * BB;
    const int nb = (int)min((int64_t)BB, B - b0);
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    float* red = reinterpret_cast<float*>(smem);  // [kWaves][RT][kRedLd]

    // Owned outputs: thread p < J * nb handles (jj, n) = (p % J, p / J).
    const bool owner = tid < J * nb;
    const int jj = owner ? tid % J : 0, nn = owner ? tid / J : 0;
    const int64_t j = j0 + jj, bb = b0 + nn;
    float h_prev = 0.f, gx_r = 0.f, gx_z = 0.f, gx_n = 0.f;
    float bias_r = 0.f, bias_z = 0.f, bias_n = 0.f, bias_hn = 0.f;
    if (owner) {
        h_prev = hstate[(t & 1) * B * H + bb * H + j];
        const float* gx = a.gx + (t * B + bb) * 3 * H;
        gx_r = gx[j];
        gx_z = gx[H + j];
        gx_n = gx[2 * H + j];
        if (a.bias) { bias_r = a.bias[j]; bias_z = a.bias[H + j]; bias_n = a.bias[2 * H + j]; }
        if (a.bias_hn) bias_hn = a.bias_hn[j];
    }

    const int KG = (int)((H * (int64_t)sizeof(T) + 63) / 64);  // 64-byte K groups
    // Wave w owns the contiguous K groups [kg_lo, kg_hi).
    const int kg_lo = (KG * wid) / kWaves, kg_hi = (KG * (wid + 1)) / kWaves;
    const int n_col = lane & 15, quarter = lane >> 4;
    const bool col_ok = n_col < nb;
    const int64_t hb_row = b0 + n_col;
    // U row of this lane in row tile m: local row m*16 + n_col = g*J + jj'.
    int64_t u_row[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) {
        const int lr = m * 16 + n_col;
        u_row[m] = lr < 3 * J ? ((lr / J) * H + j0 + lr % J) : -1;
    }
    constexpr int kBatch = 8;  // K groups requested together per lane
    const __amdgpu_buffer_rsrc_t rs_h = make_rsrc(a.hbuf, (uint32_t)((a.T + 1) * a.slot * (int64_t)sizeof(T)));
    const __amdgpu_buffer_rsrc_t rs_u = make_rsrc(a.U, (uint32_t)(3 * H * H * (int64_t)sizeof(T)));
    const int64_t hcur_off = t * a.slot;  // ring slot t holds h_{t-1}
    f32x4_t acc[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[m] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    for (int kg0 = kg_lo; kg0 < kg_hi; kg0 += kBatch) {
        uint4 hv[kBatch], uf[kBatch][MT];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int kg = kg0 + u;
            const int64_t k = (int64_t)(kg * 4 + quarter) * E;
            const bool kok = kg < kg_hi && k < H;
            const uint32_t off = (kok && col_ok) ? (uint32_t)((hcur_off + hb_row * H + k) * (int64_t)sizeof(T)) : kOob;
            hv[u] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs_h, (int)off, 0, 0));
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                const uint32_t uo = (kok && u_row[m] >= 0) ? (uint32_t)((u_row[m] * H + k) * (int64_t)sizeof(T)) : kOob;
                uf[u][m] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs_u, (int)uo, 0, 0));
            }
        }
        // Keep the scheduler from interleaving the MFMAs into the loads above:
        // all of the batch's loads are in flight before the first wait.
        __builtin_amdgcn_sched_barrier(0);
        // Past kg_hi the operands are zeros, so the MFMAs of the whole batch
        // run without a branch.
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                if constexpr (sizeof(T) == 2) mfma16_bf16(acc[m], uf[u][m], hv[u]);
                else mfma16_f32x4(acc[m], uf[u][m], hv[u]);
            }
        }
    }
    // acc[m] element v of lane l: local row m*16 + 4*(l/16) + v, batch column l%16
#pragma unroll
    for (int m = 0; m < MT; ++m) {
#pragma unroll
        for (int v = 0; v < 4; ++v) red[(wid * RT + m * 16 + 4 * quarter + v) * kRedLd + n_col] = acc[m][v];
    }
    __syncthreads();
    if (!owner) return;
    float gh[3];
#pragma unroll
    for (int g = 0; g < 3; ++g) {
        float sum = 0.0f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) sum += red[(w * RT + g * J + jj) * kRedLd + nn];
        gh[g] = sum;
    }
    const float r = gate_sigmoid(gx_r + bias_r + gh[0]);
    const float z = gate_sigmoid(gx_z + bias_z + gh[1]);
    const float n = gate_tanh(gx_n + bias_n + r * (gh[2] + bias_hn));
    const float h = (1.0f - z) * n + z * h_prev;
    if (a.h_seq) a.h_seq[(t * B + bb) * H + j] = h;
    hstate[((t + 1) & 1) * B * H + bb * H + j] = h;
    const int64_t hn = (t + 1) * a.slot + bb * H + j;  // ring slot t+1
    if constexpr (sizeof(T) == 2) static_cast<uint16_t*>(a.hbuf)[hn] = (uint16_t)f32_to_bf16(h);
    else static_cast<float*>(a.hbuf)[hn] = h;
    if (t + 1 == a.T && a.h_T) a.h_T[bb * H + j] = h;
}

// Finish check behind the persistent recurrence: if any barrier wait ran into
// its bound (sticky error word set), the results are not trustworthy, so every
// output element is overwritten with NaN.  The kernel boundary orders this
// after every store of the recurrence.
__global__ void gru_error_fill_kernel(const unsigned* sync, float* h_seq, int64_t n_seq, float* h_T, int64_t n_T) {
    if (__hip_atomic_load(sync + kSyncError, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u) return;
    const float nan = __uint_as_float(0x7fc00000u);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_seq; i += stride) h_seq[i] = nan;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_T; i += stride) h_T[i] = nan;
}

__global__ void copy_state_kernel(const float* h0, float* hT, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        hT[i] = h0 ? h0[i] : 0.0f;
}

}  // namespace

int gru_blocks_per_cu(int w_type, size_t lds) {
    const void* fn = w_type == kBF16 ? reinterpret_cast<const void*>(gru_recurrent_kernel<bf16_t>)
                                     : reinterpret_cast<const void*>(gru_recurrent_kernel<float>);
    const int n = resident_per_cu(fn, 64 * kWaves, lds);
    return n > 0 ? n : 1;
}

hipError_t launch_gru_copy_state(const float* h0, float* h_T, int64_t n, hipStream_t s) {
    int blocks = (int)((n + 255) / 256);
    if (blocks > 1024) blocks = 1024;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(copy_state_kernel, dim3(blocks), dim3(256), 0, s, h0, h_T, n);
    return hipGetLastError();
}

hipError_t launch_gru_error_fill(const GruArgs& a, hipStream_t s) {
    const int64_t n_seq = a.h_seq ? a.T * a.batch * a.H : 0, n_T = a.h_T ? a.batch * a.H : 0;
    // A few workgroups: the common case only reads the error word (a large grid costs
    // about 2 us more to dispatch); the fill itself is the rare path.
    int blocks = (int)((std::max(n_seq, n_T) + 255) / 256);
    blocks = blocks > 8 ? 8 : (blocks < 1 ? 1 : blocks);
    hipLaunchKernelGGL(gru_error_fill_kernel, dim3(blocks), dim3(256), 0, s, a.sync, a.h_seq, n_seq, a.h_T, n_T);
    return hipGetLastError();
}

bool gru_group_supported(int64_t H) { return H % 256 == 0 && H >= 256 && H <= 1024; }

size_t gru_group_lds_bytes() { return (size_t)kGWaves * kGRows * kRedLd * sizeof(float); }

hipError_t launch_gru_group(const GruArgs& a, hipStream_t s) {
    void* fn = nullptr;
    switch (a.H / 256) {
        case 1: fn = reinterpret_cast<void*>(gru_group_kernel<1>); break;
        case 2: fn = reinterpret_cast<void*>(gru_group_kernel<2>); break;
        case 3: fn = reinterpret_cast<void*>(gru_group_kernel<3>); break;
        case 4: fn = reinterpret_cast<void*>(gru_group_kernel<4>); break;
        default: return hipErrorInvalidValue;
    }
    const int P = (int)(a.H / kGruGroupUnits);
    if (a.w_type != kBF16 || a.groups <= 0 || a.xcds <= 0 || (a.batch + a.groups - 1) / a.groups > 16 ||
        a.n_wg != a.xcds * P * ((a.groups + a.xcds - 1) / a.xcds) || a.n_wg > kGruMaxWgs)
        return hipErrorInvalidValue;
    const size_t lds = gru_group_lds_bytes();
    hipError_t e = ensure_dynamic_lds(fn, lds);
    if (e != hipSuccess) return e;
    int64_t n = a.batch * a.H;
    int blocks = (int)((n + 255) / 256);
    if (blocks > 1024) blocks = 1024;
    hipLaunchKernelGGL(gru_init_kernel<bf16_t>, dim3(blocks), dim3(256), 0, s, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    GruArgs args = a;
    void* params[] = {&args};
    e = hipLaunchKernel(fn, dim3(a.n_wg), dim3(64 * kGWaves), params, (unsigned)lds, s);
    if (e != hipSuccess) return e;
    return launch_gru_error_fill(a, s);
}

int gru_group_blocks_per_cu(int64_t H) {
    void* fn = nullptr;
    switch (H / 256) {
        case 1: fn = reinterpret_cast<void*>(gru_group_kernel<1>); break;
        case 2: fn = reinterpret_cast<void*>(gru_group_kernel<2>); break;
        case 3: fn = reinterpret_cast<void*>(gru_group_kernel<3>); break;
        case 4: fn = reinterpret_cast<void*>(gru_group_kernel<4>); break;
        default: return 0;
    }
    return resident_per_cu(fn, 64 * kGWaves, gru_group_lds_bytes());
}

size_t gru_lds_bytes(int w_type, int64_t H, int J) {
    const int RT = ((3 * J + 15) / 16) * 16;
    const int64_t es = w_type == kBF16 ? 2 : 4;
    return (size_t)RT * (size_t)gru_row_bytes(H, es) + (size_t)kWaves * RT * kRedLd * sizeof(float);
}

hipError_t launch_gru_recurrent(const GruArgs& a, hipStream_t s) {
    const size_t lds = gru_lds_bytes(a.w_type, a.H, a.units_per_wg);
    void* fn = a.w_type == kBF16 ? reinterpret_cast<void*>(gru_recurrent_kernel<bf16_t>)
                                 : reinterpret_cast<void*>(gru_recurrent_kernel<float>);
    hipError_t e = ensure_dynamic_lds(fn, lds);
    if (e != hipSuccess) return e;
    int64_t n = a.batch * a.H;
    int blocks = (int)((n + 255) / 256);
    if (blocks > 1024) blocks = 1024;
    if (a.w_type == kBF16) hipLaunchKernelGGL(gru_init_kernel<bf16_t>, dim3(blocks), dim3(256), 0, s, a);
    else hipLaunchKernelGGL(gru_init_kernel<float>, dim3(blocks), dim3(256), 0, s, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    GruArgs args = a;
    void* params[] = {&args};
    e = hipLaunchKernel(fn, dim3(a.n_wg), dim3(64 * kWaves), params, (unsigned)lds, s);
    if (e != hipSuccess) return e;
    return launch_gru_error_fill(a, s);
}

// Stepwise schedule: the state init and T step kernels launched in order on
// the caller's stream (kernel boundaries order the steps).  The host enqueues
// faster than the steps run (about 2.7 us of host time per launch against
// 4-10 us per step), so no graph is built and the library keeps no state
// between calls.
static int state_blocks(const GruArgs& a) {
    const int64_t n = a.batch * a.H;
    int64_t b = (n + 255) / 256;
    return (int)(b > 1024 ? 1024 : (b < 1 ? 1 : b));
}

hipError_t launch_gru_steps(const GruArgs& a, float* hstate, hipStream_t s) {
    const bool bf = a.w_type == kBF16;
    const size_t red = (size_t)kWaves * gru_rows(a.units_per_wg) * kRedLd * sizeof(float);
    if (bf) hipLaunchKernelGGL(gru_step_init_kernel<bf16_t>, dim3(state_blocks(a)), dim3(256), 0, s, a, hstate);
    else hipLaunchKernelGGL(gru_step_init_kernel<float>, dim3(state_blocks(a)), dim3(256), 0, s, a, hstate);
    hipError_t e = hipGetLastError();
    const int mt = gru_rows(a.units_per_wg) / 16;
    for (int64_t t = 0; t < a.T && e == hipSuccess; ++t) {
        const dim3 grid(a.n_wg), block(64 * kWaves);
        switch (mt) {
            case 1:
                if (bf) hipLaunchKernelGGL((gru_step_kernel<bf16_t, 1>), grid, block, red, s, a, hstate, t);
                else hipLaunchKernelGGL((gru_step_kernel<float, 1>), grid, block, red, s, a, hstate, t);
                break;
            case 2:
                if (bf) hipLaunchKernelGGL((gru_step_kernel<bf16_t, 2>), grid, block, red, s, a, hstate, t);
                else hipLaunchKernelGGL((gru_step_kernel<float, 2>), grid, block, red, s, a, hstate, t);
                break;
            case 3:
                if (bf) hipLaunchKernelGGL((gru_step_kernel<bf16_t, 3>), grid, block, red, s, a, hstate, t);
                else hipLaunchKernelGGL((gru_step_kernel<float, 3>), grid, block, red, s, a, hstate, t);
                break;
            default: return hipErrorInvalidValue;
        }
        e = hipGetLastError();
    }
    return e;
}

// Workspace of isam_gru_forward_noalloc: a static device array, so that
// callers that cannot allocate (code under graph capture, tight serving loops)
// need not pass one.  Each device holds its own copy for the life of the
// process.  In host code `scratch` names a host-side stand-in, never a device
// address: its device address is looked up once per device with
// hipGetSymbolAddress and only that address is handed to kernels.  Every call
// on a device shares the array, so calls that overlap in time on one device
// race.
static __device__ __align__(256) unsigned char scratch[kGruScratchBytes];

hipError_t gru_scratch(void** ptr) {
    static std::mutex mu;
    static void* addr[64];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    std::unique_lock<std::mutex> lock(mu, std::defer_lock);
    try {
        lock.lock();
    } catch (...) {
        return hipErrorUnknown;
    }
    if (!addr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    return hipSuccess;
}

}  // namespace isam
