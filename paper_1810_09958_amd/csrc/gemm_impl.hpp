// MFMA tile kernel for C (+)= op(A) op(B): the dense contraction of the
// paper's first listing (Section 2), unrolled into compute tiles (Section 3.3),
// allocated to compute units (Section 3.4) and fed HBM -> LDS -> VGPR
// (Section 3.5).
//
// Design (gfx950):
//   * A workgroup owns a BM x BN output tile; 4 waves split it 2x2 (or 4x1).
//   * Both operands are staged in LDS as rows of 128 bytes of K (64 bf16 or
//     32 fp32), i.e. "K-major" whatever the global layout.  An operand whose
//     global layout is K-contiguous is copied chunk by chunk; one whose
//     layout is M/N-contiguous is loaded as E x E blocks and transposed in
//     registers on the way into LDS.
//   * 16-byte chunk c of LDS row r sits at chunk c ^ ((r ^ (r >> 3)) & 7):
//     the fragment reads (consecutive rows, one chunk) and the transposed
//     stores (rows 8 apart, one chunk) both land on distinct bank groups for
//     every 8- and 16-lane phase; the transposed stores also alternate the
//     order of their E rows between lane halves so each phase covers both
//     128-byte halves of a 256-byte bank line.
//   * Two LDS stages: the global loads for tile t+1 are issued before the
//     MFMAs of tile t and written to the other stage after them; one
//     barrier per K tile.
//   * Global loads go through buffer resources: a row or K index past the
//     matrix edge is turned into an out-of-range offset and reads as zero,
//     so ragged tiles need no branches.
//   * Rasterisation: tiles are visited in groups of `group_m` tile rows, and
//     with `xcd_remap` the round-robin dispatch over the 8 XCDs is undone so
//     that each XCD works on a contiguous run of tiles that share A and B
//     panels in its L2.
//   * Split-K (blockIdx.y) writes fp32 partials; a separate kernel reduces
//     them in split order, so results are deterministic.
#pragma once

#include "common.hpp"
#include "kernels.hpp"

namespace isam {

__device__ __forceinline__ uint32_t lds_off(int r, int c) {
    return (uint32_t)(r * 128 + ((c ^ ((r ^ (r >> 3)) & 7)) << 4));
}

// Loads one operand tile (ROWS rows of M or N, 128 bytes of K) into
// registers, then stores it K-major into LDS.
template <typename T, int ROWS, int NT, bool KC, bool VEC>
struct TileLoader {
    static constexpr int E = 16 / (int)sizeof(T);   // elements per 16-byte chunk
    static constexpr int BK = 128 / (int)sizeof(T); // K depth of a tile
    static constexpr int UNITS = KC ? ROWS * 8 : (BK / E) * (ROWS / E);
    static constexpr int NU = (UNITS + NT - 1) / NT;
    static constexpr int NREG = KC ? NU : NU * E;
    uint4 r[NREG];

    __device__ __forceinline__ static bool live(int q) { return (UNITS % NT == 0) || q < UNITS; }

    __device__ __forceinline__ static uint4 load_elems(__amdgpu_buffer_rsrc_t rs, int64_t base_el,
                                                       int64_t step_el, int nvalid) {
        // E elements at base, base+step, ...; elements >= nvalid read as zero.
        uint32_t w[4];
        if constexpr (sizeof(T) == 2) {
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                uint32_t lo = buf_load2(rs, (2 * p < nvalid) ? (uint32_t)((base_el + (2 * p) * step_el) * 2) : kOob);
                uint32_t hi = buf_load2(rs, (2 * p + 1 < nvalid) ? (uint32_t)((base_el + (2 * p + 1) * step_el) * 2) : kOob);
                w[p] = (lo & 0xffffu) | (hi << 16);
            }
        } else {
#pragma unroll
            for (int p = 0; p < 4; ++p)
                w[p] = buf_load4(rs, (p < nvalid) ? (uint32_t)((base_el + p * step_el) * 4) : kOob);
        }
        return make_uint4(w[0], w[1], w[2], w[3]);
    }

    // r0: first row (M or N index) of the tile; k0: first K index;
    // rows_total / kend: valid extents; ld: leading dimension in elements.
    __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rs, int tid, int64_t r0, int64_t k0,
                                         int64_t rows_total, int64_t kend, int64_t ld) {
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            const int q = tid + u * NT;
            const bool lv = live(q);
            if constexpr (KC) {
                const int rr = q >> 3, c = q & 7;
                const int64_t row = r0 + rr, k = k0 + c * E;
                const bool ok = lv && row < rows_total && k < kend;
                if constexpr (VEC) {
                    r[u] = buf_load16(rs, ok ? (uint32_t)((row * ld + k) * (int64_t)sizeof(T)) : kOob);
                } else {
                    int nv = ok ? (int)((kend - k) < E ? (kend - k) : E) : 0;
                    r[u] = load_elems(rs, row * ld + k, 1, nv);
                }
            } else {
                constexpr int RB = ROWS / E;
                const int rb = q % RB, kb = q / RB;
                const int64_t col = r0 + rb * E;
#pragma unroll
                for (int i = 0; i < E; ++i) {
                    const int64_t k = k0 + kb * E + i;
                    const bool ok = lv && k < kend && col < rows_total;
                    if constexpr (VEC) {
                        r[u * E + i] = buf_load16(rs, ok ? (uint32_t)((k * ld + col) * (int64_t)sizeof(T)) : kOob);
                    } else {
                        int nv = ok ? (int)((rows_total - col) < E ? (rows_total - col) : E) : 0;
                        r[u * E + i] = load_elems(rs, k * ld + col, 1, nv);
                    }
                }
            }
        }
    }

    __device__ __forceinline__ void store(char* lds, int tid) const {
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            const int q = tid + u * NT;
            if (!live(q)) continue;
            if constexpr (KC) {
                *reinterpret_cast<uint4*>(lds + lds_off(q >> 3, q & 7)) = r[u];
            } else {
                constexpr int RB = ROWS / E;
                const int rb = q % RB, kb = q / RB;
                uint4 t[E];
                if constexpr (E == 8) transpose8x8_b16(&r[u * E], t);
                else transpose4x4_b32(&r[u * E], t);
                const int flip = (rb >> 3) & 1;
                const uint32_t m = 0u - (uint32_t)flip;  // all ones when flipped
                static_for<E>([&](auto jc) {
                    constexpr int j = decltype(jc)::value;
                    // v = flip ? t[j ^ 1] : t[j], as bit operations so the
                    // register array is never indexed by a run-time value
                    const uint4 a0 = t[j], a1 = t[j ^ 1];
                    const uint4 v = make_uint4(a0.x ^ ((a0.x ^ a1.x) & m), a0.y ^ ((a0.y ^ a1.y) & m),
                                               a0.z ^ ((a0.z ^ a1.z) & m), a0.w ^ ((a0.w ^ a1.w) & m));
                    *reinterpret_cast<uint4*>(lds + lds_off(rb * E + (j ^ flip), kb)) = v;
                });
            }
        }
    }
};

struct TileMapArgs {
    int tiles_m, tiles_n, group_m, xcd_remap;
    int64_t k_per_split;
    // Two K slices summed inside the kernel (256x256 direct-to-LDS kernel
    // only).  fixup = 1: slice 0 leaves its accumulators in `partial` and
    // raises flags[tile] (one 128-byte line per tile) to `epoch`; slice 1 adds
    // them and writes C.  fixup = 2 (every workgroup resident): slice s
    // finishes the rows of wave row s; its other waves leave their
    // accumulators in `partial` and it raises its own flag (word 8 s of the
    // line), then waits for the other slice's.
    int fixup;
    uint64_t epoch;          // value slice 0 writes
    uint64_t expect;         // value slice 1 waits for (== epoch but in the timeout test)
    uint64_t wait_ticks;     // bound of slice 1's wait (100 MHz ticks)
    uint64_t* flags;
    // Stream-K schedule (persistent direct-to-LDS kernel only): the tiles are
    // cut into sk_parts contiguous ranges, one per XCD, and the (tile, K tile)
    // units of a range are dealt evenly to that XCD's workgroups; sk_nkt is
    // the number of 64-deep K tiles per output tile.  The same epoch / expect /
    // wait_ticks / flags protocol as the two-slice sum, one flag line and one
    // partial-sum tile per workgroup.
    int sk_parts, sk_nkt;
    int sk_keep;  // whole rounds left to the stream-K share (0 or 1; see the kernel)
};

// Output tile number `tile` in the grouped rasterisation: groups of group_m
// tile rows, column by column inside a group.
__device__ __forceinline__ void tile_coords(const TileMapArgs& t, int tile, int& tm, int& tn) {
    const int width = t.group_m * t.tiles_n;
    const int group = tile / width;
    const int first_m = group * t.group_m;
    const int gm = min(t.tiles_m - first_m, t.group_m);
    const int inner = tile - group * width;
    tm = first_m + inner % gm;
    tn = inner / gm;
}

__device__ __forceinline__ void map_tile(const TileMapArgs& t, int& tm, int& tn) {
    int bid = blockIdx.x;
    const int G = gridDim.x;
    if (t.xcd_remap && (G & 7) == 0) bid = (bid & 7) * (G >> 3) + (bid >> 3);
    tile_coords(t, bid, tm, tn);
}

// Problem blockIdx.z of a strided batch: offset the operand pointers.
__device__ __forceinline__ void gemm_batch_offset(GemmArgs& a) {
    if (a.batch > 1) {
        const int64_t z = blockIdx.z;
        a.A = static_cast<const char*>(a.A) + z * a.stride_a;
        a.B = static_cast<const char*>(a.B) + z * a.stride_b;
        a.C = static_cast<char*>(a.C) + z * a.stride_c;
    }
}

// No extra terms in the epilogue (see store_acc_tile).
struct NoExtra {
    static constexpr bool kActive = false;
    template <int IT>
    __device__ __forceinline__ void slab(float4 (&)[IT], int, int, int) const {}
    __device__ __forceinline__ void one(float4&, int, int) const {}
};

// Accumulators of the wave's WTM x WTN tile -> C (or the split-K partial
// sums), staged through LDS so every store is a 16-byte (fp32) or 8-byte
// (bf16) vector store.  `smem` must hold NW * 32 * (WTN*4 + 16) bytes and be
// idle (no copies in flight).  An active `extra` adds terms to each group of
// 4 accumulators before the bias: extra.slab(v, r, c, step) to the groups of
// tile rows r, r + step, ... at tile columns c..c+3, extra.one(v, r, c) to one
// group (tile-local coordinates).
template <int MI, int NI, int WTM, int WTN, int NW, typename Extra = NoExtra>
__device__ __forceinline__ void store_acc_tile(const GemmArgs& a, f32x16_t (&acc)[MI][NI], char* smem, int64_t m0,
                                               int64_t n0, int wm, int wn, int wid, int lane, bool fixup = false,
                                               const Extra& extra = Extra{}) {
    const bool split_out = gridDim.y > 1 && !fixup;
    const int split = blockIdx.y;
    constexpr int EPI_LD = WTN * 4 + 16;
    char* epi = smem + wid * 32 * EPI_LD;
    float* P = split_out ? a.partial + (int64_t)split * a.M * a.N : nullptr;
    const int64_t ldo = split_out ? a.N : a.ldc;
    const int osz = split_out ? 4 : (a.c_type == kF32 ? 4 : 2);
    char* obase = split_out ? reinterpret_cast<char*>(P) : static_cast<char*>(a.C);
    const bool vec_out = ((reinterpret_cast<uintptr_t>(obase) & 15) == 0) && ((ldo * osz) % 16 == 0);
    constexpr int Q = WTN / 4;
    // Fast path for slabs wholly inside C: lane l owns the 4-column group l % Q
    // and rows l / Q + RPI * it, so every address is a fixed per-lane base
    // plus a constant step and no element is range-checked.
    constexpr int RPI = 64 / Q, IT = 32 / RPI;
    static_assert(64 % Q == 0 && 32 % RPI == 0, "wave tile width must divide into 4-column groups per lane");
    const bool out_f32 = split_out || a.c_type == kF32;
    const bool add_c = !split_out && a.accumulate;
    const int64_t col0 = n0 + wn * WTN;
    const bool cols_ok = col0 + WTN <= a.N &&
                         (out_f32 ? vec_out
                                  : ((reinterpret_cast<uintptr_t>(obase) & 7) == 0 && (ldo * 2) % 8 == 0));
    const int rl = lane / Q, c4l = lane % Q;
    float4 bias4 = make_float4(0.f, 0.f, 0.f, 0.f);
    if (cols_ok && !split_out && a.bias) {
        const float* bp = a.bias + col0 + 4 * c4l;
        bias4 = make_float4(bp[0], bp[1], bp[2], bp[3]);
    }
    auto slab_fast = [&](int64_t row0, auto f32_c, auto addc_c) {
        constexpr bool F32 = decltype(f32_c)::value, ADDC = decltype(addc_c)::value;
        const char* src = epi + rl * EPI_LD + c4l * 16;
        char* dst = obase + ((row0 + rl) * ldo + col0 + 4 * c4l) * (F32 ? 4 : 2);
        const int64_t step = (int64_t)RPI * ldo * (F32 ? 4 : 2);
        auto finish = [&](float4 v, int it) {
            v.x += bias4.x; v.y += bias4.y; v.z += bias4.z; v.w += bias4.w;
            char* d = dst + it * step;
            if constexpr (F32) {
                if constexpr (ADDC) {
                    const float4 c = *reinterpret_cast<const float4*>(d);
                    v.x = c.x + v.x; v.y = c.y + v.y; v.z = c.z + v.z; v.w = c.w + v.w;
                }
                *reinterpret_cast<float4*>(d) = v;
            } else {
                if constexpr (ADDC) {
                    const uint2 c = *reinterpret_cast<const uint2*>(d);
                    v.x = bf16lo(c.x) + v.x; v.y = bf16hi(c.x) + v.y;
                    v.z = bf16lo(c.y) + v.z; v.w = bf16hi(c.y) + v.w;
                }
                *reinterpret_cast<uint2*>(d) = make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
            }
        };
        if constexpr (Extra::kActive) {
            // groups of CH rows: staged values, extra terms, then bias and stores
            constexpr int CH = IT < 4 ? IT : 4;
            static_for<IT / CH>([&](auto g_c) {
                constexpr int g = decltype(g_c)::value;
                float4 ex[CH];
                static_for<CH>([&](auto k_c) {
                    ex[decltype(k_c)::value] =
                        *reinterpret_cast<const float4*>(src + (g * CH + decltype(k_c)::value) * RPI * EPI_LD);
                });
                extra.template slab<CH>(ex, (int)(row0 - m0) + rl + g * CH * RPI, (int)(col0 - n0) + 4 * c4l, RPI);
                static_for<CH>([&](auto k_c) { finish(ex[decltype(k_c)::value], g * CH + decltype(k_c)::value); });
            });
        } else {
            static_for<IT>([&](auto it_c) {
                constexpr int it = decltype(it_c)::value;
                finish(*reinterpret_cast<const float4*>(src + it * RPI * EPI_LD), it);
            });
        }
    };
    static_for<MI>([&](auto i) {
        static_for<NI>([&](auto j) {
            static_for<16>([&](auto v) {
                constexpr int vv = decltype(v)::value;
                const int r = 8 * (vv >> 2) + 4 * (lane >> 5) + (vv & 3);
                *reinterpret_cast<float*>(epi + r * EPI_LD + (j * 32 + (lane & 31)) * 4) = acc[i][j][vv];
            });
        });
        // The staging rows belong to this wave alone and one wave's LDS
        // accesses are performed in order, so no workgroup barrier is needed
        // here or after the stores below (a barrier's fence would also make
        // the wave wait for its global stores to reach memory, slab by slab).
        asm volatile("" : : : "memory");
        const int64_t row0 = m0 + wm * WTM + i * 32;
        if (cols_ok && row0 + 32 <= a.M) {
            using T_ = std::true_type;
            using F_ = std::false_type;
            if (out_f32) {
                if (add_c) slab_fast(row0, T_{}, T_{});
                else slab_fast(row0, T_{}, F_{});
            } else {
                if (add_c) slab_fast(row0, F_{}, T_{});
                else slab_fast(row0, F_{}, F_{});
            }
            asm volatile("" : : : "memory");
            return;
        }
        for (int q = lane; q < 32 * Q; q += 64) {
            const int r = q / Q, c4 = q - r * Q;
            const int64_t row = row0 + r, col = col0 + c4 * 4;
            if (row >= a.M || col >= a.N) continue;
            float4 v4 = *reinterpret_cast<const float4*>(epi + r * EPI_LD + c4 * 16);
            if constexpr (Extra::kActive) extra.one(v4, (int)(row0 - m0) + r, (int)(col0 - n0) + c4 * 4);
            float vals[4] = {v4.x, v4.y, v4.z, v4.w};
            const int nv = (int)((a.N - col) < 4 ? (a.N - col) : 4);
            if (!split_out && a.bias) {
                for (int e = 0; e < nv; ++e) vals[e] += a.bias[col + e];
            }
            const int64_t idx = row * ldo + col;
            if (split_out || a.c_type == kF32) {
                float* C = reinterpret_cast<float*>(obase);
                if (nv == 4 && vec_out) {
                    if (!split_out && a.accumulate) {
                        float4 c = *reinterpret_cast<const float4*>(C + idx);
                        vals[0] += c.x; vals[1] += c.y; vals[2] += c.z; vals[3] += c.w;
                    }
                    *reinterpret_cast<float4*>(C + idx) = make_float4(vals[0], vals[1], vals[2], vals[3]);
                } else {
                    for (int e = 0; e < nv; ++e) {
                        float val = vals[e];
                        if (!split_out && a.accumulate) val += C[idx + e];
                        C[idx + e] = val;
                    }
                }
            } else {
                uint16_t* C = reinterpret_cast<uint16_t*>(obase);
                if (nv == 4 && ((reinterpret_cast<uintptr_t>(C + idx) & 7) == 0)) {
                    if (a.accumulate) {
                        uint2 c = *reinterpret_cast<const uint2*>(C + idx);
                        vals[0] += bf16lo(c.x); vals[1] += bf16hi(c.x);
                        vals[2] += bf16lo(c.y); vals[3] += bf16hi(c.y);
                    }
                    *reinterpret_cast<uint2*>(C + idx) =
                        make_uint2(pack_bf16x2(vals[0], vals[1]), pack_bf16x2(vals[2], vals[3]));
                } else {
                    for (int e = 0; e < nv; ++e) {
                        float val = vals[e];
                        if (a.accumulate) val += bf16_to_f32(C[idx + e]);
                        C[idx + e] = (uint16_t)f32_to_bf16(val);
                    }
                }
            }
        }
        asm volatile("" : : : "memory");
    });
}


template <typename T, int BM, int BN, int WM, int WN, bool TA, bool TB, bool VEC>
__global__ __launch_bounds__(64 * WM * WN) void gemm_tile_kernel(GemmArgs a, TileMapArgs tmap) {
    gemm_batch_offset(a);
    constexpr int NT = 64 * WM * WN;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int MI = WTM / 32, NI = WTN / 32;
    constexpr int BK = 128 / (int)sizeof(T);
    constexpr int STAGE = (BM + BN) * 128;
    static_assert(MI >= 1 && NI >= 1, "wave tile must be a multiple of 32x32");
    __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];

    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int wm = wid / WN, wn = wid % WN;
    int tm, tn;
    map_tile(tmap, tm, tn);
    const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
    const int split = blockIdx.y;
    const int64_t kbeg = (int64_t)split * tmap.k_per_split;
    const int64_t kend = min(a.K, kbeg + tmap.k_per_split);
    const int nk = kend > kbeg ? (int)((kend - kbeg + BK - 1) / BK) : 0;

    const int64_t a_ext = TA ? ((a.K - 1) * a.lda + a.M) : ((a.M - 1) * a.lda + a.K);
    const int64_t b_ext = TB ? ((a.N - 1) * a.ldb + a.K) : ((a.K - 1) * a.ldb + a.N);
    const __amdgpu_buffer_rsrc_t rsA = make_rsrc(a.A, (uint32_t)(a_ext * (int64_t)sizeof(T)));
    const __amdgpu_buffer_rsrc_t rsB = make_rsrc(a.B, (uint32_t)(b_ext * (int64_t)sizeof(T)));

    TileLoader<T, BM, NT, !TA, VEC> la0;
    TileLoader<T, BN, NT, TB, VEC> lb0;

    f32x16_t acc[MI][NI];
    static_for<MI>([&](auto i) {
        static_for<NI>([&](auto j) {
            static_for<16>([&](auto v) { acc[i][j][decltype(v)::value] = 0.0f; });
        });
    });

    auto gload = [&](auto& la, auto& lb, int tile) {
        const int64_t k0 = kbeg + (int64_t)tile * BK;
        la.load(rsA, tid, m0, k0, a.M, kend, a.lda);
        lb.load(rsB, tid, n0, k0, a.N, kend, a.ldb);
    };
    auto lstore = [&](const auto& la, const auto& lb, int stage) {
        la.store(smem + stage * STAGE, tid);
        lb.store(smem + stage * STAGE + BM * 128, tid);
    };
    auto compute = [&](int stage) {
        const char* As = smem + stage * STAGE;
        const char* Bs = As + BM * 128;
        static_for<4>([&](auto ks) {
            uint4 af[MI], bfr[NI];
            const int ch = ks * 2 + (lane >> 5);
            static_for<MI>([&](auto i) {
                af[i] = *reinterpret_cast<const uint4*>(As + lds_off(wm * WTM + i * 32 + (lane & 31), ch));
            });
            static_for<NI>([&](auto j) {
                bfr[j] = *reinterpret_cast<const uint4*>(Bs + lds_off(wn * WTN + j * 32 + (lane & 31), ch));
            });
            static_for<MI>([&](auto i) {
                static_for<NI>([&](auto j) {
                    if constexpr (sizeof(T) == 2) mfma32_bf16(acc[i][j], af[i], bfr[j]);
                    else mfma32_f32x4(acc[i][j], af[i], bfr[j]);
                });
            });
        });
    };

    if (nk > 0) {
        gload(la0, lb0, 0);
        lstore(la0, lb0, 0);
        __syncthreads();
        for (int t = 0; t < nk; ++t) {
            const bool more = t + 1 < nk;
            if (more) gload(la0, lb0, t + 1);
            compute(t & 1);
            if (more) lstore(la0, lb0, (t + 1) & 1);
            __syncthreads();
        }
    }

    // Epilogue: the accumulators go to C (or the split-K partial sums)
    // through a per-wave LDS buffer, one 32-row slab at a time.
    static_assert(WM * WN * 32 * (WTN * 4 + 16) <= 2 * STAGE, "epilogue staging must fit in LDS");
    store_acc_tile<MI, NI, WTM, WTN, WM * WN>(a, acc, smem, m0, n0, wm, wn, wid, lane);
}

// Function table for one element type: [tile][trans_a][trans_b][vec].
typedef void (*GemmKernelFn)(GemmArgs, TileMapArgs);

template <typename T, int BM, int BN, int WM, int WN>
struct TileKernels {
    static GemmKernelFn get(int ta, int tb, int vec) {
        static const GemmKernelFn tbl[2][2][2] = {
            {{gemm_tile_kernel<T, BM, BN, WM, WN, false, false, false>,
              gemm_tile_kernel<T, BM, BN, WM, WN, false, false, true>},
             {gemm_tile_kernel<T, BM, BN, WM, WN, false, true, false>,
              gemm_tile_kernel<T, BM, BN, WM, WN, false, true, true>}},
            {{gemm_tile_kernel<T, BM, BN, WM, WN, true, false, false>,
              gemm_tile_kernel<T, BM, BN, WM, WN, true, false, true>},
             {gemm_tile_kernel<T, BM, BN, WM, WN, true, true, false>,
              gemm_tile_kernel<T, BM, BN, WM, WN, true, true, true>}}};
        return tbl[ta][tb][vec];
    }
};

template <typename T>
GemmKernelFn gemm_kernel_for(int tile, int ta, int tb, int vec) {
    switch (tile) {
        case kTile256x256: return TileKernels<T, 256, 256, 2, 2>::get(ta, tb, vec);
        case kTile256x128: return TileKernels<T, 256, 128, 2, 2>::get(ta, tb, vec);
        case kTile128x128: return TileKernels<T, 128, 128, 2, 2>::get(ta, tb, vec);
        case kTile128x64: return TileKernels<T, 128, 64, 2, 2>::get(ta, tb, vec);
        case kTile64x64: return TileKernels<T, 64, 64, 2, 2>::get(ta, tb, vec);
        case kTile128x32: return TileKernels<T, 128, 32, 4, 1>::get(ta, tb, vec);
        default: return nullptr;
    }
}

}  // namespace isam
