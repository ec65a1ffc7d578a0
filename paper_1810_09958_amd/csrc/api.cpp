// C-ABI layer: argument validation (pure host code, no HIP call), plan
// selection, and kernel dispatch.
//
// Plan selection is this library's counterpart of the paper's "Approach"
// interface (Section 4): every tiling, split and rasterisation choice is made
// in one place (the plan_* functions below) from the problem shape and the
// device's compute-unit count, and can be overridden for tuning with the
// environment variable ISAM_GEMM_CONFIG="tile=<0-5>,splits=<n>,group=<n>,xcd=<0|1>,dma=<0|1>"
// (and small=0, rows=0, skinny=0, stream=0|1 for the special-shape kernels, sk=0|1 for
// the stream-K schedule, fixup=0 for the two-slice sum, fixup=1 for its one-way form).
// ISAM_LOG=1 prints each chosen plan to stderr.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>

#include "../../include/isam.h"
#include "kernels.hpp"

using namespace isam;

namespace {

thread_local std::string g_last_error;

isam_status_t fail(isam_status_t st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    try {
        g_last_error = buf;
    } catch (...) {
    }
    return st;
}

isam_status_t hip_fail(hipError_t e, const char* what) {
    return fail(ISAM_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Read at every call (as the kernel-side log lines do), so a process can switch it.
bool log_enabled() {
    const char* v = getenv("ISAM_LOG");
    return v && v[0] && v[0] != '0';
}

bool valid_dtype(int t) { return t == ISAM_F32 || t == ISAM_BF16; }
size_t dsize(int t) { return t == ISAM_BF16 ? 2 : 4; }

constexpr int64_t kMaxExtent = (int64_t(1) << 31) - 1;

bool overlaps(const void* a, size_t an, const void* b, size_t bn) {
    if (!a || !b || an == 0 || bn == 0) return false;
    uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + bn && b0 < a0 + an;
}

// Compute units of the current device, cached.  Falls back to the MI355X
// count when no device is visible (host-only queries such as workspace sizes).
int device_cus() {
    static std::mutex mu;
    static int cache[64];
    static bool have[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
        (void)hipGetLastError();
        return 256;
    }
    std::unique_lock<std::mutex> lk(mu, std::defer_lock);
    try {
        lk.lock();
    } catch (...) {
        return 256;
    }
    if (!have[dev]) {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) {
            (void)hipGetLastError();
            cus = 256;
        }
        cache[dev] = cus;
        have[dev] = true;
    }
    return cache[dev];
}

// Largest LDS allocation of one workgroup on the current device, cached;
// 160 KiB (gfx950) when no device is visible.
int device_lds_max() {
    static std::mutex mu;
    static int cache[64];
    static bool have[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
        (void)hipGetLastError();
        return 160 * 1024;
    }
    std::unique_lock<std::mutex> lk(mu, std::defer_lock);
    try {
        lk.lock();
    } catch (...) {
        return 160 * 1024;
    }
    if (!have[dev]) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess || v <= 0) {
            (void)hipGetLastError();
            v = 160 * 1024;
        }
        cache[dev] = v;
        have[dev] = true;
    }
    return cache[dev];
}

// ---------------------------------------------------------------------------
// GEMM plan
// ---------------------------------------------------------------------------
int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

GemmPlan plan_gemm(int64_t M, int64_t N, int64_t K, int ab_type, int cus, bool allow_skinny = true) {
    GemmPlan p{};
    p.vec = 1;
    p.k_splits = 1;
    p.k_per_split = K;
    p.group_m = 8;
    p.xcd_remap = 1;
    p.dma = 1;
    p.dma_waves = 4;  // set to 8 below for 256x256 tiles (two waves per SIMD measured faster)
    int bm, bn, bk;
    auto tiles = [&](int t) {
        tile_dims(t, ab_type, &bm, &bn, &bk);
        return cdiv(M, bm) * cdiv(N, bn);
    };
    const bool skinny_off = getenv("ISAM_GEMM_CONFIG") && strstr(getenv("ISAM_GEMM_CONFIG"), "skinny=0");
    // N < 8 and not a multiple of the vector width: the dot-product kernel
    // (NN with aligned A rows, checked at dispatch; the tile kernel is the
    // fallback).
    if (allow_skinny && !skinny_off && N < 8 && K > 0 && N % (ab_type == kBF16 ? 8 : 4) != 0) {
        p.tile = kTile128x32;
        p.skinny = 4;
        return p;
    }
    // N <= 32 with A and B in NN layout streams A through the skinny kernel
    // (layout and alignment are checked at dispatch; the tile kernel is the
    // fallback).
    if (allow_skinny && N <= 32 && K > 0 && N % (ab_type == kBF16 ? 8 : 4) == 0 && !skinny_off) {
        p.tile = kTile128x32;
        const bool rows_off = getenv("ISAM_GEMM_CONFIG") && strstr(getenv("ISAM_GEMM_CONFIG"), "rows=0");
        if (!rows_off && cdiv(M, skinny_stream_rows()) >= cus / 2) {
            // Enough 16-row workgroups to cover the CUs: one pass over A, no split.
            p.skinny = 2;
            p.k_splits = 1;
            p.k_per_split = K;
            return p;
        }
        p.skinny = 1;
        p.k_per_split = skinny_k_slice(ab_type);
        p.k_splits = (int)cdiv(K, p.k_per_split);
        return p;
    }
    // Small products (few 32x32 output tiles, moderate K): one tile per
    // workgroup with the waves splitting K (A K-contiguous and aligned, batch 1:
    // checked at dispatch; the tile kernels are the fallback).
    const bool small_off = getenv("ISAM_GEMM_CONFIG") && strstr(getenv("ISAM_GEMM_CONFIG"), "small=0");
    if (allow_skinny && !small_off && gemm_small_fits(M, N, K)) {
        p.tile = kTile64x64;
        p.small = 1;
        return p;
    }
    // Tile choice (measured on MI355X): 256x256 tiles (8 waves) whenever they
    // fill the CUs; for deep K, 256x256 tiles split along K until they do
    // (the partial sums cost one extra pass over C); otherwise the largest
    // tile that fills the CUs, unsplit.
    const int64_t t256 = tiles(kTile256x256);
    if (N <= 32) {
        p.tile = kTile128x32;
    } else if (t256 >= cus && K <= 128 && tiles(kTile128x128) >= cus) {
        // Very shallow K (pointwise-convolution products): two K tiles do not
        // pay for the 256x256 prologue and epilogue (measured, bf16:
        // 100352x256x128 34.5 us against 38.4, 100352x128x64 18.8 against
        // 31.7, 8192x8192x128 equal).
        p.tile = kTile128x128;
    } else if (t256 >= cus) {
        p.tile = kTile256x256;
    } else if (K >= 4096 && ab_type == kBF16) {
        p.tile = kTile256x256;
        tile_dims(p.tile, ab_type, &bm, &bn, &bk);
        const int64_t want = std::min<int64_t>(8, cdiv(cus, t256));
        const int64_t sp = std::max<int64_t>(1, std::min<int64_t>(want, K / (8 * bk)));
        if (sp > 1) {
            p.k_per_split = cdiv(cdiv(K, sp), bk) * bk;
            p.k_splits = (int)cdiv(K, p.k_per_split);
        }

    } else if (ab_type == kBF16 && K > 2048 && t256 * 2 >= cus) {
        // Deep K with 256x256 tiles for at least half the CUs: one partial
        // round of the large tiles beats two rounds of smaller ones
        // (measured, bf16: 3000^3 80 us against 104 for 256x128 tiles,
        // 3072x3072x2560 62 against 83, 3584x3584x3000 82 against 109).
        p.tile = kTile256x256;
    } else if (K <= 2048 && tiles(kTile128x128) >= cus) {
        // Shallow K: the 128x128 grid (measured, bf16 NT, K = 1024: 2048x3072
        // 24 us against 27 for 128x64; 4096x3072 39 us against 55 for 256x128,
        // whose 384 tiles leave half the CUs idle in the second round).
        p.tile = kTile128x128;
    } else if (tiles(kTile256x128) >= cus) {
        p.tile = kTile256x128;
    } else if (tiles(kTile128x128) >= cus) {
        p.tile = kTile128x128;
    } else if (tiles(kTile128x64) >= cus) {
        p.tile = kTile128x64;
    } else {
        p.tile = kTile64x64;
    }
    tile_dims(p.tile, ab_type, &bm, &bn, &bk);
    if (p.tile == kTile256x256) p.dma_waves = 8;
    const int64_t nt = tiles(p.tile);
    // Other tiles with a grid smaller than the CU count and deep K: split K
    // so the grid covers the CUs.
    if (p.k_splits == 1 && p.tile != kTile256x256 && nt < cus && K >= 8 * bk) {
        const int64_t want = cdiv(cus, nt);
        const int64_t sp = std::max<int64_t>(1, std::min<int64_t>(want, std::min<int64_t>(K / (4 * bk), 16)));
        if (sp > 1) {
            p.k_per_split = cdiv(cdiv(K, sp), bk) * bk;
            p.k_splits = (int)cdiv(K, p.k_per_split);
        }
    }
    if (p.k_splits <= 1) {
        p.k_splits = 1;
        p.k_per_split = K;
    }
    // Tuning override.
    if (const char* env = getenv("ISAM_GEMM_CONFIG")) {
        int v;
        const char* s;
        if ((s = strstr(env, "tile=")) && sscanf(s + 5, "%d", &v) == 1 && v >= 0 && v < kTileCount) p.tile = v;
        if ((s = strstr(env, "group=")) && sscanf(s + 6, "%d", &v) == 1 && v > 0) p.group_m = v;
        if ((s = strstr(env, "xcd=")) && sscanf(s + 4, "%d", &v) == 1) p.xcd_remap = v ? 1 : 0;
        if ((s = strstr(env, "dma=")) && sscanf(s + 4, "%d", &v) == 1) p.dma = v ? 1 : 0;
        if ((s = strstr(env, "dmaw=")) && sscanf(s + 5, "%d", &v) == 1) p.dma_waves = v == 8 ? 8 : 4;
        if ((s = strstr(env, "splits=")) && sscanf(s + 7, "%d", &v) == 1 && v >= 1) {
            tile_dims(p.tile, ab_type, &bm, &bn, &bk);
            p.k_per_split = std::max<int64_t>(bk, cdiv(cdiv(K, v), bk) * bk);
            p.k_splits = (int)std::max<int64_t>(1, cdiv(K, p.k_per_split));
            if (p.k_splits == 1) p.k_per_split = K;
        }
    }
    // Two K slices of 256x256 tiles whose workgroups t and t + tiles land on
    // one XCD (workgroups are dealt to the XCDs in turn, 32 CUs each): the
    // second slice sums the pair through that XCD's L2, with no reduction
    // pass.  ISAM_GEMM_CONFIG fixup=0 keeps the pass.
    // When the whole grid (both slices of every tile) fits on the CUs at once,
    // the slices split the finishing work instead: each publishes the half
    // tile the other finishes and waits for the other's half (fixup = 2;
    // 8192x1024x16384 bf16: 128 tiles, 256 workgroups).
    const int xcds = cus % 32 == 0 ? cus / 32 : 1;
    if (p.k_splits == 2 && p.tile == kTile256x256 && tiles(kTile256x256) % xcds == 0)
        p.fixup = 2 * tiles(kTile256x256) <= cus ? 2 : 1;
    if (const char* env = getenv("ISAM_GEMM_CONFIG")) {
        if (strstr(env, "fixup=0")) p.fixup = 0;
        if (strstr(env, "fixup=1") && p.fixup) p.fixup = 1;
    }
    // Stream-K (bf16, the three-stage-ring tiles, no K split): a persistent
    // grid; each XCD's range of tiles runs its whole rounds one tile per
    // workgroup, then deals the remaining tiles' (tile, K tile) units to its
    // workgroups in equal shares.  Taken by itself for 256x256 tiles when at
    // least one whole round exists and the last, partial round would keep at
    // most a quarter of the CUs busy, in one of two forms (measured, bf16,
    // plain grid / stream-K / hipBLASLt, µs):
    //   * shares of at least 8 K tiles: the whole rounds run first
    //     (4352x4352x4096 178 / 161 / 163, 6144x6144x4096 290 / 261 / 265,
    //     8192x4608x2048 154-176 / 153-161 / 151);
    //   * a remainder of at most an eighth of a round: it joins the last whole
    //     round (sk_keep = 1), every share 1-1.125 tiles (4352x4096x3008 133 /
    //     111 / 122, 4352x4096x1024 55 / 51 / 55; cut into one-unit shares
    //     instead, 4352x4096x1024 took 95 µs exchanging partial sums).
    // Otherwise the plain grid: with shares of a fraction of a tile, or of
    // 1.2 tiles, the workgroups of an XCD walk K at different offsets and lose
    // L2 reuse (4608x4352x2048: 97-104 against 103-108; 5000^3, half a round
    // left: 247-272 against 265-278).  ISAM_GEMM_CONFIG sk=0 / sk=1 switch it
    // off / force it (forced, the form follows the same rule; with fewer tiles
    // than workgroups every tile is shared).
    if (ab_type == kBF16 && p.k_splits == 1 && gemm_sk_tile(p.tile) && K > 0) {
        const int G = gemm_sk_grid(p.tile, cus);
        const int parts = G % 8 == 0 ? 8 : 1, gx = G / parts;
        const int64_t nt = tiles(p.tile), nkt = cdiv(K, 64);
        const int64_t tx = nt / parts, full = tx / gx, rem = tx - full * gx;
        const bool fits = nt * nkt < (int64_t(1) << 31);
        const bool long_shares = rem * nkt >= 8 * (int64_t)gx, small_rem = rem * 8 <= gx;
        const char* env = getenv("ISAM_GEMM_CONFIG");
        const bool off = env && strstr(env, "sk=0"), force = env && strstr(env, "sk=1");
        const bool pays = p.tile == kTile256x256 && full >= 1 && rem > 0 && rem * 4 <= gx && (long_shares || small_rem);
        if (fits && !off && (force || pays)) {
            p.sk = 1;
            p.sk_grid = G;
            p.sk_keep = (full >= 1 && !long_shares) ? 1 : 0;
        }
    }
    return p;
}

size_t gemm_ws_bytes(const GemmPlan& p, int64_t M, int64_t N) {
    if (p.sk) return gemm_sk_ws_bytes(p.tile, p.sk_grid);
    if (p.k_splits <= 1) return 0;
    // room for the reduction pass's partials, and (two-slice plans that may
    // sum inside the kernel) for the per-tile partials and flags
    const size_t red = (size_t)p.k_splits * (size_t)M * (size_t)N * sizeof(float);
    return p.fixup ? std::max(red, gemm_fixup_ws_bytes(M, N)) : red;
}

bool vec_ok(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K, int ab_type, const void* A,
            int64_t lda, const void* B, int64_t ldb) {
    const int64_t E = ab_type == ISAM_BF16 ? 8 : 4;
    const int64_t es = (int64_t)dsize(ab_type);
    if (((uintptr_t)A & 15) || ((uintptr_t)B & 15)) return false;
    if ((lda * es) % 16 || (ldb * es) % 16) return false;
    if ((trans_a ? M : K) % E) return false;
    if ((trans_b ? K : N) % E) return false;
    return true;
}

// Operands whose rows cannot be fetched in 16-byte pieces are copied into the
// workspace first (pack.hip), so that the product runs on the MFMA kernels that
// copy 16 bytes at a time instead of the element-wise tile kernel (bf16
// 8192x8192x8100: 13.8 ms there).  A packed A is [M][Kp] (K-contiguous, also
// when it was given transposed); a packed B keeps its layout when its rows can
// be padded ([N][Kp], or [Kp][N] with N a multiple of the vector width) and is
// transposed to [N][Kp] otherwise.  Kp is K rounded up to the vector width (to
// a multiple of 64 when both operands are copied and that adds at most 1/16);
// the padded K positions are zero in both operands.  bf16 A given as [K][M] is
// copied too, transposed, for the direct-to-LDS kernels.  Only products that the
// planner would give large tiles are packed (the copies cost about as much as
// reading and writing both operands once).
struct PackPlan {
    bool pays = false;
    bool a = false, b = false;        // operand copied
    bool a_tr = false, b_tr = false;  // copied with a transpose
    int trans_a = 0, trans_b = 0;     // layouts of the product that follows
    int64_t Kp = 0;
    int64_t b_rows = 0, b_cols = 0;   // packed B
    size_t a_bytes = 0, b_bytes = 0;  // each a multiple of 256
};

PackPlan pack_plan(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K, int ab_type, bool a_mis, bool b_mis) {
    PackPlan k;
    const int64_t E = ab_type == ISAM_BF16 ? 8 : 4, es = (int64_t)dsize(ab_type);
    auto al = [](int64_t v) { return (size_t)((v + 255) & ~(int64_t)255); };
    k.Kp = cdiv(K, E) * E;
    k.a = a_mis || k.Kp != K;
    k.b = b_mis || k.Kp != K;
    // Both copied: pad K to whole 64-deep tiles when that adds at most 1/16
    // (the kernels' whole-tile instance takes no per-copy range checks).
    if (k.a && k.b && (cdiv(K, 64) * 64 - K) * 16 <= K) k.Kp = cdiv(K, 64) * 64;
    k.trans_a = trans_a;
    k.trans_b = trans_b;
    if (k.a) {
        k.a_tr = trans_a != 0;
        k.trans_a = 0;
        k.a_bytes = al(M * k.Kp * es);
    }
    if (k.b) {
        if (trans_b || N % E == 0) {
            k.b_rows = trans_b ? N : k.Kp;
            k.b_cols = trans_b ? k.Kp : N;
        } else {
            k.b_tr = true;
            k.trans_b = 1;
            k.b_rows = N;
            k.b_cols = k.Kp;
        }
        k.b_bytes = al(k.b_rows * k.b_cols * es);
    }
    const GemmPlan q = plan_gemm(M, N, k.Kp, ab_type, device_cus());
    const bool big = !q.small && !q.skinny && q.tile != kTile64x64 && q.tile != kTile128x32;
    const bool fits = (int64_t)k.a_bytes <= kMaxExtent && (int64_t)k.b_bytes <= kMaxExtent;
    const char* env = getenv("ISAM_GEMM_CONFIG");
    k.pays = (k.a || k.b) && big && fits && !(env && strstr(env, "pack=0"));
    return k;
}

// Large fp32 products run on the bf16 matrix cores: each operand value is
// split into three bf16 terms (pack.hip) laid out as six K blocks, A as
// (h, h, m, h, l, m) and B as (h, m, h, l, h, m), so that one bf16 product over
// K' = 6 Kp forms hh + hm + mh + hl + lh + mm -- the fp32 product to within
// the dropped terms' 2^-23 relative size, accumulated in fp32.  Six bf16
// products cost less than a quarter of one fp32 product on the matrix cores
// (fp32 8192^3: 8.47 ms on the fp32 tile kernel).  Needs A [M][K] (no
// transpose), B [N][K] or [K][N] with N a multiple of 8, and workspace for
// the split copies (12 bytes per operand value); only products where the
// copies cost well under the time saved (M N >= 512 (M + N), large tiles).
constexpr uint32_t kSplitPatA = 0u | 0u << 2 | 1u << 4 | 0u << 6 | 2u << 8 | 1u << 10;
constexpr uint32_t kSplitPatB = 0u | 1u << 2 | 0u << 4 | 2u << 6 | 0u << 8 | 1u << 10;

struct SplitPlan {
    bool pays = false;
    int64_t Kp = 0;                   // K of each block
    size_t a_bytes = 0, b_bytes = 0;  // each a multiple of 256
};

SplitPlan split_plan(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K) {
    SplitPlan k;
    if (trans_a || (!trans_b && N % 8) || K <= 0) return k;
    auto al = [](int64_t v) { return (size_t)((v + 255) & ~(int64_t)255); };
    k.Kp = cdiv(K, 8) * 8;
    if ((cdiv(K, 64) * 64 - K) * 16 <= K) k.Kp = cdiv(K, 64) * 64;
    k.a_bytes = al(M * 6 * k.Kp * 2);
    k.b_bytes = al(N * 6 * k.Kp * 2);
    const GemmPlan q = plan_gemm(M, N, 6 * k.Kp, kBF16, device_cus());
    const bool big = !q.small && !q.skinny && q.tile != kTile64x64 && q.tile != kTile128x32 && q.tile != kTile128x64;
    const bool fits = (int64_t)k.a_bytes <= kMaxExtent && (int64_t)k.b_bytes <= kMaxExtent;
    const char* env = getenv("ISAM_GEMM_CONFIG");
    k.pays = big && fits && M * N >= 512 * (M + N) && !(env && strstr(env, "f32split=0"));
    return k;
}

bool pack_a_needed(int trans_a, int64_t M, int64_t K, int ab_type, const void* A, int64_t lda) {
    const int64_t E = ab_type == ISAM_BF16 ? 8 : 4, es = (int64_t)dsize(ab_type);
    return ((uintptr_t)A & 15) || (lda * es) % 16 || (trans_a ? M : K) % E;
}

bool pack_b_needed(int trans_b, int64_t N, int64_t K, int ab_type, const void* B, int64_t ldb) {
    const int64_t E = ab_type == ISAM_BF16 ? 8 : 4, es = (int64_t)dsize(ab_type);
    return ((uintptr_t)B & 15) || (ldb * es) % 16 || (trans_b ? K : N) % E;
}

isam_status_t validate_gemm(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K, int ab_type,
                            const void* A, int64_t lda, const void* B, int64_t ldb, int accumulate,
                            int c_type, const void* C, int64_t ldc, const char* who) {
    if ((trans_a != 0 && trans_a != 1) || (trans_b != 0 && trans_b != 1))
        return fail(ISAM_ERR_INVALID_ARG, "%s: trans_a/trans_b must be 0 or 1", who);
    if (accumulate != 0 && accumulate != 1)
        return fail(ISAM_ERR_INVALID_ARG, "%s: accumulate must be 0 or 1", who);
    if (M < 0 || N < 0 || K < 0)
        return fail(ISAM_ERR_INVALID_ARG, "%s: negative size M=%lld N=%lld K=%lld", who, (long long)M,
                    (long long)N, (long long)K);
    if (!valid_dtype(ab_type) || !valid_dtype(c_type))
        return fail(ISAM_ERR_INVALID_ARG, "%s: dtype must be ISAM_F32 (0) or ISAM_BF16 (1)", who);
    if (M == 0 || N == 0) return ISAM_OK;
    if (!C) return fail(ISAM_ERR_INVALID_ARG, "%s: C is NULL", who);
    if (ldc < N) return fail(ISAM_ERR_INVALID_ARG, "%s: ldc=%lld < N=%lld", who, (long long)ldc, (long long)N);
    const int64_t c_ext = (M - 1) * ldc + N;
    if (c_ext * (int64_t)dsize(c_type) > kMaxExtent)
        return fail(ISAM_ERR_UNSUPPORTED, "%s: C spans more than 2^31 bytes", who);
    if (K == 0) return ISAM_OK;
    if (!A || !B) return fail(ISAM_ERR_INVALID_ARG, "%s: A or B is NULL", who);
    const int64_t need_lda = trans_a ? M : K, need_ldb = trans_b ? K : N;
    if (lda < need_lda)
        return fail(ISAM_ERR_INVALID_ARG, "%s: lda=%lld < %lld", who, (long long)lda, (long long)need_lda);
    if (ldb < need_ldb)
        return fail(ISAM_ERR_INVALID_ARG, "%s: ldb=%lld < %lld", who, (long long)ldb, (long long)need_ldb);
    const int64_t es = (int64_t)dsize(ab_type);
    const int64_t a_ext = trans_a ? (K - 1) * lda + M : (M - 1) * lda + K;
    const int64_t b_ext = trans_b ? (N - 1) * ldb + K : (K - 1) * ldb + N;
    if (a_ext * es > kMaxExtent || b_ext * es > kMaxExtent)
        return fail(ISAM_ERR_UNSUPPORTED, "%s: an operand spans more than 2^31 bytes", who);
    const size_t cb = (size_t)c_ext * dsize(c_type);
    if (overlaps(C, cb, A, (size_t)(a_ext * es)) || overlaps(C, cb, B, (size_t)(b_ext * es)))
        return fail(ISAM_ERR_INVALID_ARG, "%s: C overlaps A or B", who);
    return ISAM_OK;
}

isam_status_t run_gemm(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K, int ab_type,
                       const void* A, int64_t lda, const void* B, int64_t ldb, int accumulate,
                       int c_type, void* C, int64_t ldc, const float* bias, void* workspace,
                       size_t workspace_bytes, hipStream_t stream, const char* who, int64_t batch = 1,
                       int64_t stride_a = 0, int64_t stride_b = 0, int64_t stride_c = 0) {
    // A strided batch is planned as one product of batch*M rows (for the tile
    // choice) and never split along K.
    GemmPlan p = batch > 1 ? plan_gemm(M * batch, N, K, ab_type, device_cus(), /*allow_skinny=*/false)
                           : plan_gemm(M, N, K, ab_type, device_cus());
    if (batch > 1) {
        p.k_splits = 1;
        p.k_per_split = K;
        p.sk = 0;
    }
    p.vec = (K == 0) ? 1 : (vec_ok(trans_a, trans_b, M, N, K, ab_type, A, lda, B, ldb) ? 1 : 0);
    if (ab_type == kF32 && batch == 1 && K > 0) {
        const SplitPlan k = split_plan(trans_a, trans_b, M, N, K);
        char* ws = static_cast<char*>(workspace);
        const size_t split_bytes = k.a_bytes + k.b_bytes;
        if (k.pays && ws && ((uintptr_t)ws & 255) == 0 && workspace_bytes >= split_bytes) {
            const int64_t es = (int64_t)dsize(ab_type);
            const size_t a_b = (size_t)(((M - 1) * lda + K) * es);
            const size_t b_b = (size_t)((trans_b ? (N - 1) * ldb + K : (K - 1) * ldb + N) * es);
            const size_t c_b = (size_t)((M - 1) * ldc + N) * dsize(c_type);
            if (overlaps(ws, split_bytes, A, a_b) || overlaps(ws, split_bytes, B, b_b) ||
                overlaps(ws, split_bytes, C, c_b))
                return fail(ISAM_ERR_INVALID_ARG, "%s: workspace overlaps A, B or C", who);
            if (log_enabled())
                fprintf(stderr, "[isam] %s fp32 split into bf16 terms: K %lld -> 6 x %lld\n", who, (long long)K,
                        (long long)k.Kp);
            const int cus = device_cus();
            uint16_t* As = reinterpret_cast<uint16_t*>(ws);
            uint16_t* Bs = reinterpret_cast<uint16_t*>(ws + k.a_bytes);
            const float* Af = static_cast<const float*>(A);
            const float* Bf = static_cast<const float*>(B);
            hipError_t e = launch_split6(Af, M, K, lda, As, M, k.Kp, k.Kp, false, kSplitPatA, cus, stream);
            if (e == hipSuccess)
                e = trans_b ? launch_split6(Bf, N, K, ldb, Bs, N, k.Kp, k.Kp, false, kSplitPatB, cus, stream)
                            : launch_split6(Bf, K, N, ldb, Bs, k.Kp, N, k.Kp, true, kSplitPatB, cus, stream);
            if (e != hipSuccess) return hip_fail(e, who);
            return run_gemm(0, trans_b, M, N, 6 * k.Kp, kBF16, As, 6 * k.Kp, Bs, trans_b ? 6 * k.Kp : N, accumulate,
                            c_type, C, ldc, bias, ws + split_bytes, workspace_bytes - split_bytes, stream, who);
        }
    }
    // bf16 A given as [K][M] is also copied (transposed): the direct-to-LDS
    // kernels need A K-contiguous (4096^3 with A transposed: 197 us on the
    // vector tile kernel, 141 us with the copy).
    if ((!p.vec || (trans_a && ab_type == kBF16)) && batch == 1 && K > 0) {
        const PackPlan k = pack_plan(trans_a, trans_b, M, N, K, ab_type,
                                     (trans_a && ab_type == kBF16) || pack_a_needed(trans_a, M, K, ab_type, A, lda),
                                     pack_b_needed(trans_b, N, K, ab_type, B, ldb));
        const size_t pack_bytes = k.a_bytes + k.b_bytes;
        char* ws = static_cast<char*>(workspace);
        if (k.pays && ws && ((uintptr_t)ws & 255) == 0 && workspace_bytes >= pack_bytes) {
            const int64_t es = (int64_t)dsize(ab_type);
            const void* Ap = k.a ? ws : A;
            const void* Bp = k.b ? ws + k.a_bytes : B;
            const int64_t ldap = k.a ? k.Kp : lda, ldbp = k.b ? k.b_cols : ldb;
            if (vec_ok(k.trans_a, k.trans_b, M, N, k.Kp, ab_type, Ap, ldap, Bp, ldbp)) {
                const size_t a_b = (size_t)((trans_a ? (K - 1) * lda + M : (M - 1) * lda + K) * es);
                const size_t b_b = (size_t)((trans_b ? (N - 1) * ldb + K : (K - 1) * ldb + N) * es);
                const size_t c_b = (size_t)((M - 1) * ldc + N) * dsize(c_type);
                if (overlaps(ws, pack_bytes, A, a_b) || overlaps(ws, pack_bytes, B, b_b) ||
                    overlaps(ws, pack_bytes, C, c_b))
                    return fail(ISAM_ERR_INVALID_ARG, "%s: workspace overlaps A, B or C", who);
                if (log_enabled())
                    fprintf(stderr, "[isam] %s packed operands: A %d%s, B %d%s, K %lld -> %lld\n", who, (int)k.a,
                            k.a_tr ? " (transposed)" : "", (int)k.b, k.b_tr ? " (transposed)" : "", (long long)K,
                            (long long)k.Kp);
                const int cus = device_cus();
                hipError_t e = hipSuccess;
                if (k.a)
                    e = k.a_tr ? launch_pack(A, K, M, lda, ws, M, k.Kp, (int)es, true, cus, stream)
                               : launch_pack(A, M, K, lda, ws, M, k.Kp, (int)es, false, cus, stream);
                if (e == hipSuccess && k.b)
                    e = trans_b || !k.b_tr ? launch_pack(B, trans_b ? N : K, trans_b ? K : N, ldb, ws + k.a_bytes,
                                                         k.b_rows, k.b_cols, (int)es, false, cus, stream)
                                           : launch_pack(B, K, N, ldb, ws + k.a_bytes, k.b_rows, k.b_cols, (int)es,
                                                         true, cus, stream);
                if (e != hipSuccess) return hip_fail(e, who);
                return run_gemm(k.trans_a, k.trans_b, M, N, k.Kp, ab_type, Ap, ldap, Bp, ldbp, accumulate, c_type, C,
                                ldc, bias, ws + pack_bytes, workspace_bytes - pack_bytes, stream, who);
            }
        }
    }
    if (p.skinny == 4) {
        // the narrow kernel reads A in 16-byte pieces and B element-wise
        const int64_t es = (int64_t)dsize(ab_type);
        if (trans_a || trans_b || K == 0 || ((uintptr_t)A & 15) || (lda * es) % 16) {
            p = plan_gemm(M, N, K, ab_type, device_cus(), /*allow_skinny=*/false);
            p.vec = (K == 0) ? 1 : (vec_ok(trans_a, trans_b, M, N, K, ab_type, A, lda, B, ldb) ? 1 : 0);
        }
    } else if (p.small && (!p.vec || trans_a || K == 0)) {
        p = plan_gemm(M, N, K, ab_type, device_cus(), /*allow_skinny=*/false);
        p.vec = (K == 0) ? 1 : (vec_ok(trans_a, trans_b, M, N, K, ab_type, A, lda, B, ldb) ? 1 : 0);
    } else if (p.skinny && (!p.vec || trans_a || trans_b || K == 0)) {
        p = plan_gemm(M, N, K, ab_type, device_cus(), /*allow_skinny=*/false);
        p.vec = (K == 0) ? 1 : (vec_ok(trans_a, trans_b, M, N, K, ab_type, A, lda, B, ldb) ? 1 : 0);
    }
    // Stream-K needs the direct-to-LDS kernel (bf16, A K-contiguous, aligned rows) and its
    // workspace; otherwise the same tiles run one per workgroup.
    if (p.sk && (trans_a || !p.vec || !workspace || workspace_bytes < gemm_ws_bytes(p, M, N))) p.sk = 0;
    if (p.k_splits > 1 && (!workspace || workspace_bytes < gemm_ws_bytes(p, M, N))) {
        if (p.skinny) p = plan_gemm(M, N, K, ab_type, device_cus(), /*allow_skinny=*/false);
        p.k_splits = 1;
        p.k_per_split = K;
        p.vec = (K == 0) ? 1 : (vec_ok(trans_a, trans_b, M, N, K, ab_type, A, lda, B, ldb) ? 1 : 0);
    }
    if (p.k_splits > 1 || p.sk) {
        // The split-K partial sums must not land on an operand.
        const int64_t es = (int64_t)dsize(ab_type);
        const size_t a_b = (size_t)((trans_a ? (K - 1) * lda + M : (M - 1) * lda + K) * es);
        const size_t b_b = (size_t)((trans_b ? (N - 1) * ldb + K : (K - 1) * ldb + N) * es);
        const size_t c_b = (size_t)((M - 1) * ldc + N) * dsize(c_type);
        const size_t w_b = gemm_ws_bytes(p, M, N);
        if (overlaps(workspace, w_b, A, a_b) || overlaps(workspace, w_b, B, b_b) || overlaps(workspace, w_b, C, c_b))
            return fail(ISAM_ERR_INVALID_ARG, "%s: workspace overlaps A, B or C", who);
    }
    if (!p.vec) {
        // The element-wise loader is instantiated for the small tiles only.
        if (p.tile != kTile64x64 && p.tile != kTile128x32) p.tile = kTile64x64;
    }
    if (log_enabled())
        fprintf(stderr, "[isam] %s M=%lld N=%lld K=%lld ta=%d tb=%d ab=%d c=%d tile=%d vec=%d splits=%d kps=%lld group=%d xcd=%d dma=%d skinny=%d small=%d sk=%d\n",
                who, (long long)M, (long long)N, (long long)K, trans_a, trans_b, ab_type, c_type, p.tile, p.vec,
                p.k_splits, (long long)p.k_per_split, p.group_m, p.xcd_remap, p.dma, p.skinny, p.small, p.sk);
    GemmArgs a{};
    a.A = A;
    a.B = B;
    a.C = C;
    a.partial = static_cast<float*>(workspace);
    a.bias = bias;
    a.M = M;
    a.N = N;
    a.K = K;
    a.lda = lda;
    a.ldb = ldb;
    a.ldc = ldc;
    a.trans_a = trans_a;
    a.trans_b = trans_b;
    a.ab_type = ab_type;
    a.c_type = c_type;
    a.accumulate = accumulate;
    a.batch = batch;
    a.stride_a = stride_a;
    a.stride_b = stride_b;
    a.stride_c = stride_c;
    // Very shallow bf16 products with at least one 32-row tile per CU take the
    // streaming kernel (B in registers, A streamed once through LDS by producer
    // waves; measured, bf16 out: 100352x256x128 24.8 us against 35.2 for the
    // 128x128 tiles, 100352x128x64 14.6 against 19.0, 200704x64x32 19.4
    // against 30.9, 8192x256x128 7.5 against 8.3); ISAM_GEMM_CONFIG stream=0 /
    // stream=1 switch it off / force it where it fits.
    {
        const char* env = getenv("ISAM_GEMM_CONFIG");
        const bool off = env && strstr(env, "stream=0"), force = env && strstr(env, "stream=1");
        if (!off && batch == 1 && !p.skinny && !p.small && gemm_stream_fits(a) &&
            (force || (K <= kStreamMaxK && cdiv(M, 32) >= (int64_t)device_cus()))) {
            if (log_enabled()) fprintf(stderr, "[isam] %s streaming kernel\n", who);
            hipError_t e = launch_gemm_stream(a, device_cus(), stream);
            if (e != hipSuccess) return hip_fail(e, who);
            return ISAM_OK;
        }
    }
    hipError_t e = launch_gemm(a, p, stream);
    if (e != hipSuccess) return hip_fail(e, who);
    return ISAM_OK;
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

}  // namespace

// ---------------------------------------------------------------------------
// Exported entry points
// ---------------------------------------------------------------------------
extern "C" {

isam_status_t isam_gemm(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K, int ab_type,
                        const void* A, int64_t lda, const void* B, int64_t ldb, int accumulate,
                        int c_type, void* C, int64_t ldc, void* workspace, size_t workspace_bytes,
                        void* stream) {
    g_last_error.clear();
    isam_status_t st = validate_gemm(trans_a, trans_b, M, N, K, ab_type, A, lda, B, ldb, accumulate,
                                     c_type, C, ldc, "isam_gemm");
    if (st != ISAM_OK || M == 0 || N == 0) return st;
    return run_gemm(trans_a, trans_b, M, N, K, ab_type, A, lda, B, ldb, accumulate, c_type, C, ldc,
                    nullptr, workspace, workspace_bytes, static_cast<hipStream_t>(stream), "isam_gemm");
}

size_t isam_gemm_workspace_size(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                                int ab_type, int c_type) {
    (void)c_type;
    if (M <= 0 || N <= 0 || K <= 0 || !valid_dtype(ab_type)) return 0;
    if ((trans_a != 0 && trans_a != 1) || (trans_b != 0 && trans_b != 1)) return 0;
    size_t ws = gemm_ws_bytes(plan_gemm(M, N, K, ab_type, device_cus()), M, N);
    // Rows that the sizes alone make unfit for 16-byte copies (a contiguous
    // dimension off the vector width), and bf16 A given as [K][M]: room to pack
    // them, and what the packed product then uses.
    if (ab_type == ISAM_F32) {
        const SplitPlan k = split_plan(trans_a, trans_b, M, N, K);
        if (k.pays)
            return std::max(ws, k.a_bytes + k.b_bytes +
                                    gemm_ws_bytes(plan_gemm(M, N, 6 * k.Kp, kBF16, device_cus()), M, N));
    }
    const int64_t E = ab_type == ISAM_BF16 ? 8 : 4;
    const bool a_mis = (trans_a ? M : K) % E != 0 || (trans_a && ab_type == ISAM_BF16),
               b_mis = (trans_b ? K : N) % E != 0;
    if (a_mis || b_mis) {
        const PackPlan k = pack_plan(trans_a, trans_b, M, N, K, ab_type, a_mis, b_mis);
        if (k.pays)
            ws = std::max(ws, k.a_bytes + k.b_bytes + gemm_ws_bytes(plan_gemm(M, N, k.Kp, ab_type, device_cus()), M, N));
    }
    return ws;
}

static bool dw_out_dims(int64_t H, int64_t W, int64_t kh, int64_t kw, int64_t stride, int64_t pad,
                        int64_t* Ho, int64_t* Wo) {
    if (stride <= 0) return false;
    *Ho = (H + 2 * pad - kh) / stride + 1;
    *Wo = (W + 2 * pad - kw) / stride + 1;
    return H + 2 * pad >= kh && W + 2 * pad >= kw && *Ho > 0 && *Wo > 0;
}

static size_t dwsep_ws(int64_t batch, int64_t Ho, int64_t Wo, int64_t C_in, int64_t cm,
                       int64_t C_out, int in_type) {
    const int64_t M = batch * Ho * Wo, K = C_in * cm;
    const size_t y = align256((size_t)M * (size_t)K * dsize(in_type));
    const GemmPlan p = plan_gemm(M, C_out, K, in_type, device_cus());
    return y + gemm_ws_bytes(p, M, C_out);
}

// Which separable-convolution path runs: 1 = fused bf16 kernel, 2 = fused
// fp32 kernel (both keep the depthwise result on chip and need no
// workspace), 0 = depthwise kernel into the workspace, then the pointwise
// GEMM.  The fused kernels need 16-byte aligned x, dw_filter, pw_weight and
// y; ISAM_DWSEP_FUSED=0 turns them off.
static int dwsep_path(const DwArgs& d, int64_t C_out, int out_type, const void* pw, const void* y) {
    const char* env = getenv("ISAM_DWSEP_FUSED");
    if (env && env[0] == '0') return 0;
    if (((uintptr_t)y & 15) || ((uintptr_t)pw & 15)) return 0;
    const int lds_max = device_lds_max();
    if (dwsep_fused_rows(d, C_out, lds_max) > 0) return 1;
    if (out_type == ISAM_F32 && dwsep_fused_f32_ok(d, C_out, lds_max)) return 2;
    return 0;
}

static DwArgs dw_args(int64_t batch, int64_t H, int64_t W, int64_t C_in, int64_t depth_mult, int64_t kh,
                      int64_t kw, int64_t stride, int64_t pad, int64_t Ho, int64_t Wo, int in_type,
                      const void* x, const void* dw_filter, void* Y) {
    DwArgs d{};
    d.x = x;
    d.w = dw_filter;
    d.y = Y;
    d.batch = batch;
    d.H = H;
    d.W = W;
    d.C = C_in;
    d.cm = depth_mult;
    d.kh = kh;
    d.kw = kw;
    d.stride = stride;
    d.pad = pad;
    d.Ho = Ho;
    d.Wo = Wo;
    d.in_type = in_type;
    d.y_type = in_type;
    return d;
}

size_t isam_dwsep_conv_workspace_size(int64_t batch, int64_t H, int64_t W, int64_t C_in,
                                      int64_t depth_mult, int64_t kh, int64_t kw, int64_t stride,
                                      int64_t pad, int64_t C_out, int in_type, int out_type) {
    int64_t Ho, Wo;
    if (batch <= 0 || C_in <= 0 || depth_mult <= 0 || C_out <= 0 || kh <= 0 || kw <= 0 || pad < 0 ||
        !valid_dtype(in_type) || !valid_dtype(out_type) || !dw_out_dims(H, W, kh, kw, stride, pad, &Ho, &Wo))
        return 0;
    // The fused paths need no workspace (the answer assumes 16-byte aligned
    // tensors, as every torch allocation is).
    const DwArgs d = dw_args(batch, H, W, C_in, depth_mult, kh, kw, stride, pad, Ho, Wo, in_type, nullptr,
                             nullptr, nullptr);
    if (dwsep_path(d, C_out, out_type, nullptr, nullptr)) return 0;
    return dwsep_ws(batch, Ho, Wo, C_in, depth_mult, C_out, in_type);
}

isam_status_t isam_dwsep_conv(int64_t batch, int64_t H, int64_t W, int64_t C_in, int64_t depth_mult,
                              int64_t kh, int64_t kw, int64_t stride, int64_t pad, int64_t C_out,
                              int in_type, const void* x, const void* dw_filter, const void* pw_weight,
                              int out_type, void* y, void* workspace, size_t workspace_bytes,
                              void* stream) {
    g_last_error.clear();
    const char* who = "isam_dwsep_conv";
    if (batch < 0 || H <= 0 || W <= 0 || C_in <= 0 || depth_mult <= 0 || kh <= 0 || kw <= 0 ||
        stride <= 0 || pad < 0 || C_out <= 0)
        return fail(ISAM_ERR_INVALID_ARG, "%s: sizes must be positive (batch, pad >= 0)", who);
    if (!valid_dtype(in_type) || !valid_dtype(out_type))
        return fail(ISAM_ERR_INVALID_ARG, "%s: dtype must be ISAM_F32 (0) or ISAM_BF16 (1)", who);
    int64_t Ho, Wo;
    if (!dw_out_dims(H, W, kh, kw, stride, pad, &Ho, &Wo))
        return fail(ISAM_ERR_INVALID_ARG, "%s: empty output (kernel larger than padded image)", who);
    if (batch == 0) return ISAM_OK;
    if (!x || !dw_filter || !pw_weight || !y)
        return fail(ISAM_ERR_INVALID_ARG, "%s: NULL tensor pointer", who);
    const size_t es = dsize(in_type);
    const int64_t Mp = batch * Ho * Wo, Cm = C_in * depth_mult;
    const int64_t x_el = batch * H * W * C_in, y_el = Mp * C_out, Y_el = Mp * Cm;
    if ((int64_t)(x_el * es) > kMaxExtent || (int64_t)(Y_el * es) > kMaxExtent ||
        (int64_t)(y_el * dsize(out_type)) > kMaxExtent)
        return fail(ISAM_ERR_UNSUPPORTED, "%s: a tensor spans more than 2^31 bytes", who);
    const size_t yb = (size_t)y_el * dsize(out_type);
    if (overlaps(y, yb, x, (size_t)x_el * es) ||
        overlaps(y, yb, dw_filter, (size_t)(kh * kw * Cm) * es) ||
        overlaps(y, yb, pw_weight, (size_t)(Cm * C_out) * es))
        return fail(ISAM_ERR_INVALID_ARG, "%s: y overlaps an input", who);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const size_t y_bytes = align256((size_t)Y_el * es);
    DwArgs d = dw_args(batch, H, W, C_in, depth_mult, kh, kw, stride, pad, Ho, Wo, in_type, x, dw_filter, workspace);
    // Fused paths: the depthwise result stays in LDS and feeds the MFMA
    // product directly (bf16 input, or fp32 input and output; 3x3 stride 1
    // pad 1 shapes that fit).  No workspace is touched.
    const int path = dwsep_path(d, C_out, out_type, pw_weight, y);
    if (path == 1) {
        if (log_enabled()) fprintf(stderr, "[isam] dwsep fused bf16\n");
        hipError_t e = launch_dwsep_fused(d, pw_weight, y, C_out, out_type, device_lds_max(), device_cus(), s);
        return e == hipSuccess ? ISAM_OK : hip_fail(e, who);
    }
    if (path == 2) {
        if (log_enabled()) fprintf(stderr, "[isam] dwsep fused fp32\n");
        hipError_t e = launch_dwsep_fused_f32(d, pw_weight, y, C_out, device_cus(), s);
        return e == hipSuccess ? ISAM_OK : hip_fail(e, who);
    }
    const size_t need = dwsep_ws(batch, Ho, Wo, C_in, depth_mult, C_out, in_type);
    if (!workspace || workspace_bytes < y_bytes)
        return fail(ISAM_ERR_WORKSPACE, "%s: workspace of %zu bytes < %zu required", who, workspace_bytes, need);
    if (overlaps(workspace, workspace_bytes, y, yb) || overlaps(workspace, workspace_bytes, x, (size_t)x_el * es) ||
        overlaps(workspace, workspace_bytes, dw_filter, (size_t)(kh * kw * Cm) * es) ||
        overlaps(workspace, workspace_bytes, pw_weight, (size_t)(Cm * C_out) * es))
        return fail(ISAM_ERR_INVALID_ARG, "%s: workspace overlaps a tensor", who);
    hipError_t e = launch_depthwise(d, s);
    if (e != hipSuccess) return hip_fail(e, who);
    char* gws = static_cast<char*>(workspace) + y_bytes;
    const size_t gws_bytes = workspace_bytes - y_bytes;
    return run_gemm(0, 0, Mp, C_out, Cm, in_type, workspace, Cm, pw_weight, C_out, 0, out_type, y, C_out,
                    nullptr, gws_bytes ? gws : nullptr, gws_bytes, s, who);
}

size_t isam_gru_forward_workspace_size(int64_t T, int64_t batch, int64_t input_size,
                                       int64_t hidden_size, int w_type) {
    (void)input_size;
    if (T < 0 || batch <= 0 || hidden_size <= 0 || !valid_dtype(w_type)) return 0;
    const size_t gx = align256((size_t)T * (size_t)batch * 3 * (size_t)hidden_size * sizeof(float));
    const size_t hb = align256(((size_t)T + 1) * (size_t)gru_slot_elems(batch, hidden_size, (int64_t)dsize(w_type)) *
                               dsize(w_type));
    const size_t hs = align256(2 * (size_t)batch * (size_t)hidden_size * sizeof(float));
    return gx + hb + kGruSyncBytes + hs;
}

}  // extern "C"

// Shared body of isam_gru_forward and isam_gru_forward_noalloc.  With
// no_alloc, the workspace is the library's static scratch on the current
// device (looked up after validation), so nothing is allocated.
static isam_status_t gru_forward_impl(int64_t T, int64_t batch, int64_t input_size, int64_t hidden_size,
                                      int w_type, const void* x, const float* h0, const void* W,
                                      const void* U, const float* bias, const float* bias_hn,
                                      float* h_seq, float* h_T, void* workspace, size_t workspace_bytes,
                                      void* stream, const char* who, bool no_alloc) {
    if (T < 0 || batch < 0 || input_size <= 0 || hidden_size <= 0)
        return fail(ISAM_ERR_INVALID_ARG, "%s: T, batch >= 0 and input_size, hidden_size > 0 required", who);
    if (!valid_dtype(w_type)) return fail(ISAM_ERR_INVALID_ARG, "%s: w_type must be 0 or 1", who);
    if (!h_seq && !h_T) return fail(ISAM_ERR_INVALID_ARG, "%s: h_seq and h_T are both NULL", who);
    const int64_t H = hidden_size, I = input_size;
    const int64_t E = w_type == ISAM_BF16 ? 8 : 4;
    if (H % E) return fail(ISAM_ERR_UNSUPPORTED, "%s: hidden_size must be a multiple of %lld", who, (long long)E);
    if (batch == 0) return ISAM_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const size_t es = dsize(w_type);
    const size_t state = (size_t)batch * H * sizeof(float);
    if (h_seq && h_T && overlaps(h_seq, (size_t)T * state, h_T, state))
        return fail(ISAM_ERR_INVALID_ARG, "%s: h_seq overlaps h_T", who);
    if (T == 0) {
        if (!h_T) return ISAM_OK;
        if (h0 && overlaps(h0, state, h_T, state)) return fail(ISAM_ERR_INVALID_ARG, "%s: h_T overlaps h0", who);
        hipError_t e = launch_gru_copy_state(h0, h_T, batch * H, s);
        return e == hipSuccess ? ISAM_OK : hip_fail(e, who);
    }
    if (!x || !W || !U) return fail(ISAM_ERR_INVALID_ARG, "%s: x, W or U is NULL", who);
    if ((uintptr_t)U & 15) return fail(ISAM_ERR_UNSUPPORTED, "%s: U must be 16-byte aligned", who);
    const size_t xb = (size_t)T * batch * I * es, wb = (size_t)3 * H * I * es, ub = (size_t)3 * H * H * es;
    if ((int64_t)xb > kMaxExtent || (int64_t)wb > kMaxExtent || (int64_t)ub > kMaxExtent ||
        (int64_t)((size_t)T * batch * 3 * H * sizeof(float)) > kMaxExtent ||
        (int64_t)(((size_t)T + 1) * (size_t)gru_slot_elems(batch, H, (int64_t)es) * es) > kMaxExtent)
        return fail(ISAM_ERR_UNSUPPORTED, "%s: a tensor spans more than 2^31 bytes", who);
    const void* ins[6] = {x, W, U, h0, bias, bias_hn};
    const size_t inb[6] = {xb, wb, ub, state, (size_t)3 * H * sizeof(float), (size_t)H * sizeof(float)};
    for (int i = 0; i < 6; ++i) {
        if ((h_seq && overlaps(h_seq, (size_t)T * state, ins[i], inb[i])) || (h_T && overlaps(h_T, state, ins[i], inb[i])))
            return fail(ISAM_ERR_INVALID_ARG, "%s: an output overlaps an input", who);
    }
    const size_t need = isam_gru_forward_workspace_size(T, batch, I, H, w_type);
    if (no_alloc) {
        if (need > kGruScratchBytes)
            return fail(ISAM_ERR_WORKSPACE, "%s: these sizes need %zu bytes of scratch; the static scratch holds %zu",
                        who, need, (size_t)kGruScratchBytes);
        hipError_t se = gru_scratch(&workspace);
        if (se != hipSuccess) return hip_fail(se, who);
        workspace_bytes = kGruScratchBytes;
    }
    if (!workspace || workspace_bytes < need)
        return fail(ISAM_ERR_WORKSPACE, "%s: workspace of %zu bytes < %zu required", who, workspace_bytes, need);
    if ((h_seq && overlaps(workspace, need, h_seq, (size_t)T * state)) || (h_T && overlaps(workspace, need, h_T, state)))
        return fail(ISAM_ERR_INVALID_ARG, "%s: workspace overlaps an output", who);

    // Plan: batch groups of up to 16 columns (one 16-wide MFMA tile); hidden
    // units per workgroup J the smallest power of two that lets every
    // workgroup stay resident, at most 16 (three gates x 16 = 48 rows).
    const int BB = (int)std::min<int64_t>(batch, 16);
    const int64_t n_bg = cdiv(batch, BB);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, who);
    int cus = device_cus();
    int lds_max = 0;
    e = hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
    if (e != hipSuccess) return hip_fail(e, who);
    // Three schedules.  The batch-group kernel below, where it applies; else
    // one persistent kernel with U resident in LDS and a grid barrier between
    // steps, or one kernel per step, which re-reads U from the memory-side
    // cache every step (the L2 does not keep it across kernel boundaries) but
    // pays no grid barrier.  Measured on MI355X (T = 64, I = 1024): the
    // stepwise schedule is faster up to batch 16 while U is at most 16 MB
    // (fp32 H = 1024 batch 4: 375 vs 508 us), and up to batch 4 while U is at
    // most 32 MB (bf16 H = 2048 batch 4: 430 vs 511 us); the persistent one
    // elsewhere.  ISAM_GRU_MODE=group|persistent|steps overrides; the stepwise
    // schedule also runs whenever the persistent kernel has no resident tiling.
    const char* mode_env = getenv("ISAM_GRU_MODE");
    const double u_mb = 3.0 * (double)H * (double)H * (double)es / (1 << 20);
    bool step_mode = (batch <= 16 && u_mb <= 16.0) || (batch <= 4 && u_mb <= 32.0);
    if (mode_env && strcmp(mode_env, "persistent") == 0) step_mode = false;
    if (mode_env && strcmp(mode_env, "steps") == 0) step_mode = true;
    // Batch-group schedule (bf16, hidden 256..1024 in steps of 256): G barrier
    // domains of P = H/32 workgroups, each domain a slice of at most 16 batch
    // columns with the whole of U in its workgroups' registers.  As many
    // domains as the batch, the CUs and the barrier area allow.
    // Workgroups are dealt to the XCDs round-robin (32 CUs each on gfx950), so
    // a domain of P workgroups taken at a stride of the XCD count lands on
    // one XCD; the grid is X * P * ceil(G / X) workgroups.
    int groups = 0, group_wgs = 0;
    const int xcds = cus % 32 == 0 ? cus / 32 : 1;
    const bool group_allowed = !(mode_env && (strcmp(mode_env, "persistent") == 0 || strcmp(mode_env, "steps") == 0));
    if (group_allowed && w_type == ISAM_BF16 && gru_group_supported(H)) {
        const int P = (int)(H / kGruGroupUnits);
        const int64_t resident = (int64_t)cus * gru_group_blocks_per_cu(H);
        const int64_t max_domains = kGruBarrierBytes / 4 / 512 - 1;
        for (int64_t g = std::min<int64_t>(batch, max_domains); g >= 1; --g) {
            const int64_t wgs = (int64_t)xcds * P * cdiv(g, xcds);
            if (wgs <= resident && wgs <= kGruMaxWgs) {
                if (cdiv(batch, g) <= 16) { groups = (int)g; group_wgs = (int)wgs; }
                break;
            }
        }
    }
    if (mode_env && strcmp(mode_env, "group") == 0 && !groups)
        return fail(ISAM_ERR_UNSUPPORTED, "%s: ISAM_GRU_MODE=group needs bf16 weights, hidden 256/512/768/1024 and "
                    "at most 16 batch columns per domain", who);
    // Units per workgroup: the smallest power of two whose grid fits one
    // workgroup per CU (measured faster than packing two per CU); if none
    // does, the smallest that fits at the occupancy limit.  Batch groups
    // have separate barriers.
    int J = 0;
    int n_wg = 0;
    if (groups) {
        step_mode = false;
        J = kGruGroupUnits;
        n_wg = group_wgs;
    } else if (!step_mode) {
        for (int pass = 0; pass < 2 && !J; ++pass) {
            for (int cand = 1; cand <= 16; cand *= 2) {
                if (H % cand) continue;
                if (cand * BB > 256) break;
                const size_t lds = gru_lds_bytes(w_type, H, cand);
                if (lds > (size_t)lds_max) break;
                const int64_t wgs = (H / cand) * n_bg;
                const int per_cu = pass == 0 ? 1 : gru_blocks_per_cu(w_type, lds);
                if (wgs <= (int64_t)cus * per_cu) { J = cand; n_wg = (int)wgs; break; }
            }
        }
        const char* jenv = getenv("ISAM_GRU_J");
        if (J && jenv) {  // tuning override, ignored when it does not fit
            const int v = atoi(jenv);
            const size_t lds = (v >= 1 && v <= 16) ? gru_lds_bytes(w_type, H, v) : 0;
            if (v >= 1 && v <= 16 && H % v == 0 && v * BB <= 256 && lds <= (size_t)lds_max &&
                (H / v) * n_bg <= (int64_t)cus * std::min(2, gru_blocks_per_cu(w_type, lds))) {
                J = v;
                n_wg = (int)((H / v) * n_bg);
            }
        }
        if (!J || n_bg > kGruBarrierBytes / 4 / 512 - 1) step_mode = true;  // one 512-word barrier domain per batch group
    }
    if (step_mode) {
        // No residency constraint: the smallest power of two whose grid fits
        // one workgroup per CU, else the largest that divides H.
        for (int cand = 1; cand <= 16; cand *= 2) {
            if (H % cand || cand * BB > 256) continue;
            J = cand;
            if ((H / cand) * n_bg <= (int64_t)cus) break;
        }
        if (const char* env = getenv("ISAM_GRU_J")) {  // tuning override, ignored when invalid
            const int v = atoi(env);
            if (v >= 1 && v <= 16 && H % v == 0 && v * BB <= 256) J = v;
        }
        if ((H / J) * n_bg > INT32_MAX) return fail(ISAM_ERR_UNSUPPORTED, "%s: grid too large", who);
        n_wg = (int)((H / J) * n_bg);
    }
    if (log_enabled())
        fprintf(stderr, "[isam] gru T=%lld B=%lld I=%lld H=%lld w=%d mode=%s J=%d BB=%d wgs=%d groups=%d\n", (long long)T,
                (long long)batch, (long long)I, (long long)H, w_type,
                groups ? "group" : (step_mode ? "steps" : "persistent"), J, BB, n_wg, groups);

    char* ws = static_cast<char*>(workspace);
    float* gx = reinterpret_cast<float*>(ws);
    const size_t gx_b = align256((size_t)T * batch * 3 * H * sizeof(float));
    void* hbuf = ws + gx_b;
    const int64_t slot = gru_slot_elems(batch, H, (int64_t)es);
    const size_t hb_b = align256(((size_t)T + 1) * (size_t)slot * es);
    unsigned* sync = reinterpret_cast<unsigned*>(ws + gx_b + hb_b);
    float* hstate = reinterpret_cast<float*>(ws + gx_b + hb_b + kGruSyncBytes);

    // Input projection for all steps: Gx[T*batch][3H] = x[T*batch][I] . W^T.
    isam_status_t st = run_gemm(0, 1, T * batch, 3 * H, I, w_type, x, I, W, I, 0, ISAM_F32, gx, 3 * H,
                                nullptr, nullptr, 0, s, who);
    if (st != ISAM_OK) return st;
    GruArgs g{};
    g.T = T;
    g.batch = batch;
    g.I = I;
    g.H = H;
    g.w_type = w_type;
    g.gx = gx;
    g.h0 = h0;
    g.U = U;
    g.bias = bias;
    g.bias_hn = bias_hn;
    g.h_seq = h_seq;
    g.h_T = h_T;
    g.hbuf = hbuf;
    g.slot = slot;
    g.sync = sync;
    g.timeout_ticks = kGruTimeoutTicks;
    // Test hook: a barrier target one arrival beyond the grid is never met, so
    // every wait ends at a 100 us bound and the outputs come back as NaN.
    if (const char* st_env = getenv("ISAM_GRU_TEST_STALL"); st_env && st_env[0] == '1') {
        g.stall = 1;
        g.timeout_ticks = 10000;
    }
    g.units_per_wg = J;
    g.batch_per_wg = BB;
    g.n_wg = n_wg;
    // First-level barrier groups of 8 workgroups (measured fastest), larger
    // when a domain would otherwise need more group counters than it has.
    g.barrier_group = (int)std::max<int64_t>(8, cdiv(H / J, kGruMaxGroupsPerDomain));
    g.groups = groups;
    g.xcds = xcds;
    if (groups) {
        g.barrier_group = 16;  // two first-level counters for 32 members (measured best of 4..32)
        if (const char* bg_env = getenv("ISAM_GRU_BGROUP")) {  // tuning override
            const int v = atoi(bg_env);
            if (v >= 1 && cdiv(n_wg / groups, v) <= kGruMaxGroupsPerDomain) g.barrier_group = v;
        }
        if (const char* sc_env = getenv("ISAM_GRU_GROUP_SCOPE"); sc_env && strcmp(sc_env, "device") == 0)
            g.device_scope = 1;
        e = launch_gru_group(g, s);
    } else {
        e = step_mode ? launch_gru_steps(g, hstate, s) : launch_gru_recurrent(g, s);
    }
    if (e != hipSuccess) return hip_fail(e, who);
    return ISAM_OK;
}

extern "C" isam_status_t isam_gru_forward(int64_t T, int64_t batch, int64_t input_size, int64_t hidden_size,
                                          int w_type, const void* x, const float* h0, const void* W,
                                          const void* U, const float* bias, const float* bias_hn,
                                          float* h_seq, float* h_T, void* workspace,
                                          size_t workspace_bytes, void* stream) {
    g_last_error.clear();
    return gru_forward_impl(T, batch, input_size, hidden_size, w_type, x, h0, W, U, bias, bias_hn, h_seq, h_T,
                            workspace, workspace_bytes, stream, "isam_gru_forward", false);
}

extern "C" isam_status_t isam_gru_forward_noalloc(int64_t T, int64_t batch, int64_t input_size,
                                                  int64_t hidden_size, int w_type, const void* x, const float* h0,
                                                  const void* W, const void* U, const float* bias,
                                                  const float* bias_hn, float* h_seq, float* h_T, void* stream) {
    g_last_error.clear();
    return gru_forward_impl(T, batch, input_size, hidden_size, w_type, x, h0, W, U, bias, bias_hn, h_seq, h_T,
                            nullptr, 0, stream, "isam_gru_forward_noalloc", true);
}

extern "C" isam_status_t isam_conv1d(int64_t batch, int64_t L, int64_t Ki, int64_t D, int64_t Ko, int ab_type,
                                     const void* A, const void* B, int accumulate, int c_type, void* C,
                                     void* stream) {
    g_last_error.clear();
    const char* who = "isam_conv1d";
    if (batch < 0 || L < 0 || Ki <= 0 || D <= 0 || Ko < 0)
        return fail(ISAM_ERR_INVALID_ARG, "%s: batch, L, Ko >= 0 and Ki, D > 0 required", who);
    if (!valid_dtype(ab_type) || !valid_dtype(c_type)) return fail(ISAM_ERR_INVALID_ARG, "%s: bad dtype", who);
    if (accumulate != 0 && accumulate != 1) return fail(ISAM_ERR_INVALID_ARG, "%s: accumulate must be 0 or 1", who);
    const int64_t X = L - D + 1;  // valid output positions
    if (batch == 0 || Ko == 0 || X <= 0) return ISAM_OK;
    if (!A || !B || !C) return fail(ISAM_ERR_INVALID_ARG, "%s: NULL tensor", who);
    const int64_t es = (int64_t)dsize(ab_type), cs = (int64_t)dsize(c_type);
    const int64_t a_bytes = batch * L * Ki * es, b_bytes = D * Ki * Ko * es, c_bytes = batch * X * Ko * cs;
    if (L * Ki * es > kMaxExtent || b_bytes > kMaxExtent || X * Ko * cs > kMaxExtent)
        return fail(ISAM_ERR_UNSUPPORTED, "%s: a tensor of one sequence spans more than 2^31 bytes", who);
    if (batch > 65535) return fail(ISAM_ERR_UNSUPPORTED, "%s: more than 65535 sequences in one call", who);
    if (overlaps(C, (size_t)c_bytes, A, (size_t)a_bytes) || overlaps(C, (size_t)c_bytes, B, (size_t)b_bytes))
        return fail(ISAM_ERR_INVALID_ARG, "%s: C overlaps A or B", who);
    // Sequence i is one product C_i[X][Ko] = A'_i[X][D*Ki] . B'[D*Ki][Ko]: row x of
    // A'_i is the D*Ki contiguous values A[i][x .. x+D-1][:], i.e. rows of A_i
    // read with leading dimension Ki (consecutive rows overlap), and B' is B
    // read as [D*Ki][Ko].
    return run_gemm(0, 0, X, Ko, D * Ki, ab_type, A, Ki, B, Ko, accumulate, c_type, C, Ko, nullptr, nullptr, 0,
                    static_cast<hipStream_t>(stream), who, batch, L * Ki * es, 0, X * Ko * cs);
}

extern "C" {

const char* isam_status_string(int status) {
    switch (status) {
        case ISAM_OK: return "ISAM_OK";
        case ISAM_ERR_INVALID_ARG: return "ISAM_ERR_INVALID_ARG: invalid argument";
        case ISAM_ERR_UNSUPPORTED: return "ISAM_ERR_UNSUPPORTED: unsupported configuration";
        case ISAM_ERR_WORKSPACE: return "ISAM_ERR_WORKSPACE: workspace missing or too small";
        case ISAM_ERR_HIP: return "ISAM_ERR_HIP: HIP runtime error";
        default: return "unknown isam status";
    }
}

const char* isam_last_error(void) { return g_last_error.c_str(); }

int isam_version(void) { return 101; }

}  // extern "C"
