// Internal launch interface between the C-ABI layer (api.cpp) and the HIP
// kernels.  Nothing here is exported.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace isam {

enum Dtype : int { kF32 = 0, kBF16 = 1 };

// One GEMM launch: C[M][N] (+)= op(A)[M][K] . op(B)[K][N].
struct GemmArgs {
    const void* A;
    const void* B;
    void* C;
    float* partial;        // split-K partial sums [k_splits][M][N] fp32 (k_splits > 1)
    const float* bias;     // optional per-column bias added in the epilogue (fp32, length N)
    int64_t M, N, K;
    int64_t lda, ldb, ldc;
    int trans_a, trans_b;
    int ab_type;           // kF32 / kBF16
    int c_type;            // kF32 / kBF16
    int accumulate;        // C += instead of C =
    // Strided batch (grid z): problem z uses A, B, C offset by z times these
    // byte strides.  batch == 1 for a single product; batched launches never
    // split K and never take the skinny kernels.
    int64_t batch;
    int64_t stride_a, stride_b, stride_c;
};

// Tile configurations of the MFMA tile kernel (see gemm.hip).
enum TileCfg : int {
    kTile256x256 = 0,  // 4 waves, 128x128 per wave
    kTile256x128 = 1,  // 4 waves, 128x64 per wave
    kTile128x128 = 2,  // 4 waves, 64x64 per wave
    kTile128x64 = 3,   // 4 waves, 64x32 per wave
    kTile64x64 = 4,    // 4 waves, 32x32 per wave
    kTile128x32 = 5,   // 4 waves, 32x32 per wave (tall-skinny)
    kTileCount
};

struct GemmPlan {
    int tile;        // TileCfg
    int vec;         // 1: 16-byte vector loads (needs alignment); 0: element loads
    int k_splits;    // >= 1
    int64_t k_per_split;  // multiple of the tile K depth
    int group_m;     // tile-row group size of the rasterisation
    int xcd_remap;   // spread consecutive tiles of one group over one XCD
    int dma;         // 1: direct-to-LDS kernel where it applies (bf16, A K-contiguous, vec)
    int dma_waves;   // 4 or 8 waves per workgroup for the direct-to-LDS kernel
    int fixup;       // 1: a two-slice split on 256x256 tiles may sum its slices inside the kernel
                     // 2: the same, each slice finishing half of the tile (whole grid resident)
    int skinny;      // 1: streaming kernel for N <= 32 (k_splits = K slices of skinny_k_slice);
                     // 2: bf16 row-streaming kernel (16 rows per workgroup, whole K, no split);
                     // 4: narrow dot-product kernel (N < 8, not a multiple of the vector width)
    int small;       // 1: small-product kernel (one 32x32 tile per workgroup, waves split K)
    int sk;          // 1: stream-K schedule of the direct-to-LDS kernel (persistent grid of
                     //    sk_grid workgroups sharing the (tile, K tile) units evenly)
    int sk_grid;
    int sk_keep;     // whole rounds left to the stream-K shares (0 or 1)
};
// Stream-K schedule: persistent grid size for a tile shape (one workgroup per
// CU; two for 128x128 tiles, whose ring takes half the LDS) and its workspace
// (one fp32 partial-sum tile and one 128-byte flag line per workgroup).
int gemm_sk_grid(int tile, int cus);
size_t gemm_sk_ws_bytes(int tile, int grid);
bool gemm_sk_tile(int tile);
// Small products: at most kSmallMaxTiles output tiles of 32x32 and K <= kSmallMaxK
// (A K-contiguous, 16-byte aligned operands, batch 1: checked by the caller).
constexpr int64_t kSmallMaxTiles = 64;
constexpr int64_t kSmallMaxK = 1024;
bool gemm_small_fits(int64_t M, int64_t N, int64_t K);
// Very shallow bf16 products (K <= 256, N <= 256, NN): B in registers, A streamed.
bool gemm_stream_fits(const GemmArgs& a);
constexpr int64_t kStreamMaxK = 256;  // planner: deepest K routed to it by default
hipError_t launch_gemm_stream(const GemmArgs& a, int cus, hipStream_t s);
hipError_t launch_gemm_small(const GemmArgs& a, hipStream_t s);
int64_t skinny_k_slice(int ab_type);
int skinny_rows_per_wg(int ab_type);
hipError_t launch_skinny(const GemmArgs& a, int splits, hipStream_t s);
int skinny_stream_rows();
hipError_t launch_skinny_rows(const GemmArgs& a, hipStream_t s);
// Narrow product (N < 8): dot-product kernel streaming A once (NN, A rows
// 16-byte aligned, any ldb).
hipError_t launch_narrow(const GemmArgs& a, hipStream_t s);

void tile_dims(int tile, int ab_type, int* bm, int* bn, int* bk);

// Launch facts cached per device and kernel (launch_cache.cpp): raise a
// kernel's dynamic-LDS limit to at least `lds` bytes, and its resident
// workgroups per CU at `threads` threads and `lds` dynamic LDS bytes (0 when
// the runtime cannot say).
hipError_t ensure_dynamic_lds(const void* fn, size_t lds);
int resident_per_cu(const void* fn, int threads, size_t lds);
hipError_t launch_gemm(const GemmArgs& a, const GemmPlan& p, hipStream_t s);
// Copies src[s_rows][s_cols] (leading dimension ld, elements of esize = 2 or 4
// bytes) into the dense dst[d_rows][d_cols] -- transposed (dst[i][j] =
// src[j][i]) if asked -- with zeros outside the source; d_cols * esize must
// be a multiple of 16 and dst 16-byte aligned for the plain copy.
// fp32 operand split into six bf16 K blocks of kp values (terms by the 2-bit
// fields of pattern: 0 = h, 1 = m, 2 = l).  k_rows = false: src [s_rows][K],
// dst [d_rows][6 kp] (d_cols = kp); k_rows = true: src [K][s_cols], dst
// [6 kp][d_cols] (d_rows = kp).  d_cols a multiple of 8, dst 16-byte aligned.
hipError_t launch_split6(const float* src, int64_t s_rows, int64_t s_cols, int64_t ld, uint16_t* dst,
                         int64_t d_rows, int64_t d_cols, int64_t kp, bool k_rows, uint32_t pattern, int cus,
                         hipStream_t s);
hipError_t launch_pack(const void* src, int64_t s_rows, int64_t s_cols, int64_t ld, void* dst, int64_t d_rows,
                       int64_t d_cols, int esize, bool transpose, int cus, hipStream_t s);

// Depthwise kh x kw convolution, NHWC.  Y is [batch][Ho][Wo][C*cm] in y_type.
struct DwArgs {
    const void* x;
    const void* w;  // [kh][kw][C][cm]
    void* y;
    int64_t batch, H, W, C, cm, kh, kw, stride, pad, Ho, Wo;
    int in_type, y_type;
};
hipError_t launch_depthwise(const DwArgs& a, hipStream_t s);
// Fused depthwise + pointwise (bf16 input): rows per tile, 0 if not applicable.
int dwsep_fused_rows(const DwArgs& d, int64_t C_out, int lds_max);
hipError_t launch_dwsep_fused(const DwArgs& d, const void* pw, void* out, int64_t C_out, int out_type, int lds_max,
                              int cus, hipStream_t s);
// Fused depthwise + pointwise, fp32 in and out (fp32 MFMA).
bool dwsep_fused_f32_ok(const DwArgs& d, int64_t C_out, int lds_max);
hipError_t launch_dwsep_fused_f32(const DwArgs& d, const void* pw, void* out, int64_t C_out, int cus, hipStream_t s);

// GRU recurrence (the input projection is a GemmArgs launch done before).
struct GruArgs {
    int64_t T, batch, I, H;
    int w_type;
    const float* gx;        // [T*batch][3H] fp32: x W^T (no bias)
    const float* h0;        // [batch][H] fp32 or null
    const void* U;          // [3H][H]
    const float* bias;      // [3H] or null
    const float* bias_hn;   // [H] or null
    float* h_seq;           // [T][batch][H] or null
    float* h_T;             // [batch][H] or null
    void* hbuf;             // [T+1] slots of `slot` elements in w_type: ring of per-step MFMA
                            // copies of h, slot t holding h_{t-1} as [batch][H]
    int64_t slot;           // elements per ring slot: batch*H rounded up to a multiple of 256 bytes
    unsigned* sync;         // barrier counters and error word (kGruSyncBytes, zeroed by the launch)
    uint64_t timeout_ticks; // bound on one barrier wait, in ticks of the 100 MHz constant clock
    int stall;              // 1: barrier targets one arrival beyond the grid (never met), so every
                            // wait runs into the bound; exercises the timeout path
    int units_per_wg;       // J
    int batch_per_wg;       // BB
    int n_wg;
    int barrier_group;      // workgroups per first-level barrier counter
    int groups;             // batch-group schedule: barrier domains (batch groups); 0 otherwise
    int device_scope;       // batch-group schedule: 1 = exchange through device scope even when a
                            // domain sits on one XCD
    int xcds;               // batch-group schedule: width of the round-robin dispatch over XCDs
};
// Barrier layout of the GRU kernel: per batch group a domain of 512 words
// holds the domain counter and up to 31 first-level group counters (64
// bytes apart).
constexpr int kGruMaxGroupsPerDomain = 31;
size_t gru_lds_bytes(int w_type, int64_t H, int J);
// Resident workgroups of the recurrent kernel per compute unit at this LDS size.
int gru_blocks_per_cu(int w_type, size_t lds);
// Barrier area of the GRU workspace: the domain counters of the grid barrier
// in the first 32 KiB, then per-domain flag words (64 per domain) and the XCC
// id of every workgroup (batch-group schedule).
constexpr int kGruBarrierBytes = 32768;
constexpr int kGruSyncBytes = 65536;
constexpr int kGruFlagWord = 8192;    // flags of domain d: words kGruFlagWord + 64 d ..
constexpr int kGruXccWord = 12288;    // XCC id of workgroup b: word kGruXccWord + b
constexpr int kGruMaxWgs = 4096;
// Ring slot stride in elements: whole 256-byte blocks, so no cache line holds
// parts of two slots.
inline int64_t gru_slot_elems(int64_t batch, int64_t H, int64_t es) { return (batch * H * es + 255) / 256 * 256 / es; }
hipError_t launch_gru_recurrent(const GruArgs& a, hipStream_t s);
// Batch-group persistent recurrence (bf16): `groups` independent barrier
// domains, each a set of n_wg / groups workgroups that own kGruGroupUnits
// hidden units apiece with their rows of U held in registers, and each a
// contiguous slice of the batch.  Needs H = 256 * KS (KS in 1..4), at most 16
// batch columns per group and every workgroup resident.
constexpr int kGruGroupUnits = 32;
bool gru_group_supported(int64_t H);
size_t gru_group_lds_bytes();
hipError_t launch_gru_group(const GruArgs& a, hipStream_t s);
// Resident workgroups of the batch-group kernel per compute unit (0: none).
int gru_group_blocks_per_cu(int64_t H);
// NaN into h_seq and h_T if the recurrence's sticky error word is set.
hipError_t launch_gru_error_fill(const GruArgs& a, hipStream_t s);
// Bound on one barrier wait of the persistent recurrence (2 s at 100 MHz).
constexpr uint64_t kGruTimeoutTicks = 200000000ull;
// Bounded wait of a GEMM tile's second K slice for the first (100 MHz ticks).
constexpr uint64_t kFixupTimeoutTicks = 200000000ull;
// Workspace of a two-slice split summed inside the kernel: one 256x256 fp32
// tile of partial sums per output tile, then one 128-byte flag line per tile.
size_t gemm_fixup_ws_bytes(int64_t M, int64_t N);
// Stepwise recurrence (state init + one kernel per step, launched in order);
// hstate is a [2][batch][H] fp32 workspace.
hipError_t launch_gru_steps(const GruArgs& a, float* hstate, hipStream_t s);
// Static scratch of the allocation-free GRU entry point: its device address on
// the current device (looked up once per device).
constexpr size_t kGruScratchBytes = size_t(64) << 20;
hipError_t gru_scratch(void** ptr);
// T == 0: h_T = h0 (or zeros when h0 is null).
hipError_t launch_gru_copy_state(const float* h0, float* h_T, int64_t n, hipStream_t s);

}  // namespace isam
