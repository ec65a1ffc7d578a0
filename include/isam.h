/*
 * isam.h -- C ABI of the MI355X (gfx950) library for the dense hot path that
 * ISA Mapper (Sotoudeh et al., SysML 2019, arXiv 1810.09958) maps deep
 * learning layers onto: matrix multiplication, the separable depthwise
 * convolution factored into a depthwise stencil plus a matrix multiplication,
 * and the GRU recurrence.
 *
 * Conventions for every entry point
 *   - Tensor pointers are DEVICE pointers (hipMalloc'd or torch CUDA tensors)
 *     unless stated otherwise.  Layouts are row-major; images are NHWC.
 *   - bf16 tensors hold 16-bit bfloat16 patterns; fp32 accumulation always.
 *   - The caller owns every buffer, including the workspace.  The library
 *     allocates no device memory.  Pointers are borrowed until the work
 *     queued on `stream` has finished.
 *   - Calls are asynchronous: they validate their arguments on the host,
 *     enqueue kernels on `stream` (a hipStream_t; NULL = default stream) and
 *     return.  There is no host synchronisation inside a call.
 *   - Validation happens before any HIP call.  A non-OK status means nothing
 *     was launched, except ISAM_ERR_HIP, which reports a failed launch.
 *     isam_last_error() holds a readable reason for the last non-OK status
 *     on the calling thread.  No C++ exception crosses this interface.
 *   - Outputs must not overlap inputs (detected by address range).
 *   - Each operand's addressed extent must be below 2^31 bytes
 *     (ISAM_ERR_UNSUPPORTED otherwise).
 *   - Entry points are thread-safe.  The library keeps no state between
 *     calls other than per-device caches filled once and never changed: CU
 *     count, LDS size, the dynamic-LDS limit set on each kernel that needs
 *     one, resident workgroups per CU of the persistent kernels, and the
 *     address of the static scratch that isam_gru_forward_noalloc uses; and one process-wide 64-bit counter
 *     (random start) that gives each in-kernel split-K or stream-K sum of
 *     isam_gemm its own flag value.
 */
#ifndef ISAM_H
#define ISAM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { ISAM_F32 = 0, ISAM_BF16 = 1 } isam_dtype_t;

typedef enum {
    ISAM_OK = 0,
    ISAM_ERR_INVALID_ARG = 1, /* bad size, pointer, leading dimension, dtype or aliasing */
    ISAM_ERR_UNSUPPORTED = 2, /* valid request outside what the library implements */
    ISAM_ERR_WORKSPACE = 3,   /* workspace missing or smaller than the *_workspace_size query */
    ISAM_ERR_HIP = 4          /* a HIP launch failed; isam_last_error() has the HIP message */
} isam_status_t;

/*
 * Matrix multiplication, the paper's first listing (Section 2):
 *   C[i][j] (+)= sum_k a(i,k) * b(k,j)
 * The listing accumulates into C; accumulate = 1 keeps that form (C += A.B),
 * accumulate = 0 overwrites (C = A.B).  The K order of the sum is free
 * (Section 2.1); results are compared with a tolerance, not bit for bit.
 *
 *   trans_a = 0: A is [M][K], element a(i,k) = A[i*lda + k], lda >= K
 *   trans_a = 1: A is [K][M], element a(i,k) = A[k*lda + i], lda >= M
 *   trans_b = 0: B is [K][N], element b(k,j) = B[k*ldb + j], ldb >= N
 *   trans_b = 1: B is [N][K], element b(k,j) = B[j*ldb + k], ldb >= K
 *   C is [M][N] with ldc >= N, dtype c_type (ISAM_F32 or ISAM_BF16; bf16
 *   outputs are rounded to nearest-even from the fp32 accumulator).
 *   ab_type is the shared dtype of A and B.
 * M == 0 or N == 0: no-op.  K == 0: C = 0 (accumulate = 0) or unchanged.
 * workspace: device buffer of at least isam_gemm_workspace_size(...) bytes,
 * used for split-K partial sums; with a smaller (or NULL) workspace the call
 * still succeeds on a plan without split-K.  Deep products split along K into
 * two slices on 256x256 tiles sum the slices inside the kernel when both
 * slices of every tile run on one XCD (tile count a multiple of the XCD
 * count, K a multiple of 64, workspace 256-byte aligned): the second slice
 * waits for the first's flag in the workspace (a bounded wait; if it ever
 * expires the tile's outputs are NaN) and adds its partial sums in a fixed
 * order, so results stay deterministic; when every workgroup of the grid is
 * resident at once, each slice instead finishes half of the tile's rows with
 * the other slice's partial sums for that half (the same sums).  Other split plans sum the slices
 * in a second kernel.  bf16 products whose tile count leaves most compute
 * units idle in a last partial round (A not transposed, 16-byte aligned
 * rows, workspace 256-byte aligned) run a stream-K schedule instead
 * (Section 3.4's allocation of work to processing units): a persistent grid
 * sized to what the device holds at once, the workgroups of one XCD splitting
 * that XCD's range of tiles: whole tiles round by round first, then equal
 * shares of the remaining (output tile, 64-deep K tile) units; a tile's owner
 * starts from the partial sums the later shares of its K range left in the
 * workspace (one fp32 tile and one flag line per workgroup), added in a fixed
 * order, with the same bounded wait and NaN on expiry.
 * Operands whose rows cannot be copied 16 bytes at a time (K, or M with
 * trans_a / N without trans_b, not a multiple of 8 bf16 / 4 fp32 values, or a
 * base pointer or leading dimension off 16 bytes), and bf16 A with trans_a,
 * are first copied into the start of the workspace when the product is large
 * enough for the large tiles and the workspace (256-byte aligned) holds the
 * copies: A as [M][Kp], B as [Kp][N] (trans_b = 0, N a multiple of the vector
 * width) or [N][Kp], each rounded up to 256 bytes, with zeros in the padded K
 * positions (Kp: K rounded up to the vector width, or to a multiple of 64 when
 * both operands are copied and that adds at most K/16); the rest of the
 * workspace serves the packed product as above.  isam_gemm_workspace_size
 * includes these bytes when the sizes alone call for them; a caller passing
 * misaligned pointers or leading dimensions adds them itself, or the product
 * runs on the element-wise tile kernel.  A workspace that overlaps A, B or C
 * is rejected.
 * Large fp32 products (A [M][K]; B [N][K], or [K][N] with N a multiple of 8;
 * M*N >= 512*(M+N); workspace 256-byte aligned and holding the copies) run on
 * the bf16 matrix cores: each operand value x is split into three bf16 terms
 * h = bf16(x), m = bf16(x - h), l = bf16(x - h - m), copied into the start of
 * the workspace as six K blocks (12 bytes per operand value), and one bf16
 * product over K' = 6*Kp sums hh + hm + mh + hl + lh + mm in fp32: the fp32
 * product to within the dropped terms (below 2^-23 of |a*b|).  Inputs must be
 * finite and below 3.39e38 in magnitude there (an infinite input gives NaN
 * instead of +-inf).  isam_gemm_workspace_size includes these bytes when the
 * split applies; with a smaller workspace the fp32 tile kernel runs.  The
 * workspace needs no initial contents; concurrent calls must not share one.
 */
isam_status_t isam_gemm(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                        int ab_type, const void* A, int64_t lda, const void* B, int64_t ldb,
                        int accumulate, int c_type, void* C, int64_t ldc,
                        void* workspace, size_t workspace_bytes, void* stream);

/* Workspace (bytes) the preferred plan of isam_gemm needs for these sizes (split-K or
 * stream-K partial sums, packed or split operand copies); 0 if none. */
size_t isam_gemm_workspace_size(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K,
                                int ab_type, int c_type);

/*
 * Separable depthwise convolution, the paper's third listing (Section 2):
 *   y[b][i][j][k] = sum_{di,dj,q,r} x~[b][s*i+di-pad][s*j+dj-pad][q]
 *                                   * D[di][dj][q][r] * P[c*q + r][k]
 * computed in the factored form the mapper exposes by distributing the
 * pointwise product out of the (di, dj) sum (Section 2.3): first the
 * depthwise stencil Y[b][i][j][c*q+r] = sum_{di,dj} x~ * D, then the
 * pointwise matrix product y = Y . P with M = batch*Ho*Wo, K = C_in*c,
 * N = C_out.  x~ is x with zero padding `pad`.
 *
 *   x          [batch][H][W][C_in]                  (in_type)
 *   dw_filter  [kh][kw][C_in][depth_mult]           (in_type)
 *   pw_weight  [C_in*depth_mult][C_out]             (in_type)
 *   y          [batch][Ho][Wo][C_out]               (out_type)
 *   Ho = (H + 2*pad - kh)/stride + 1, Wo = (W + 2*pad - kw)/stride + 1 (both > 0)
 * The intermediate Y is held in the workspace in in_type (bf16 Y is rounded
 * to nearest-even).  batch == 0: no-op.
 * Precision: fp32 inputs give fp32-level results.  Where the fused fp32
 * kernel runs (3x3, stride 1, pad 1, multiplier 1; see the workspace query),
 * each fp32 product of the pointwise step is formed from a three-way bf16
 * split of both operands (six bf16 products, fp32 accumulation; the dropped
 * terms are below 2^-23 of the product).
 */
isam_status_t isam_dwsep_conv(int64_t batch, int64_t H, int64_t W, int64_t C_in, int64_t depth_mult,
                              int64_t kh, int64_t kw, int64_t stride, int64_t pad, int64_t C_out,
                              int in_type, const void* x, const void* dw_filter, const void* pw_weight,
                              int out_type, void* y, void* workspace, size_t workspace_bytes,
                              void* stream);

size_t isam_dwsep_conv_workspace_size(int64_t batch, int64_t H, int64_t W, int64_t C_in,
                                      int64_t depth_mult, int64_t kh, int64_t kw, int64_t stride,
                                      int64_t pad, int64_t C_out, int in_type, int out_type);

/*
 * GRU forward over T steps.  GRU cells map onto matrix products plus
 * element-wise work (Section 6.1); the recurrence is scheduled as a priming
 * iteration, a recursive iteration with the weights persistent on chip, and a
 * finish iteration (Section 3.6), with the gate math fused to the products
 * (Section 6.2.2).  Cell, with gate blocks stacked r, z, n in W and U:
 *   r   = sigmoid(W_r x_t + U_r h_{t-1} + b_r)
 *   z   = sigmoid(W_z x_t + U_z h_{t-1} + b_z)
 *   n   = tanh(W_n x_t + b_n + r * (U_n h_{t-1} + b_hn))
 *   h_t = (1 - z) * n + z * h_{t-1}
 *
 *   x        [T][batch][input_size]      (w_type)
 *   W        [3*hidden][input_size]      (w_type)
 *   U        [3*hidden][hidden]          (w_type)
 *   h0       [batch][hidden] fp32, or NULL for zeros
 *   bias     [3*hidden] fp32 (b_r, b_z, b_n), or NULL
 *   bias_hn  [hidden] fp32, or NULL (the PyTorch b_hn form)
 *   h_seq    [T][batch][hidden] fp32 output, or NULL
 *   h_T      [batch][hidden] fp32 output, or NULL (at least one of the two)
 * hidden must be a multiple of 8 (bf16) or 4 (fp32).  The bf16 path rounds
 * h_{t-1} to bf16 only as the matrix-core operand; the state stays fp32.
 * T == 0: h_T = h0 (or zeros).  batch == 0: no-op.
 * Schedules (the faster one for the shape runs; the environment variable
 * ISAM_GRU_MODE = group | persistent | steps overrides):
 *   - batch-group (bf16 weights, hidden 256, 512, 768 or 1024, at most 16
 *     batch columns per domain): independent barrier domains of hidden/32
 *     workgroups, one batch slice each, U rows held in registers;
 *   - persistent: one kernel with U held in on-chip memory and a grid barrier
 *     per step;
 *   - stepwise: the priming, recursive and finish iterations as separate
 *     kernels, one per step, launched in order (no co-residency needed, so
 *     any hidden size that meets the multiple rule is supported).
 * The persistent and stepwise schedules give the same values bit for bit.
 * The batch-group and persistent schedules launch no more workgroups than
 * the device holds at once, as an ordinary kernel, and need all of them
 * resident: a barrier wait that exceeds 2 s (never on a device with no other
 * work; possible if work on other streams -- another persistent GRU call,
 * say -- keeps CUs occupied that long) ends the recurrence early and fills
 * h_seq and h_T with NaN.  Calls on one workspace must not overlap in time.
 */
isam_status_t isam_gru_forward(int64_t T, int64_t batch, int64_t input_size, int64_t hidden_size,
                               int w_type, const void* x, const float* h0, const void* W,
                               const void* U, const float* bias, const float* bias_hn,
                               float* h_seq, float* h_T, void* workspace, size_t workspace_bytes,
                               void* stream);

size_t isam_gru_forward_workspace_size(int64_t T, int64_t batch, int64_t input_size,
                                       int64_t hidden_size, int w_type);

/*
 * isam_gru_forward without a workspace argument and without any allocation,
 * for callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  Arguments,
 * results and errors are those of isam_gru_forward (bit for bit the same
 * outputs); the workspace is instead a static 64 MiB device array of the
 * library (one per device, held until the process ends), so sizes whose
 * isam_gru_forward_workspace_size exceeds 64 MiB are rejected with
 * ISAM_ERR_WORKSPACE (T = 64, batch 32, hidden 1024 needs about 28 MiB).
 * Every call on one device shares that array: calls that overlap in time on
 * the same device race and must be serialised by the caller (one stream, or
 * events).  No hipMalloc, hipFree or allocating library call is made.
 */
isam_status_t isam_gru_forward_noalloc(int64_t T, int64_t batch, int64_t input_size, int64_t hidden_size,
                                       int w_type, const void* x, const float* h0, const void* W,
                                       const void* U, const float* bias, const float* bias_hn,
                                       float* h_seq, float* h_T, void* stream);

/*
 * 1D convolution of the paper's second listing (Section 2), valid positions,
 * stride 1:
 *   C[i][x][ko] (+)= sum_{d < D} sum_{ki < Ki} A[i][x+d][ki] * B[d][ki][ko]
 * for x < X = L - D + 1.  Computed as the matrix-multiply mapping of Section
 * 2.2 without materialising anything: per sequence i one product
 * C_i[X][Ko] = A'_i[X][D*Ki] . B'[D*Ki][Ko], where row x of A'_i is the D*Ki
 * contiguous values A[i][x .. x+D-1][:] (rows of A_i read with leading
 * dimension Ki) and B' is B read as [D*Ki][Ko]; all sequences in one launch.
 *
 *   A  [batch][L][Ki]   (ab_type)        B  [D][Ki][Ko] (ab_type)
 *   C  [batch][X][Ko]   (c_type), fp32 accumulation, bf16 output rounded RNE
 * accumulate = 1 adds to C.  batch, Ko == 0 or X <= 0: no-op.  No workspace.
 * Errors: INVALID_ARG (bad sizes or dtype, NULL tensor, C overlapping A or B),
 * UNSUPPORTED (one sequence's A or C, or B, over 2^31 bytes; batch > 65535).
 */
isam_status_t isam_conv1d(int64_t batch, int64_t L, int64_t Ki, int64_t D, int64_t Ko, int ab_type,
                          const void* A, const void* B, int accumulate, int c_type, void* C,
                          void* stream);

/* Static text for a status code. */
const char* isam_status_string(int status);
/* Detail of the last non-OK status returned on the calling thread ("" if none). */
const char* isam_last_error(void);
/* Library version, major*10000 + minor*100 + patch. */
int isam_version(void);  /* 101: adds isam_conv1d */

#ifdef __cplusplus
}
#endif

#endif /* ISAM_H */
