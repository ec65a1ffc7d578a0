/*
 * CPU ORACLE -- test infrastructure only.
 *
 * Plain, slow, obviously correct fp64 definitions of what the GPU library
 * computes.  Only the test suite, the smoke check and the benchmark's CPU
 * baseline leg may load this library; the product path never does.  It shares
 * no code, header or constant with the HIP sources.
 *
 * Conventions
 *   - Inputs are fp32 (dtype 0) or bf16 (dtype 1, passed as uint16 bit
 *     patterns).  bf16 is widened exactly: bits << 16 -> fp32 -> fp64.
 *   - Every reduction is a plain fp64 sum in ascending index order.
 *   - Outputs are fp64 arrays owned by the caller.
 *   - `threads` <= 0 means "OpenMP default".  Parallelism is over
 *     independent outputs only; it never changes an output's summation order.
 *
 * Paper: Sotoudeh et al., "ISA Mapper: A Compute and Hardware Agnostic Deep
 * Learning Compiler", SysML 2019 (arXiv 1810.09958).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define REF_F32 0
#define REF_BF16 1

static double ld_elem(const void* p, int dtype, int64_t i) {
    if (dtype == REF_F32) return (double)((const float*)p)[i];
    uint32_t bits = ((uint32_t)((const uint16_t*)p)[i]) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static void set_threads(int threads) {
#ifdef _OPENMP
    if (threads > 0) omp_set_num_threads(threads);
#else
    (void)threads;
#endif
}

int isam_ref_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/*
 * Matrix multiplication, the paper's first listing (Section 2): for every
 * (i, j), C[i][j] += sum over k of A[i][k] * B[k][j]; the loop order is free
 * (Section 2.1), the oracle sums k in ascending order.
 *
 *   a(i,k) = A[i*lda + k] (trans_a = 0) or A[k*lda + i] (trans_a = 1)
 *   b(k,j) = B[k*ldb + j] (trans_b = 0) or B[j*ldb + k] (trans_b = 1)
 *   C[i][j] = (C_in ? C_in[i][j] : 0) + sum_k a(i,k) b(k,j)       [M][N] dense
 *   S[i][j] = (C_in ? |C_in[i][j]| : 0) + sum_k |a(i,k)| |b(k,j)|  (optional)
 *
 * The inner loop runs over j with k fixed, so each C[i][j] still receives its
 * K products in ascending k.
 */
int isam_ref_gemm(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K, int ab_type,
                  const void* A, int64_t lda, const void* B, int64_t ldb,
                  const double* C_in, double* C, double* S, int threads) {
    if (M < 0 || N < 0 || K < 0 || !C) return 1;
    if (M == 0 || N == 0) return 0;
    set_threads(threads);
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < M; ++i) {
        double* c = C + i * N;
        double* s = S ? S + i * N : NULL;
        for (int64_t j = 0; j < N; ++j) {
            c[j] = C_in ? C_in[i * N + j] : 0.0;
            if (s) s[j] = C_in ? fabs(C_in[i * N + j]) : 0.0;
        }
        for (int64_t k = 0; k < K; ++k) {
            double a = ld_elem(A, ab_type, trans_a ? k * lda + i : i * lda + k);
            for (int64_t j = 0; j < N; ++j) {
                double b = ld_elem(B, ab_type, trans_b ? j * ldb + k : k * ldb + j);
                c[j] += a * b;
                if (s) s[j] += fabs(a) * fabs(b);
            }
        }
    }
    return 0;
}

/*
 * 1D convolution, the paper's second listing (Section 2): for every sequence i,
 * position x and output channel ko,
 *   C[i][x][ko] = (C_in ? C_in[i][x][ko] : 0) + sum over d, ki of A[i][x+d][ki] * B[d][ki][ko]
 * over the valid positions x < X = L - D + 1 (the listing has no padding and
 * stride 1).  S (optional) is the same sum of |A| |B| (+ |C_in|).
 *   A [batch][L][Ki], B [D][Ki][Ko], C, S [batch][X][Ko] fp64.
 * Summation order: d ascending, then ki ascending.
 */
int isam_ref_conv1d(int64_t batch, int64_t L, int64_t Ki, int64_t D, int64_t Ko, int dtype,
                    const void* A, const void* B, const double* C_in, double* C, double* S, int threads) {
    if (batch < 0 || L < 0 || Ki <= 0 || D <= 0 || Ko < 0 || !C) return 1;
    const int64_t X = L - D + 1;
    if (batch == 0 || Ko == 0 || X <= 0) return 0;
    set_threads(threads);
#pragma omp parallel for collapse(2) schedule(dynamic, 4)
    for (int64_t i = 0; i < batch; ++i) {
        for (int64_t x = 0; x < X; ++x) {
            for (int64_t ko = 0; ko < Ko; ++ko) {
                const int64_t o = (i * X + x) * Ko + ko;
                double acc = C_in ? C_in[o] : 0.0;
                double nrm = C_in ? fabs(C_in[o]) : 0.0;
                for (int64_t d = 0; d < D; ++d) {
                    for (int64_t ki = 0; ki < Ki; ++ki) {
                        const double a = ld_elem(A, dtype, (i * L + x + d) * Ki + ki);
                        const double b = ld_elem(B, dtype, (d * Ki + ki) * Ko + ko);
                        acc += a * b;
                        nrm += fabs(a) * fabs(b);
                    }
                }
                C[o] = acc;
                if (S) S[o] = nrm;
            }
        }
    }
    return 0;
}

/*
 * Depthwise half of the separable depthwise convolution (third listing,
 * Section 2), after factoring the pointwise weight out of the (di, dj)
 * reduction (Section 2.3):
 *
 *   Y[b][i][j][c*q + r] = sum_{di<kh, dj<kw} X~[b][s*i+di-pad][s*j+dj-pad][q] * D[di][dj][q][r]
 *
 * X~ is X with zeros outside [0,H) x [0,W).  x is NHWC [batch][H][W][C_in],
 * D is [kh][kw][C_in][c], Y is [batch][Ho][Wo][C_in*c] with
 * Ho = (H + 2 pad - kh)/s + 1, Wo likewise.  SY (optional) is the same sum of
 * |X~| |D|.  Summation order: di ascending, then dj ascending.
 */
int isam_ref_depthwise(int64_t batch, int64_t H, int64_t W, int64_t C_in, int64_t cm,
                       int64_t kh, int64_t kw, int64_t stride, int64_t pad, int dtype,
                       const void* x, const void* dw, double* Y, double* SY, int threads) {
    if (batch < 0 || H <= 0 || W <= 0 || C_in <= 0 || cm <= 0 || kh <= 0 || kw <= 0 ||
        stride <= 0 || pad < 0 || !Y)
        return 1;
    int64_t Ho = (H + 2 * pad - kh) / stride + 1, Wo = (W + 2 * pad - kw) / stride + 1;
    if (Ho <= 0 || Wo <= 0) return 1;
    int64_t Cm = C_in * cm;
    set_threads(threads);
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < batch; ++b)
        for (int64_t i = 0; i < Ho; ++i)
            for (int64_t j = 0; j < Wo; ++j)
                for (int64_t q = 0; q < C_in; ++q)
                    for (int64_t r = 0; r < cm; ++r) {
                        double acc = 0.0, sacc = 0.0;
                        for (int64_t di = 0; di < kh; ++di)
                            for (int64_t dj = 0; dj < kw; ++dj) {
                                int64_t y = stride * i + di - pad, xx = stride * j + dj - pad;
                                double xv = 0.0;
                                if (y >= 0 && y < H && xx >= 0 && xx < W)
                                    xv = ld_elem(x, dtype, ((b * H + y) * W + xx) * C_in + q);
                                double dv = ld_elem(dw, dtype, ((di * kw + dj) * C_in + q) * cm + r);
                                acc += xv * dv;
                                sacc += fabs(xv) * fabs(dv);
                            }
                        int64_t o = ((b * Ho + i) * Wo + j) * Cm + cm * q + r;
                        Y[o] = acc;
                        if (SY) SY[o] = sacc;
                    }
    return 0;
}

/*
 * Separable depthwise convolution, factored form (Section 2.3): the depthwise
 * result Y above, then the pointwise reduction over the intermediate channel
 * m = c*q + r,
 *
 *   Z[b][i][j][k] = sum_m Y[b][i][j][m] * P[m][k],   P is [C_in*c][C_out]
 *   S[b][i][j][k] = sum_m SY[b][i][j][m] * |P[m][k]|  (= sum of |X~||D||P| over all 8 indices)
 *
 * Y is not rounded between the two reductions.  Z, S are [batch][Ho][Wo][C_out].
 */
int isam_ref_dwsep(int64_t batch, int64_t H, int64_t W, int64_t C_in, int64_t cm,
                   int64_t kh, int64_t kw, int64_t stride, int64_t pad, int64_t C_out, int dtype,
                   const void* x, const void* dw, const void* pw, double* Z, double* S, int threads) {
    if (C_out <= 0 || !Z) return 1;
    int64_t Ho = (H + 2 * pad - kh) / stride + 1, Wo = (W + 2 * pad - kw) / stride + 1;
    if (batch < 0 || Ho <= 0 || Wo <= 0 || stride <= 0) return 1;
    int64_t Mp = batch * Ho * Wo, Cm = C_in * cm;
    double* Y = (double*)malloc(sizeof(double) * (size_t)(Mp * Cm > 0 ? Mp * Cm : 1));
    double* SY = S ? (double*)malloc(sizeof(double) * (size_t)(Mp * Cm > 0 ? Mp * Cm : 1)) : NULL;
    if (!Y || (S && !SY)) { free(Y); free(SY); return 2; }
    int rc = isam_ref_depthwise(batch, H, W, C_in, cm, kh, kw, stride, pad, dtype, x, dw, Y, SY, threads);
    if (rc == 0) {
        set_threads(threads);
#pragma omp parallel for schedule(static)
        for (int64_t p = 0; p < Mp; ++p)
            for (int64_t k = 0; k < C_out; ++k) {
                double acc = 0.0, sacc = 0.0;
                for (int64_t m = 0; m < Cm; ++m) {
                    double pv = ld_elem(pw, dtype, m * C_out + k);
                    acc += Y[p * Cm + m] * pv;
                    if (SY) sacc += SY[p * Cm + m] * fabs(pv);
                }
                Z[p * C_out + k] = acc;
                if (S) S[p * C_out + k] = sacc;
            }
    }
    free(Y);
    free(SY);
    return rc;
}

/*
 * Separable depthwise convolution, unfactored: the third listing's single sum
 * over (di, dj, q, r) of X~ * D * P for every output, with no intermediate
 * buffer.  Self-test only (it checks that the factoring of Section 2.3 does not
 * change the result beyond fp64 round-off).
 */
int isam_ref_dwsep_direct(int64_t batch, int64_t H, int64_t W, int64_t C_in, int64_t cm,
                          int64_t kh, int64_t kw, int64_t stride, int64_t pad, int64_t C_out,
                          int dtype, const void* x, const void* dw, const void* pw, double* Z) {
    if (!Z || stride <= 0) return 1;
    int64_t Ho = (H + 2 * pad - kh) / stride + 1, Wo = (W + 2 * pad - kw) / stride + 1;
    if (batch < 0 || Ho <= 0 || Wo <= 0) return 1;
    for (int64_t b = 0; b < batch; ++b)
        for (int64_t i = 0; i < Ho; ++i)
            for (int64_t j = 0; j < Wo; ++j)
                for (int64_t k = 0; k < C_out; ++k) {
                    double acc = 0.0;
                    for (int64_t di = 0; di < kh; ++di)
                        for (int64_t dj = 0; dj < kw; ++dj)
                            for (int64_t q = 0; q < C_in; ++q)
                                for (int64_t r = 0; r < cm; ++r) {
                                    int64_t y = stride * i + di - pad, xx = stride * j + dj - pad;
                                    if (y < 0 || y >= H || xx < 0 || xx >= W) continue;
                                    acc += ld_elem(x, dtype, ((b * H + y) * W + xx) * C_in + q) *
                                           ld_elem(dw, dtype, ((di * kw + dj) * C_in + q) * cm + r) *
                                           ld_elem(pw, dtype, (cm * q + r) * C_out + k);
                                }
                    Z[((b * Ho + i) * Wo + j) * C_out + k] = acc;
                }
    return 0;
}

static double sigmoid(double v) { return 1.0 / (1.0 + exp(-v)); }

/*
 * GRU forward over T steps.  The paper maps GRU cells onto matrix multiply plus
 * element-wise instructions (Section 6.1) and schedules the recurrence as
 * priming / recursive / finish iterations (Section 3.6); it does not print the
 * cell.  The cell used here is the standard one:
 *
 *   r   = sigmoid(W_r x_t + U_r h_{t-1} + b_r)
 *   z   = sigmoid(W_z x_t + U_z h_{t-1} + b_z)
 *   n   = tanh(W_n x_t + b_n + r * (U_n h_{t-1} + bhn))
 *   h_t = (1 - z) * n + z * h_{t-1}
 *
 * W is [3H][I] and U is [3H][H], gate blocks stacked r, z, n (rows g*H .. g*H+H-1).
 * x is [T][batch][I] (weight dtype), h0 is [batch][H] fp64 or NULL (zeros),
 * bias [3H] and bhn [H] are fp32 or NULL (zeros).  h_seq receives h_1 .. h_T
 * as [T][batch][H].  Each projection sums its index in ascending order; the
 * U_n h_{t-1} product is completed before it is multiplied by r.
 */
int isam_ref_gru(int64_t T, int64_t batch, int64_t I, int64_t H, int dtype,
                 const void* x, const double* h0, const void* W, const void* U,
                 const float* bias, const float* bhn, double* h_seq, int threads) {
    if (T < 0 || batch < 0 || I <= 0 || H <= 0 || !h_seq) return 1;
    if (T == 0 || batch == 0) return 0;
    double* h = (double*)malloc(sizeof(double) * (size_t)(batch * H));
    double* hn = (double*)malloc(sizeof(double) * (size_t)(batch * H));
    if (!h || !hn) { free(h); free(hn); return 2; }
    for (int64_t i = 0; i < batch * H; ++i) h[i] = h0 ? h0[i] : 0.0;
    set_threads(threads);
    for (int64_t t = 0; t < T; ++t) {
#pragma omp parallel for collapse(2) schedule(static)
        for (int64_t b = 0; b < batch; ++b)
            for (int64_t j = 0; j < H; ++j) {
                double gx[3], gh[3];
                for (int g = 0; g < 3; ++g) {
                    int64_t row = g * H + j;
                    double sx = 0.0, sh = 0.0;
                    for (int64_t k = 0; k < I; ++k)
                        sx += ld_elem(W, dtype, row * I + k) * ld_elem(x, dtype, (t * batch + b) * I + k);
                    for (int64_t k = 0; k < H; ++k)
                        sh += ld_elem(U, dtype, row * H + k) * h[b * H + k];
                    gx[g] = sx + (bias ? (double)bias[row] : 0.0);
                    gh[g] = sh;
                }
                double r = sigmoid(gx[0] + gh[0]);
                double z = sigmoid(gx[1] + gh[1]);
                double n = tanh(gx[2] + r * (gh[2] + (bhn ? (double)bhn[j] : 0.0)));
                hn[b * H + j] = (1.0 - z) * n + z * h[b * H + j];
            }
        memcpy(h, hn, sizeof(double) * (size_t)(batch * H));
        memcpy(h_seq + t * batch * H, h, sizeof(double) * (size_t)(batch * H));
    }
    free(h);
    free(hn);
    return 0;
}
