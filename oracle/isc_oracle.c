/*
 * isc_oracle.c -- CPU reference ("oracle") for the sparse-input convolution.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file: only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark use it.  It shares no source, header, table or helper with
 * the HIP library; every definition below is written out from the paper
 * (Shi & Chu, "Speeding up Convolutional Neural Networks By Exploiting the
 * Sparsity of Rectifier Units", arXiv 1704.07724) in plain C, slow and
 * obviously correct, accumulating in fp64.
 *
 * Notation follows the paper's parameter table ("Parameters of Convolution",
 * Tab. 1): C input maps of H x W, K output maps, R x S filters, padding P,
 * stride T.  Batch N is the leading dimension of the input and output.
 *
 * Readings of the paper (each one is listed in the design notes):
 *   - output size: Ho = floor((H + 2P - R) / T) + 1 (the printed formula
 *     (H + 2P - R + 1) / T is not an integer for T > 1; both agree at T = 1);
 *   - Eq. 1 extended to batch, stride and zero padding, cross-correlation
 *     (no filter flip, as the i + r index in Eq. 1 shows);
 *   - a value counts as zero iff its bit pattern with the sign cleared is
 *     all zero (+0 and -0 are zero; denormals, Inf and NaN are not);
 *   - the nonzero "vector with column and row information" (Sec. "Sparse
 *     Convolution", ISC step 1) lists the nonzeros of each (n, c) plane in
 *     row-major order, so the list is unique.
 *
 * Build: gcc -O2 -fopenmp -shared -fPIC isc_oracle.c -o liboracle.so
 */
#include <stdint.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Threads the parallel loops below use (for reporting CPU-baseline runs). */
int oracle_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Set the thread count of the parallel loops (n >= 1); timing only. */
void oracle_set_threads(int n)
{
#ifdef _OPENMP
    if (n >= 1)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Output extent along one axis: floor((in + 2*pad - k) / stride) + 1, or 0
 * when the padded input is shorter than the filter. */
int oracle_out_size(int in, int k, int pad, int stride)
{
    long num = (long)in + 2L * pad - k;
    if (stride < 1 || num < 0) return 0;
    return (int)(num / stride) + 1;
}

/* The zero test of ISC step 1, on the bit pattern so that it does not depend
 * on any floating-point mode. */
static int oracle_is_nonzero(float v)
{
    uint32_t b;
    memcpy(&b, &v, sizeof b);
    return (b & 0x7fffffffu) != 0u;
}

/* Input value with zero padding: X^[n, c, y, x] = X[n, c, y, x] inside the
 * H x W map, 0 outside. */
static double oracle_xhat(const float *x, long n, long c, long y, long xx,
                          int C, int H, int W)
{
    if (y < 0 || y >= H || xx < 0 || xx >= W) return 0.0;
    return (double)x[((n * C + c) * H + y) * W + xx];
}

/* One output element of Eq. 1 (Sec. "Sparsity of ReLUs"), extended with
 * batch, stride and padding:
 *   O[n,k,i,j] = sum_c sum_r sum_s W[k,c,r,s] * X^[n, c, i*T + r - P, j*T + s - P]
 * Each fp32 x fp32 product is exact in fp64; products are summed in fp64 in
 * (c, r, s) order. */
static double oracle_conv_point(const float *x, const float *w,
                                long n, long k, long i, long j,
                                int C, int H, int W, int R, int S, int T, int P)
{
    double acc = 0.0;
    for (long c = 0; c < C; ++c)
        for (long r = 0; r < R; ++r)
            for (long s = 0; s < S; ++s) {
                double xv = oracle_xhat(x, n, c, i * T + r - P, j * T + s - P, C, H, W);
                double wv = (double)w[((k * C + c) * R + r) * S + s];
                acc += wv * xv;
            }
    return acc;
}

/* Full direct convolution, output N x K x Ho x Wo in fp64.  Parallel over
 * (n, k) only; each output element is computed by oracle_conv_point. */
void oracle_conv2d_f64(const float *x, const float *w,
                       int N, int C, int H, int W, int K, int R, int S,
                       int T, int P, double *out)
{
    const int Ho = oracle_out_size(H, R, P, T);
    const int Wo = oracle_out_size(W, S, P, T);
    const long NK = (long)N * K;
#pragma omp parallel for schedule(dynamic, 1)
    for (long nk = 0; nk < NK; ++nk) {
        const long n = nk / K, k = nk % K;
        for (long i = 0; i < Ho; ++i)
            for (long j = 0; j < Wo; ++j)
                out[((n * K + k) * Ho + i) * Wo + j] =
                    oracle_conv_point(x, w, n, k, i, j, C, H, W, R, S, T, P);
    }
}

/* The same definition evaluated only at the listed flat output indices
 * (index = ((n*K + k)*Ho + i)*Wo + j), for spot checks at full size. */
void oracle_conv2d_f64_at(const float *x, const float *w,
                          int N, int C, int H, int W, int K, int R, int S,
                          int T, int P, const int64_t *idx, int64_t count,
                          double *out)
{
    const long Ho = oracle_out_size(H, R, P, T);
    const long Wo = oracle_out_size(W, S, P, T);
    (void)N;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < count; ++t) {
        long f = (long)idx[t];
        const long j = f % Wo; f /= Wo;
        const long i = f % Ho; f /= Ho;
        const long k = f % K;
        const long n = f / K;
        out[t] = oracle_conv_point(x, w, n, k, i, j, C, H, W, R, S, T, P);
    }
}

/* ISC step 1 (Sec. "Sparse Convolution"): for every (n, c) plane, list the
 * nonzero inputs with their row and column, row-major.
 *   row_ptr[(n*C + c)*(H+1) + y] = number of nonzeros of the plane in rows < y
 *   (so row_ptr[... + H] is the plane's count);
 *   entry e of plane p is stored at slot p*H*W + e: value bits in v[],
 *   row in ys[], column in xs[].
 * Returns the total number of nonzeros. */
int64_t oracle_compact(const float *x, int N, int C, int H, int W,
                       int32_t *row_ptr, float *v, int32_t *ys, int32_t *xs)
{
    int64_t total = 0;
    const long planes = (long)N * C;
    const long HW = (long)H * W;
    for (long p = 0; p < planes; ++p) {
        int32_t cnt = 0;
        for (long y = 0; y < H; ++y) {
            row_ptr[p * (H + 1) + y] = cnt;
            for (long xx = 0; xx < W; ++xx) {
                float val = x[p * HW + y * W + xx];
                if (oracle_is_nonzero(val)) {
                    memcpy(&v[p * HW + cnt], &val, sizeof val);
                    ys[p * HW + cnt] = (int32_t)y;
                    xs[p * HW + cnt] = (int32_t)xx;
                    ++cnt;
                }
            }
        }
        row_ptr[p * (H + 1) + H] = cnt;
        total += cnt;
    }
    return total;
}

/* Number of output taps one input coordinate u (along an axis with filter
 * size k, padding pad, stride t and output extent out) contributes to: the
 * filter offsets q in [0, k) with u + pad - q divisible by t and
 * 0 <= (u + pad - q)/t < out.  Counted by enumeration. */
static long oracle_taps_1d(long u, int k, int pad, int t, int out)
{
    long cnt = 0;
    for (long q = 0; q < k; ++q) {
        long num = u + pad - q;
        if (num < 0 || num % t != 0) continue;
        if (num / t < out) ++cnt;
    }
    return cnt;
}

/* Exact nonzero multiply-accumulate count of the zero-skipping convolution
 * (the paper's rho * Ho*Wo*R*S*K*C of Sec. "Sparse Convolution" without the
 * approximation at the borders): the sum over nonzero inputs of K times the
 * number of (r, s) taps that land on a valid output. */
int64_t oracle_nz_macs(const float *x, int N, int C, int H, int W,
                       int K, int R, int S, int T, int P)
{
    const int Ho = oracle_out_size(H, R, P, T);
    const int Wo = oracle_out_size(W, S, P, T);
    int64_t macs = 0;
    for (long p = 0; p < (long)N * C; ++p)
        for (long y = 0; y < H; ++y)
            for (long xx = 0; xx < W; ++xx)
                if (oracle_is_nonzero(x[(p * H + y) * W + xx]))
                    macs += (int64_t)K * oracle_taps_1d(y, R, P, T, Ho)
                                       * oracle_taps_1d(xx, S, P, T, Wo);
    return macs;
}

/* The unrolled input matrix M_I of the matrix-multiplication formulation
 * (Sec. "Sparse Convolution", Fig. 3), extended with batch as extra columns:
 *   col[(c*R + r)*S + s][(n*Ho + i)*Wo + j] = X^[n, c, i*T + r - P, j*T + s - P]
 * with row length ldc >= N*Ho*Wo; entries past N*Ho*Wo are left untouched. */
void oracle_im2col(const float *x, int N, int C, int H, int W, int R, int S,
                   int T, int P, int64_t ldc, float *col)
{
    const long Ho = oracle_out_size(H, R, P, T);
    const long Wo = oracle_out_size(W, S, P, T);
    for (long c = 0; c < C; ++c)
        for (long r = 0; r < R; ++r)
            for (long s = 0; s < S; ++s) {
                const long row = (c * R + r) * S + s;
                for (long n = 0; n < N; ++n)
                    for (long i = 0; i < Ho; ++i)
                        for (long j = 0; j < Wo; ++j) {
                            long y = i * T + r - P, xx = j * T + s - P;
                            float val = 0.0f;
                            if (y >= 0 && y < H && xx >= 0 && xx < W)
                                val = x[((n * C + c) * H + y) * W + xx];
                            col[row * ldc + (n * Ho + i) * Wo + j] = val;
                        }
            }
}

/* The rectifier of Eq. 2 (Sec. "Sparsity of ReLUs"), f(v) = max(0, v),
 * applied in place to n entries of an fp64 convolution output; returns how
 * many entries are nonzero afterwards -- the nonzero count of the next
 * layer's input, from which its sparsity 1 - rho follows. */
int64_t oracle_rectify_f64(double *y, int64_t n)
{
    int64_t nnz = 0;
    for (int64_t i = 0; i < n; ++i) {
        if (y[i] > 0.0)
            ++nnz;
        else
            y[i] = 0.0;
    }
    return nnz;
}

/* Weight gradient of Eq. 1 for training (the paper measures the sparsity of
 * the rectified inputs during training, Sec. "Sparsity of ReLUs"): with
 * dy = dLoss/dO of shape N x K x Ho x Wo,
 *   dw[k,c,r,s] = sum_{n,i,j} dy[n,k,i,j] * X^[n, c, i*T + r - P, j*T + s - P]
 * (X^ = x inside the map, 0 outside), fp64 accumulation in (n, i, j) order.
 * dw is K x C x R x S. */
void oracle_conv2d_dw_f64(const float *x, const float *dy, int N, int C, int H, int W,
                          int K, int R, int S, int T, int P, double *dw)
{
    const long Ho = oracle_out_size(H, R, P, T);
    const long Wo = oracle_out_size(W, S, P, T);
    #pragma omp parallel for collapse(2) schedule(static)
    for (long k = 0; k < K; ++k)
        for (long c = 0; c < C; ++c)
            for (long r = 0; r < R; ++r)
                for (long s = 0; s < S; ++s) {
                    double acc = 0.0;
                    for (long n = 0; n < N; ++n)
                        for (long i = 0; i < Ho; ++i)
                            for (long j = 0; j < Wo; ++j) {
                                double xv = oracle_xhat(x, n, c, i * T + r - P, j * T + s - P, C, H, W);
                                acc += (double)dy[((n * K + k) * Ho + i) * Wo + j] * xv;
                            }
                    dw[((k * C + c) * R + r) * S + s] = acc;
                }
}
