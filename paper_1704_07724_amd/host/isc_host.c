/* The paper's ISC on the host CPU (Sec. "Sparse Convolution"), for the
 * CPU speedup trend of Tab. 2: one image at a time, one core unless asked,
 * compiled for AVX2/FMA so that step 2's K-contiguous weight vectors are
 * multiplied 8 floats at a time.  Also the host im2col of Fig. 3, for the
 * dense baseline (im2col, then a BLAS GEMM on the host).
 *
 * Not on the GPU path: the library behind include/isc.h never calls this
 * code, and this code calls nothing of it.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* ISC step 2's kernel layout: wt[((c*R + r)*S + s)*K + k] = w[k][c][r][s]. */
void isc_host_repack(const float *w, int K, int C, int R, int S, float *wt) {
    const int64_t crs = (int64_t)C * R * S;
    for (int k = 0; k < K; ++k)
        for (int64_t q = 0; q < crs; ++q) wt[q * K + k] = w[(int64_t)k * crs + q];
}

/* acc[0 .. K) += v * wv[0 .. K) (vectorised by the compiler: 8 lanes). */
static inline void axpy(float *restrict acc, const float *restrict wv, float v, int K) {
    for (int k = 0; k < K; ++k) acc[k] += v * wv[k];
}

/* One image: x [C][H][W], y [K][Ho][Wo]; scratch: list (3 * H*W floats) and
 * the step-2 accumulator acc [Ho*Wo][K]. */
static void isc_image(const float *x, const float *wt, float *y, int C, int H, int W, int K, int R, int S, int T,
                      int P, int Ho, int Wo, float *list_v, int *list_y, int *list_x, float *acc) {
    memset(acc, 0, sizeof(float) * (size_t)Ho * Wo * K);
    for (int c = 0; c < C; ++c) {
        /* step 1: the plane's nonzero values with their row and column */
        const float *xp = x + (size_t)c * H * W;
        int n = 0;
        for (int iy = 0; iy < H; ++iy)
            for (int ix = 0; ix < W; ++ix) {
                const float v = xp[iy * W + ix];
                uint32_t bits;
                memcpy(&bits, &v, 4);
                if (bits & 0x7fffffffu) {
                    list_v[n] = v;
                    list_y[n] = iy;
                    list_x[n] = ix;
                    ++n;
                }
            }
        /* step 2: each nonzero times the K-contiguous weights of every tap
         * that reaches an output: output (oy, ox) = ((iy + P - r) / T,
         * (ix + P - s) / T) where both divide and land in range */
        const float *wc = wt + (size_t)c * R * S * K;
        for (int e = 0; e < n; ++e) {
            const float v = list_v[e];
            const int iy = list_y[e], ix = list_x[e];
            for (int r = 0; r < R; ++r) {
                const int ty = iy + P - r;
                if (ty < 0 || ty % T) continue;
                const int oy = ty / T;
                if (oy >= Ho) continue;
                for (int s = 0; s < S; ++s) {
                    const int tx = ix + P - s;
                    if (tx < 0 || tx % T) continue;
                    const int ox = tx / T;
                    if (ox >= Wo) continue;
                    axpy(acc + ((size_t)oy * Wo + ox) * K, wc + (size_t)(r * S + s) * K, v, K);
                }
            }
        }
    }
    /* step 3: the accumulator [position][k] transposed to [k][position] */
    const int hw = Ho * Wo;
    for (int p = 0; p < hw; ++p)
        for (int k = 0; k < K; ++k) y[(size_t)k * hw + p] = acc[(size_t)p * K + k];
}

/* y = conv(x, w) for N images by ISC, wt from isc_host_repack.  threads:
 * images spread over that many OpenMP threads (1: one core, as the paper
 * measures).  Returns 0, or -1 when scratch memory cannot be had. */
int isc_host_conv2d(const float *x, const float *wt, float *y, int N, int C, int H, int W, int K, int R, int S,
                    int T, int P, int threads) {
    const int Ho = (H + 2 * P - R) / T + 1, Wo = (W + 2 * P - S) / T + 1;
    if (threads < 1) threads = 1;
    int failed = 0;
#pragma omp parallel num_threads(threads)
    {
        float *list_v = (float *)malloc(sizeof(float) * (size_t)H * W);
        int *list_y = (int *)malloc(sizeof(int) * (size_t)H * W);
        int *list_x = (int *)malloc(sizeof(int) * (size_t)H * W);
        float *acc = (float *)aligned_alloc(64, ((sizeof(float) * (size_t)Ho * Wo * K) + 63) / 64 * 64);
        if (!list_v || !list_y || !list_x || !acc) {
#pragma omp atomic write
            failed = 1;
        } else {
#pragma omp for schedule(static)
            for (int n = 0; n < N; ++n)
                isc_image(x + (size_t)n * C * H * W, wt, y + (size_t)n * K * Ho * Wo, C, H, W, K, R, S, T, P, Ho, Wo,
                          list_v, list_y, list_x, acc);
        }
        free(list_v);
        free(list_y);
        free(list_x);
        free(acc);
    }
    return failed ? -1 : 0;
}

/* Fig. 3's input matrix for one image: col[(c*R + r)*S + s][oy*Wo + ox] =
 * x[c][oy*T + r - P][ox*T + s - P] (zero outside the input). */
void isc_host_im2col(const float *x, int C, int H, int W, int R, int S, int T, int P, float *col) {
    const int Ho = (H + 2 * P - R) / T + 1, Wo = (W + 2 * P - S) / T + 1;
    for (int c = 0; c < C; ++c)
        for (int r = 0; r < R; ++r)
            for (int s = 0; s < S; ++s) {
                float *row = col + ((size_t)(c * R + r) * S + s) * Ho * Wo;
                for (int oy = 0; oy < Ho; ++oy) {
                    const int iy = oy * T + r - P;
                    for (int ox = 0; ox < Wo; ++ox) {
                        const int ix = ox * T + s - P;
                        row[oy * Wo + ox] = (iy >= 0 && iy < H && ix >= 0 && ix < W) ? x[((size_t)c * H + iy) * W + ix] : 0.0f;
                    }
                }
            }
}
