/*
 * Plain CPU oracle for the fused sparse direct convolution.
 *
 * TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the benchmark's
 * CPU-baseline leg may load or call this code. It shares nothing with the GPU
 * library: no headers, no helpers, no tables.
 *
 * What it computes (paper, "Optimizing Sparse Neural Networks", paragraph
 * "Sparse Convolution with CSR", together with the dense convolution of
 * "The Tiramisu Embedded DSL" and the Conv -> ReLU -> Maxpool block of the
 * "Evaluation" section):
 *
 *   pre[n,k,y,x] = b[k] + sum over nonzero taps (c,r,s) of row k of
 *                  W[k,c,r,s] * Xpad[n, c, y*stride + r, x*stride + s]
 *                  (+ res[n,k,y,x] when a residual is given)
 *   o            = relu ? max(pre, 0) : pre
 *   out          = pool ? max over a,b in {0,1} of o[n,k,2i+a,2j+b] : o
 *
 * Xpad is X surrounded by `pad` zeros; here the zero border is expressed as a
 * bounds test on the unpadded X, so the oracle never builds a padded copy.
 * Sums are taken in double precision, tap by tap in (c, r, s) order, which is
 * the order the paper's CSR loop visits the nonzeros of one output channel.
 * The oracle also returns, per output, the sum of |w * x| over the same terms
 * (the max of it over the pooling window when pooling), which bounds the
 * rounding error of any fp32 evaluation order.
 *
 * The residual is the shortcut of a ResNet basic block (the paper's ResNet
 * benchmark, "Evaluation"): the block input added to the second convolution's
 * pre-activation, before its ReLU. Its magnitude is added to the sum of
 * |w * x| of that output, since an fp32 evaluation rounds it too.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* An entry is a nonzero of the sparse filter: with a mask, every position whose
 * mask byte is nonzero (an explicit 0.0 value stays an entry); without one,
 * every value that compares unequal to 0.0f (so -0.0 is dropped, NaN is kept). */
static int oracle_is_entry(const float *w, const uint8_t *mask, size_t i) {
    if (mask) return mask[i] != 0;
    return w[i] != 0.0f;
}

/*
 * CSR packing of the filter (paper, "Sparse Convolution with CSR"): the
 * (K, C, R, S) tensor is viewed as a K x (C*R*S) matrix whose column is the
 * flattened tap (c, r, s); each row is compressed. Besides the column index,
 * every entry carries the tap's offset inside one zero-padded input image of
 * C planes of Hp x Wp, which is what the paper's loop adds to the output
 * position: offset = c*Hp*Wp + r*Wp + s.
 *
 * rowptr has K+1 slots; colidx, offset and vals need room for K*C*R*S entries.
 * Returns the number of entries.
 */
long long oracle_pack_csr(const float *w, const uint8_t *mask, int K, int C, int R, int S, int Hp, int Wp,
                          int32_t *rowptr, int32_t *colidx, int32_t *offset, float *vals) {
    long long nnz = 0;
    rowptr[0] = 0;
    for (int k = 0; k < K; ++k) {
        for (int c = 0; c < C; ++c)
            for (int r = 0; r < R; ++r)
                for (int s = 0; s < S; ++s) {
                    size_t i = (((size_t)k * C + c) * R + r) * S + s;
                    if (!oracle_is_entry(w, mask, i)) continue;
                    colidx[nnz] = (int32_t)((c * R + r) * S + s);
                    offset[nnz] = (int32_t)(c * Hp * Wp + r * Wp + s);
                    memcpy(&vals[nnz], &w[i], sizeof(float));
                    ++nnz;
                }
        rowptr[k + 1] = (int32_t)nnz;
    }
    return nnz;
}

/* Output extent of the convolution (before pooling). */
static int oracle_out_extent(int in, int f, int stride, int pad) {
    return (in + 2 * pad - f) / stride + 1;
}

/* One output plane (n, k): sums, activation and pooling as described above. */
static void oracle_plane(const float *x, int C, int H, int W, const float *w, const uint8_t *mask, int R, int S,
                         const float *bias, const float *res, int K, int stride, int pad, int relu, int pool, int n,
                         int k, double *acc, double *ab, double *out, double *absout) {
    const int Ho = oracle_out_extent(H, R, stride, pad);
    const int Wo = oracle_out_extent(W, S, stride, pad);
    const double b = bias ? (double)bias[k] : 0.0;
    for (int i = 0; i < Ho * Wo; ++i) {
        acc[i] = b;
        ab[i] = 0.0;
    }
    /* Walk the nonzeros of filter row k in (c, r, s) order. */
    for (int c = 0; c < C; ++c)
        for (int r = 0; r < R; ++r)
            for (int s = 0; s < S; ++s) {
                size_t wi = (((size_t)k * C + c) * R + r) * S + s;
                if (!oracle_is_entry(w, mask, wi)) continue;
                const double coeff = (double)w[wi];
                const float *plane = x + ((size_t)n * C + c) * H * W;
                for (int y = 0; y < Ho; ++y) {
                    const int iy = y * stride + r - pad;
                    for (int xo = 0; xo < Wo; ++xo) {
                        const int ix = xo * stride + s - pad;
                        double v = 0.0;
                        if (iy >= 0 && iy < H && ix >= 0 && ix < W) v = (double)plane[(size_t)iy * W + ix];
                        acc[y * Wo + xo] += coeff * v;
                        ab[y * Wo + xo] += fabs(coeff * v);
                    }
                }
            }
    if (res) {
        const float *rp = res + ((size_t)n * K + k) * Ho * Wo;
        for (int i = 0; i < Ho * Wo; ++i) {
            acc[i] += (double)rp[i];
            ab[i] += fabs((double)rp[i]);
        }
    }
    if (relu)
        for (int i = 0; i < Ho * Wo; ++i) acc[i] = acc[i] > 0.0 ? acc[i] : 0.0;
    if (!pool) {
        memcpy(out, acc, sizeof(double) * Ho * Wo);
        memcpy(absout, ab, sizeof(double) * Ho * Wo);
        return;
    }
    const int Hq = Ho / 2, Wq = Wo / 2;
    for (int i = 0; i < Hq; ++i)
        for (int j = 0; j < Wq; ++j) {
            double m = acc[(2 * i) * Wo + 2 * j];
            double a = ab[(2 * i) * Wo + 2 * j];
            for (int di = 0; di < 2; ++di)
                for (int dj = 0; dj < 2; ++dj) {
                    const double v = acc[(2 * i + di) * Wo + 2 * j + dj];
                    const double t = ab[(2 * i + di) * Wo + 2 * j + dj];
                    if (v > m) m = v;
                    if (t > a) a = t;
                }
            out[i * Wq + j] = m;
            absout[i * Wq + j] = a;
        }
}

/*
 * Fused sparse convolution over dense-stored sparse weights.
 *   x      [N][C][H][W] fp32 (unpadded)
 *   w      [K][C][R][S] fp32, mask same shape (nullable, see oracle_is_entry)
 *   bias   [K] (nullable = zero bias)
 *   res    [N][K][Ho][Wo] (nullable = no residual), on the convolution's own
 *          output grid (before pooling)
 *   pairs  nullable; if given, npairs (n, k) pairs, and out/absout hold one
 *          plane per pair in that order; otherwise all N*K planes, n-major.
 *   out, absout: double, plane size Ho*Wo, or (Ho/2)*(Wo/2) when pooling.
 *   nthreads: OpenMP threads (<= 0: the runtime default).
 * Returns 0, or -1 when the shapes give an empty output.
 */
int oracle_conv_res(const float *x, int N, int C, int H, int W, const float *w, const uint8_t *mask, int K, int R,
                    int S, const float *bias, const float *res, int stride, int pad, int relu, int pool,
                    const int32_t *pairs, int npairs, double *out, double *absout, int nthreads) {
    const int Ho = oracle_out_extent(H, R, stride, pad);
    const int Wo = oracle_out_extent(W, S, stride, pad);
    if (Ho < 1 || Wo < 1) return -1;
    const int Hq = pool ? Ho / 2 : Ho, Wq = pool ? Wo / 2 : Wo;
    const long long plane_out = (long long)Hq * Wq;
    const long long nplanes = pairs ? npairs : (long long)N * K;
#ifdef _OPENMP
    if (nthreads <= 0) nthreads = omp_get_max_threads();
#pragma omp parallel num_threads(nthreads)
#endif
    {
        double *acc = (double *)malloc(sizeof(double) * Ho * Wo);
        double *ab = (double *)malloc(sizeof(double) * Ho * Wo);
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
        for (long long p = 0; p < nplanes; ++p) {
            const int n = pairs ? pairs[2 * p] : (int)(p / K);
            const int k = pairs ? pairs[2 * p + 1] : (int)(p % K);
            oracle_plane(x, C, H, W, w, mask, R, S, bias, res, K, stride, pad, relu, pool, n, k, acc, ab,
                         out + p * plane_out, absout + p * plane_out);
        }
        free(acc);
        free(ab);
    }
    return 0;
}

/*
 * Bilinear resize of NCHW planes from Hin x Win to H x W (the "Resize" step of
 * the paper's Resize-Conv-ReLU-Maxpool block, "Evaluation"; the paper does not
 * give the interpolation mode, this reads it as bilinear with half-pixel
 * centres). Output pixel (y, x) samples the input at
 *   sy = (y + 1/2) * Hin / H - 1/2,   sx = (x + 1/2) * Win / W - 1/2,
 * clamped below at 0; with i0 = floor(s), i1 = min(i0 + 1, in - 1) and
 * t = s - i0 per axis, the value is
 *   (1-ty) * ((1-tx) v[i0y][i0x] + tx v[i0y][i1x]) + ty * ((1-tx) v[i1y][i0x] + tx v[i1y][i1x]).
 * The coordinates are taken as exact fractions (numerator (2y+1)*Hin - H over
 * 2H), the arithmetic in double. absout receives the sum of |weight * value|
 * of the four terms, which bounds the rounding of an fp32 evaluation.
 */
void oracle_resize_bilinear(const float *x, int N, int C, int Hin, int Win, int H, int W, double *out,
                            double *absout) {
    for (long long pl = 0; pl < (long long)N * C; ++pl) {
        const float *src = x + pl * Hin * Win;
        for (int y = 0; y < H; ++y) {
            long long ny = (2LL * y + 1) * Hin - H;   /* sy = ny / (2H) */
            if (ny < 0) ny = 0;
            const long long y0 = ny / (2LL * H);
            const long long y1 = y0 + 1 < Hin ? y0 + 1 : Hin - 1;
            const double ty = (double)(ny - y0 * 2LL * H) / (2.0 * H);
            for (int xo = 0; xo < W; ++xo) {
                long long nx = (2LL * xo + 1) * Win - W;
                if (nx < 0) nx = 0;
                const long long x0 = nx / (2LL * W);
                const long long x1 = x0 + 1 < Win ? x0 + 1 : Win - 1;
                const double tx = (double)(nx - x0 * 2LL * W) / (2.0 * W);
                const double v00 = src[y0 * Win + x0], v01 = src[y0 * Win + x1];
                const double v10 = src[y1 * Win + x0], v11 = src[y1 * Win + x1];
                const double w00 = (1 - ty) * (1 - tx), w01 = (1 - ty) * tx, w10 = ty * (1 - tx), w11 = ty * tx;
                const size_t o = (size_t)pl * H * W + (size_t)y * W + xo;
                out[o] = w00 * v00 + w01 * v01 + w10 * v10 + w11 * v11;
                absout[o] = fabs(w00 * v00) + fabs(w01 * v01) + fabs(w10 * v10) + fabs(w11 * v11);
            }
        }
    }
}

/* oracle_conv_res without a residual. */
int oracle_conv(const float *x, int N, int C, int H, int W, const float *w, const uint8_t *mask, int K, int R,
                int S, const float *bias, int stride, int pad, int relu, int pool, const int32_t *pairs,
                int npairs, double *out, double *absout, int nthreads) {
    return oracle_conv_res(x, N, C, H, W, w, mask, K, R, S, bias, NULL, stride, pad, relu, pool, pairs, npairs, out,
                           absout, nthreads);
}

/* Number of threads the OpenMP runtime would use by default. */
int oracle_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
