/*
 * afno_oracle.c -- float64 CPU oracle for the AFNO spectral token-mixing filter.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or load
 * this file: only the tests, the smoke check and the benchmark's CPU-baseline leg
 * use it.  It shares no code, header, table or helper with the HIP library.
 *
 * What it computes (FourCastNet, section "Model Innovations": the three spatial
 * mixing steps -- an FFT over the token grid, a block-diagonal MLP applied per
 * token in Fourier space with weights shared by all tokens, an inverse FFT;
 * section "Implementation Details" (b) "Spectral convolution": real-to-complex /
 * complex-to-real transforms batched over batch and channels, complex weights
 * stored as real tensors with (re, im) as the fastest index, activations acting on
 * the real and imaginary parts independently).  Softshrink, the hard mode cutoff
 * and the residual come from the AFNO layer the paper builds on (its reference to
 * the Adaptive Fourier Neural Operator); their exact readings are listed in the
 * design notes and repeated at each function below.
 *
 * Everything is the plain definition, written out:
 *   - direct O(N^2) DFTs along W (real to half-complex) and along H (complex),
 *     "ortho" normalisation 1/sqrt(N) per axis, forward sign -, inverse sign +,
 *     twiddles cos/sin of 2*pi*((k*n) mod N)/N evaluated in double;
 *   - naive complex matrix products for the block MLP;
 *   - the complex-to-real inverse keeps only the real part of the kw=0 and
 *     kw=W/2 bins and weights every other bin twice (the half-spectrum form of
 *     the inverse real DFT).
 * Arrays are float64, row-major, complex values stored as (re, im) pairs.
 * Layouts:  x, out  [B][H][W][C];   spectra [B][H][Wm][C][2] with Wm = W/2+1;
 *           w1 [nb][bs][hs][2];  b1 [nb][hs][2];  w2 [nb][hs][bs][2];  b2 [nb][bs][2];
 *           hs = bs = C / nb.
 * Return value: 0 on success, -1 on an argument it does not accept.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifndef M_PI
#define M_PI 3.14159265358979323846
#endif

/* cos/sin of 2*pi*m/N for m in [0, N): the DFT kernel, evaluated in double. */
static double* unit_roots(long N) {
    double* t = (double*)malloc(sizeof(double) * 2 * (size_t)N);
    if (!t) return NULL;
    for (long m = 0; m < N; ++m) {
        double th = 2.0 * M_PI * (double)m / (double)N;
        t[2 * m] = cos(th);
        t[2 * m + 1] = sin(th);
    }
    return t;
}

/* Hard mode cutoff (reading of keep_fraction): per axis, on low |frequency|.
 * kept_h = floor((H/2+1) * keep), rows kept when |signed kh| < kept_h where the
 * signed index of kh is kh for kh <= H/2 and kh - H above;
 * kept_w = floor((W/2+1) * keep), columns kept when kw < kept_w.
 * The products are taken in double. */
void orc_keep_counts(long H, long W, double keep, long* kept_h, long* kept_w) {
    long Kh = H / 2 + 1, Wm = W / 2 + 1;
    *kept_h = (long)floor((double)Kh * keep);
    *kept_w = (long)floor((double)Wm * keep);
}

int orc_mode_kept(long kh, long kw, long H, long kept_h, long kept_w) {
    long s = (kh <= H / 2) ? kh : kh - H;
    if (s < 0) s = -s;
    return (s < kept_h) && (kw < kept_w);
}

/* Step 1, first axis: real-to-complex DFT along W of every (b, h, c) line.
 *   S1[b][h][kw][c] = (1/sqrt(W)) * sum_w x[b][h][w][c] * exp(-2*pi*i*kw*w/W),
 *   kw in [0, W/2]. */
int orc_dft_w_r2c(const double* x, long B, long H, long W, long C, double* S1) {
    if (B < 0 || H <= 0 || W <= 0 || C <= 0) return -1;
    long Wm = W / 2 + 1;
    double* t = unit_roots(W);
    if (!t) return -1;
    double sc = 1.0 / sqrt((double)W);
#pragma omp parallel for collapse(2) schedule(static)
    for (long b = 0; b < B; ++b)
        for (long h = 0; h < H; ++h) {
            const double* xr = x + ((size_t)b * H + h) * W * C;
            for (long kw = 0; kw < Wm; ++kw) {
                double* o = S1 + (((size_t)b * H + h) * Wm + kw) * C * 2;
                for (long c = 0; c < C; ++c) { o[2 * c] = 0.0; o[2 * c + 1] = 0.0; }
                for (long w = 0; w < W; ++w) {
                    long m = (kw * w) % W;
                    double cr = t[2 * m], si = t[2 * m + 1];  /* exp(-i th) = cr - i si */
                    const double* xv = xr + (size_t)w * C;
                    for (long c = 0; c < C; ++c) {
                        o[2 * c] += xv[c] * cr;
                        o[2 * c + 1] -= xv[c] * si;
                    }
                }
                for (long c = 0; c < 2 * C; ++c) o[c] *= sc;
            }
        }
    free(t);
    return 0;
}

/* Step 1, second axis (sign = -1) and step 3, first axis (sign = +1):
 * complex DFT along H of every (b, kw, c) line of a [B][H][Wm][C][2] array.
 *   out[b][k][kw][c] = (1/sqrt(H)) * sum_h in[b][h][kw][c] * exp(sign*2*pi*i*k*h/H). */
int orc_dft_h(const double* in, long B, long H, long Wm, long C, int sign, double* out) {
    if (B < 0 || H <= 0 || Wm <= 0 || C <= 0 || (sign != 1 && sign != -1)) return -1;
    double* t = unit_roots(H);
    if (!t) return -1;
    double sc = 1.0 / sqrt((double)H);
#pragma omp parallel for collapse(2) schedule(static)
    for (long b = 0; b < B; ++b)
        for (long k = 0; k < H; ++k) {
            for (long kw = 0; kw < Wm; ++kw) {
                double* o = out + (((size_t)b * H + k) * Wm + kw) * C * 2;
                for (long c = 0; c < 2 * C; ++c) o[c] = 0.0;
                for (long h = 0; h < H; ++h) {
                    long m = (k * h) % H;
                    double cr = t[2 * m], si = sign * t[2 * m + 1];  /* exp(sign i th) */
                    const double* v = in + (((size_t)b * H + h) * Wm + kw) * C * 2;
                    for (long c = 0; c < C; ++c) {
                        double vr = v[2 * c], vi = v[2 * c + 1];
                        o[2 * c] += vr * cr - vi * si;
                        o[2 * c + 1] += vr * si + vi * cr;
                    }
                }
                for (long c = 0; c < 2 * C; ++c) o[c] *= sc;
            }
        }
    free(t);
    return 0;
}

/* Step 3, second axis: complex-to-real inverse along W of a half spectrum.
 *   y[b][h][w][c] = (1/sqrt(W)) * sum_{kw=0}^{W/2} c_kw * Re(Y1[b][h][kw][c] * exp(+2*pi*i*kw*w/W)),
 *   c_kw = 1 for kw = 0 and (W even) kw = W/2, else 2.
 * The imaginary parts of the kw = 0 and kw = W/2 bins therefore do not contribute. */
int orc_dft_w_c2r(const double* Y1, long B, long H, long W, long C, double* y) {
    if (B < 0 || H <= 0 || W <= 0 || C <= 0) return -1;
    long Wm = W / 2 + 1;
    double* t = unit_roots(W);
    if (!t) return -1;
    double sc = 1.0 / sqrt((double)W);
#pragma omp parallel for collapse(2) schedule(static)
    for (long b = 0; b < B; ++b)
        for (long h = 0; h < H; ++h) {
            for (long w = 0; w < W; ++w) {
                double* o = y + (((size_t)b * H + h) * W + w) * C;
                for (long c = 0; c < C; ++c) o[c] = 0.0;
                for (long kw = 0; kw < Wm; ++kw) {
                    double ck = (kw == 0 || (W % 2 == 0 && kw == W / 2)) ? 1.0 : 2.0;
                    long m = (kw * w) % W;
                    double cr = t[2 * m], si = t[2 * m + 1];  /* exp(+i th) */
                    const double* v = Y1 + (((size_t)b * H + h) * Wm + kw) * C * 2;
                    for (long c = 0; c < C; ++c)
                        o[c] += ck * (v[2 * c] * cr - v[2 * c + 1] * si);
                }
                for (long c = 0; c < C; ++c) o[c] *= sc;
            }
        }
    free(t);
    return 0;
}

/* Step 2: the block-diagonal complex two-layer MLP applied to every mode, then
 * softshrink, then the hard mode cutoff.
 * For a kept mode (kh, kw) and block k, with X the mode's bs input channels of block k and
 * hs hidden units per block (w1 [nb][bs][hs], b1 [nb][hs], w2 [nb][hs][bs], b2 [nb][bs]):
 *   v[j] = b1[k][j] + sum_i X[i] * w1[k][i][j]          (true complex products)
 *   h[j] = ReLU(Re v[j]) + i * ReLU(Im v[j])            (parts independently)
 *   o[i] = b2[k][i] + sum_j h[j] * w2[k][j][i]
 *   Y[i] = S(Re o[i]) + i * S(Im o[i]),  S(v) = v - lam (v > lam), v + lam (v < -lam), else 0.
 * A mode outside the cutoff gets Y = 0. */
int orc_block_mlp_h(const double* X, const double* w1, const double* b1, const double* w2,
                    const double* b2, long B, long H, long Wm, long C, long nb, long hs,
                    double lam, long kept_h, long kept_w, double* Y) {
    if (B < 0 || H <= 0 || Wm <= 0 || C <= 0 || nb <= 0 || C % nb != 0 || hs <= 0) return -1;
    long bs = C / nb;
#pragma omp parallel
    {
        double* hid = (double*)malloc(sizeof(double) * 2 * (size_t)hs);
#pragma omp for collapse(2) schedule(static)
        for (long b = 0; b < B; ++b)
            for (long kh = 0; kh < H; ++kh) {
                for (long kw = 0; kw < Wm; ++kw) {
                    const double* xm = X + (((size_t)b * H + kh) * Wm + kw) * C * 2;
                    double* ym = Y + (((size_t)b * H + kh) * Wm + kw) * C * 2;
                    if (!orc_mode_kept(kh, kw, H, kept_h, kept_w)) {
                        for (long c = 0; c < 2 * C; ++c) ym[c] = 0.0;
                        continue;
                    }
                    for (long k = 0; k < nb; ++k) {
                        const double* xb = xm + (size_t)k * bs * 2;
                        const double* W1 = w1 + (size_t)k * bs * hs * 2;
                        const double* B1 = b1 + (size_t)k * hs * 2;
                        const double* W2 = w2 + (size_t)k * hs * bs * 2;
                        const double* B2 = b2 + (size_t)k * bs * 2;
                        for (long j = 0; j < hs; ++j) { hid[2 * j] = B1[2 * j]; hid[2 * j + 1] = B1[2 * j + 1]; }
                        for (long i = 0; i < bs; ++i) {
                            double xr = xb[2 * i], xi = xb[2 * i + 1];
                            const double* wr = W1 + (size_t)i * hs * 2;
                            for (long j = 0; j < hs; ++j) {
                                hid[2 * j] += xr * wr[2 * j] - xi * wr[2 * j + 1];
                                hid[2 * j + 1] += xr * wr[2 * j + 1] + xi * wr[2 * j];
                            }
                        }
                        for (long j = 0; j < 2 * hs; ++j) hid[j] = hid[j] > 0.0 ? hid[j] : 0.0;
                        double* yb = ym + (size_t)k * bs * 2;
                        for (long i = 0; i < bs; ++i) { yb[2 * i] = B2[2 * i]; yb[2 * i + 1] = B2[2 * i + 1]; }
                        for (long j = 0; j < hs; ++j) {
                            double hr = hid[2 * j], hi = hid[2 * j + 1];
                            const double* wr = W2 + (size_t)j * bs * 2;
                            for (long i = 0; i < bs; ++i) {
                                yb[2 * i] += hr * wr[2 * i] - hi * wr[2 * i + 1];
                                yb[2 * i + 1] += hr * wr[2 * i + 1] + hi * wr[2 * i];
                            }
                        }
                        for (long i = 0; i < 2 * bs; ++i) {
                            double v = yb[i];
                            yb[i] = v > lam ? v - lam : (v < -lam ? v + lam : 0.0);
                        }
                    }
                }
            }
        free(hid);
    }
    return 0;
}

/* The block MLP with hidden size equal to the block size. */
int orc_block_mlp(const double* X, const double* w1, const double* b1, const double* w2,
                  const double* b2, long B, long H, long Wm, long C, long nb, double lam,
                  long kept_h, long kept_w, double* Y) {
    if (nb <= 0 || C % nb != 0) return -1;
    return orc_block_mlp_h(X, w1, b1, w2, b2, B, H, Wm, C, nb, C / nb, lam, kept_h, kept_w, Y);
}

/* The whole filter: out = x + irfft2(MLP(rfft2(x))), axis order W then H forward,
 * H then W inverse.  Optional stage outputs (NULL to skip):
 *   spec_fwd [B][H][Wm][C][2]  the forward spectrum (after both axes);
 *   spec_mlp [B][H][Wm][C][2]  the spectrum after the MLP, softshrink and cutoff;
 *   delta    [B][H][W][C]      the filter output y = out - x before the residual add.
 * Samples are processed one at a time to bound memory. */
int orc_filter_forward_h(const double* x, const double* w1, const double* b1, const double* w2,
                         const double* b2, long B, long H, long W, long C, long nb, long hs,
                         double lam, double keep, double* out, double* spec_fwd,
                         double* spec_mlp, double* delta) {
    if (B < 0 || H <= 0 || W <= 0 || C <= 0 || nb <= 0 || C % nb != 0 || hs <= 0) return -1;
    if (!(lam >= 0.0) || !(keep > 0.0 && keep <= 1.0)) return -1;
    long Wm = W / 2 + 1, kept_h, kept_w;
    orc_keep_counts(H, W, keep, &kept_h, &kept_w);
    size_t nspec = (size_t)H * Wm * C * 2, nx = (size_t)H * W * C;
    double* s1 = (double*)malloc(sizeof(double) * nspec);
    double* s2 = (double*)malloc(sizeof(double) * nspec);
    double* y = (double*)malloc(sizeof(double) * nx);
    if (!s1 || !s2 || !y) { free(s1); free(s2); free(y); return -1; }
    int rc = 0;
    for (long b = 0; b < B && rc == 0; ++b) {
        const double* xb = x + (size_t)b * nx;
        rc |= orc_dft_w_r2c(xb, 1, H, W, C, s1);
        rc |= orc_dft_h(s1, 1, H, Wm, C, -1, s2);
        if (spec_fwd) memcpy(spec_fwd + (size_t)b * nspec, s2, sizeof(double) * nspec);
        rc |= orc_block_mlp_h(s2, w1, b1, w2, b2, 1, H, Wm, C, nb, hs, lam, kept_h, kept_w, s1);
        if (spec_mlp) memcpy(spec_mlp + (size_t)b * nspec, s1, sizeof(double) * nspec);
        rc |= orc_dft_h(s1, 1, H, Wm, C, +1, s2);
        rc |= orc_dft_w_c2r(s2, 1, H, W, C, y);
        if (delta) memcpy(delta + (size_t)b * nx, y, sizeof(double) * nx);
        double* ob = out + (size_t)b * nx;
        for (size_t i = 0; i < nx; ++i) ob[i] = xb[i] + y[i];
    }
    free(s1); free(s2); free(y);
    return rc;
}

/* The whole filter with hidden size equal to the block size. */
int orc_filter_forward(const double* x, const double* w1, const double* b1, const double* w2,
                       const double* b2, long B, long H, long W, long C, long nb, double lam,
                       double keep, double* out, double* spec_fwd, double* spec_mlp,
                       double* delta) {
    if (nb <= 0 || C % nb != 0) return -1;
    return orc_filter_forward_h(x, w1, b1, w2, b2, B, H, W, C, nb, C / nb, lam, keep, out,
                                spec_fwd, spec_mlp, delta);
}

/* Brute-force 2-D DFT of real input, one sum over all (h, w) per output bin
 * (no separation into axes); for cross-checking the separable sums on small grids.
 *   X[b][kh][kw][c] = (1/sqrt(H*W)) * sum_{h,w} x[b][h][w][c] * exp(-2*pi*i*(kh*h/H + kw*w/W)),
 *   kw in [0, W/2].  The phase is reduced as ((kh*h*W + kw*w*H) mod (H*W)) / (H*W). */
int orc_dft2_bruteforce(const double* x, long B, long H, long W, long C, double* X) {
    if (B < 0 || H <= 0 || W <= 0 || C <= 0) return -1;
    long Wm = W / 2 + 1, N = H * W;
    double sc = 1.0 / sqrt((double)N);
    for (long b = 0; b < B; ++b)
        for (long kh = 0; kh < H; ++kh)
            for (long kw = 0; kw < Wm; ++kw) {
                double* o = X + (((size_t)b * H + kh) * Wm + kw) * C * 2;
                for (long c = 0; c < 2 * C; ++c) o[c] = 0.0;
                for (long h = 0; h < H; ++h)
                    for (long w = 0; w < W; ++w) {
                        long m = (kh * h * W + kw * w * H) % N;
                        double th = 2.0 * M_PI * (double)m / (double)N;
                        double cr = cos(th), si = sin(th);
                        const double* xv = x + (((size_t)b * H + h) * W + w) * C;
                        for (long c = 0; c < C; ++c) {
                            o[2 * c] += xv[c] * cr;
                            o[2 * c + 1] -= xv[c] * si;
                        }
                    }
                for (long c = 0; c < 2 * C; ++c) o[c] *= sc;
            }
    return 0;
}

/* Brute-force inverse of a half spectrum, one sum over all (kh, kw) per output point:
 *   y[b][h][w][c] = (1/sqrt(H*W)) * sum_{kh, kw<=W/2} c_kw * Re(Y[b][kh][kw][c] * exp(+2*pi*i*(kh*h/H + kw*w/W))). */
int orc_idft2_bruteforce(const double* Y, long B, long H, long W, long C, double* y) {
    if (B < 0 || H <= 0 || W <= 0 || C <= 0) return -1;
    long Wm = W / 2 + 1, N = H * W;
    double sc = 1.0 / sqrt((double)N);
    for (long b = 0; b < B; ++b)
        for (long h = 0; h < H; ++h)
            for (long w = 0; w < W; ++w) {
                double* o = y + (((size_t)b * H + h) * W + w) * C;
                for (long c = 0; c < C; ++c) o[c] = 0.0;
                for (long kh = 0; kh < H; ++kh)
                    for (long kw = 0; kw < Wm; ++kw) {
                        double ck = (kw == 0 || (W % 2 == 0 && kw == W / 2)) ? 1.0 : 2.0;
                        long m = (kh * h * W + kw * w * H) % N;
                        double th = 2.0 * M_PI * (double)m / (double)N;
                        double cr = cos(th), si = sin(th);
                        const double* v = Y + (((size_t)b * H + kh) * Wm + kw) * C * 2;
                        for (long c = 0; c < C; ++c)
                            o[c] += ck * (v[2 * c] * cr - v[2 * c + 1] * si);
                    }
                for (long c = 0; c < C; ++c) o[c] *= sc;
            }
    return 0;
}

int orc_num_threads(void) {
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}
