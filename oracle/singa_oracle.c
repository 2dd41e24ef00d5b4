/*
 * singa_oracle.c -- plain fp64 CPU reference for the SINGA conv-training hot
 * path (arXiv 1603.07846).  TEST INFRASTRUCTURE ONLY: see singa_oracle.h.
 *
 * Every routine is the textbook definition, written output element by output
 * element.  Nothing is blocked, reordered or fused: a reader should be able
 * to check each loop against the formula in the header by eye.
 *
 * Build: gcc -O2 -fopenmp -fPIC -shared -o liboracle.so singa_oracle.c -lm
 */
#include "singa_oracle.h"

#include <math.h>
#include <stddef.h>
#include <string.h>

/* ------------------------------------------------------------------ sizes */

int64_t oracle_conv_out(int64_t in, int64_t k, int64_t pad, int64_t stride)
{
    /* floor division of a non-negative numerator (callers keep it >= 0) */
    return (in + 2 * pad - k) / stride + 1;
}

int64_t oracle_pool_out(int64_t in, int64_t k, int64_t pad, int64_t stride, int ceil_mode)
{
    int64_t span = in + 2 * pad - k;
    int64_t out;
    if (ceil_mode) {
        out = (span + stride - 1) / stride + 1;
        /* a last window that would start inside the right padding is dropped */
        if (pad > 0 && (out - 1) * stride >= in + pad)
            out -= 1;
    } else {
        out = span / stride + 1;
    }
    return out;
}

/* ------------------------------------------------------------ convolution */

/* y[n,k,p,q] (bias excluded) */
static double conv_fwd_elem(int64_t C, int64_t H, int64_t W, int64_t R, int64_t S,
                            int64_t ph, int64_t pw, int64_t sh, int64_t sw,
                            const double* x, const double* w,
                            int64_t n, int64_t k, int64_t p, int64_t q)
{
    double acc = 0.0;
    for (int64_t c = 0; c < C; ++c) {
        for (int64_t r = 0; r < R; ++r) {
            int64_t h = p * sh - ph + r;
            if (h < 0 || h >= H)
                continue;
            for (int64_t s = 0; s < S; ++s) {
                int64_t ww = q * sw - pw + s;
                if (ww < 0 || ww >= W)
                    continue;
                acc += w[((k * C + c) * R + r) * S + s] * x[((n * C + c) * H + h) * W + ww];
            }
        }
    }
    return acc;
}

/* dx[n,c,h,w] */
static double conv_bwd_data_elem(int64_t C, int64_t K,
                                 int64_t R, int64_t S, int64_t P, int64_t Q,
                                 int64_t ph, int64_t pw, int64_t sh, int64_t sw,
                                 const double* dy, const double* w,
                                 int64_t n, int64_t c, int64_t h, int64_t ww)
{
    double acc = 0.0;
    for (int64_t k = 0; k < K; ++k) {
        for (int64_t r = 0; r < R; ++r) {
            /* output row p reads input row h through tap r iff p*sh - ph + r == h */
            int64_t pnum = h + ph - r;
            if (pnum < 0 || pnum % sh != 0)
                continue;
            int64_t p = pnum / sh;
            if (p >= P)
                continue;
            for (int64_t s = 0; s < S; ++s) {
                int64_t qnum = ww + pw - s;
                if (qnum < 0 || qnum % sw != 0)
                    continue;
                int64_t q = qnum / sw;
                if (q >= Q)
                    continue;
                acc += w[((k * C + c) * R + r) * S + s] * dy[((n * K + k) * P + p) * Q + q];
            }
        }
    }
    return acc;
}

/* dw[k,c,r,s] */
static double conv_bwd_filter_elem(int64_t N, int64_t C, int64_t H, int64_t W, int64_t K,
                                   int64_t P, int64_t Q,
                                   int64_t ph, int64_t pw, int64_t sh, int64_t sw,
                                   const double* x, const double* dy,
                                   int64_t k, int64_t c, int64_t r, int64_t s)
{
    double acc = 0.0;
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t p = 0; p < P; ++p) {
            int64_t h = p * sh - ph + r;
            if (h < 0 || h >= H)
                continue;
            for (int64_t q = 0; q < Q; ++q) {
                int64_t ww = q * sw - pw + s;
                if (ww < 0 || ww >= W)
                    continue;
                acc += dy[((n * K + k) * P + p) * Q + q] * x[((n * C + c) * H + h) * W + ww];
            }
        }
    }
    return acc;
}

void oracle_conv_fwd(int64_t N, int64_t C, int64_t H, int64_t W,
                     int64_t K, int64_t R, int64_t S,
                     int64_t ph, int64_t pw, int64_t sh, int64_t sw,
                     const double* x, const double* w, const double* b, double* y)
{
    int64_t P = oracle_conv_out(H, R, ph, sh);
    int64_t Q = oracle_conv_out(W, S, pw, sw);
    int64_t total = N * K * P * Q;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < total; ++i) {
        int64_t q = i % Q, p = (i / Q) % P, k = (i / (Q * P)) % K, n = i / (Q * P * K);
        double v = conv_fwd_elem(C, H, W, R, S, ph, pw, sh, sw, x, w, n, k, p, q);
        y[i] = (b ? b[k] : 0.0) + v;
    }
}

void oracle_conv_bwd_data(int64_t N, int64_t C, int64_t H, int64_t W,
                          int64_t K, int64_t R, int64_t S,
                          int64_t ph, int64_t pw, int64_t sh, int64_t sw,
                          const double* dy, const double* w, double* dx)
{
    int64_t P = oracle_conv_out(H, R, ph, sh);
    int64_t Q = oracle_conv_out(W, S, pw, sw);
    int64_t total = N * C * H * W;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < total; ++i) {
        int64_t ww = i % W, h = (i / W) % H, c = (i / (W * H)) % C, n = i / (W * H * C);
        dx[i] = conv_bwd_data_elem(C, K, R, S, P, Q, ph, pw, sh, sw, dy, w, n, c, h, ww);
    }
}

void oracle_conv_bwd_filter(int64_t N, int64_t C, int64_t H, int64_t W,
                            int64_t K, int64_t R, int64_t S,
                            int64_t ph, int64_t pw, int64_t sh, int64_t sw,
                            const double* x, const double* dy, double* dw, double* db)
{
    int64_t P = oracle_conv_out(H, R, ph, sh);
    int64_t Q = oracle_conv_out(W, S, pw, sw);
    int64_t total = K * C * R * S;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < total; ++i) {
        int64_t s = i % S, r = (i / S) % R, c = (i / (S * R)) % C, k = i / (S * R * C);
        dw[i] = conv_bwd_filter_elem(N, C, H, W, K, P, Q, ph, pw, sh, sw, x, dy, k, c, r, s);
    }
    if (db) {
#pragma omp parallel for schedule(static)
        for (int64_t k = 0; k < K; ++k) {
            double acc = 0.0;
            for (int64_t n = 0; n < N; ++n)
                for (int64_t j = 0; j < P * Q; ++j)
                    acc += dy[(n * K + k) * P * Q + j];
            db[k] = acc;
        }
    }
}

void oracle_conv_fwd_points(int64_t N, int64_t C, int64_t H, int64_t W,
                            int64_t K, int64_t R, int64_t S,
                            int64_t ph, int64_t pw, int64_t sh, int64_t sw,
                            const double* x, const double* w, const double* b,
                            int64_t npts, const int64_t* idx, double* out)
{
    int64_t P = oracle_conv_out(H, R, ph, sh);
    int64_t Q = oracle_conv_out(W, S, pw, sw);
    (void)N;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < npts; ++t) {
        int64_t i = idx[t];
        int64_t q = i % Q, p = (i / Q) % P, k = (i / (Q * P)) % K, n = i / (Q * P * K);
        out[t] = (b ? b[k] : 0.0) + conv_fwd_elem(C, H, W, R, S, ph, pw, sh, sw, x, w, n, k, p, q);
    }
}

void oracle_conv_bwd_data_points(int64_t N, int64_t C, int64_t H, int64_t W,
                                 int64_t K, int64_t R, int64_t S,
                                 int64_t ph, int64_t pw, int64_t sh, int64_t sw,
                                 const double* dy, const double* w,
                                 int64_t npts, const int64_t* idx, double* out)
{
    int64_t P = oracle_conv_out(H, R, ph, sh);
    int64_t Q = oracle_conv_out(W, S, pw, sw);
    (void)N;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < npts; ++t) {
        int64_t i = idx[t];
        int64_t ww = i % W, h = (i / W) % H, c = (i / (W * H)) % C, n = i / (W * H * C);
        out[t] = conv_bwd_data_elem(C, K, R, S, P, Q, ph, pw, sh, sw, dy, w, n, c, h, ww);
    }
}

void oracle_conv_bwd_filter_points(int64_t N, int64_t C, int64_t H, int64_t W,
                                   int64_t K, int64_t R, int64_t S,
                                   int64_t ph, int64_t pw, int64_t sh, int64_t sw,
                                   const double* x, const double* dy,
                                   int64_t npts, const int64_t* idx, double* out)
{
    int64_t P = oracle_conv_out(H, R, ph, sh);
    int64_t Q = oracle_conv_out(W, S, pw, sw);
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t t = 0; t < npts; ++t) {
        int64_t i = idx[t];
        int64_t s = i % S, r = (i / S) % R, c = (i / (S * R)) % C, k = i / (S * R * C);
        out[t] = conv_bwd_filter_elem(N, C, H, W, K, P, Q, ph, pw, sh, sw, x, dy, k, c, r, s);
    }
}

/* ---------------------------------------------------------- inner product */

void oracle_fc_fwd(int64_t N, int64_t I, int64_t J,
                   const double* x, const double* w, const double* b, double* y)
{
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < N * J; ++t) {
        int64_t n = t / J, j = t % J;
        double acc = 0.0;
        for (int64_t i = 0; i < I; ++i)
            acc += x[n * I + i] * w[j * I + i];
        y[t] = (b ? b[j] : 0.0) + acc;
    }
}

void oracle_fc_bwd(int64_t N, int64_t I, int64_t J,
                   const double* x, const double* w, const double* dy,
                   double* dx, double* dw, double* db)
{
    /* dx[n,i] = sum_j dy[n,j] w[j,i] */
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < N * I; ++t) {
        int64_t n = t / I, i = t % I;
        double acc = 0.0;
        for (int64_t j = 0; j < J; ++j)
            acc += dy[n * J + j] * w[j * I + i];
        dx[t] = acc;
    }
    /* dw[j,i] = sum_n dy[n,j] x[n,i] */
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < J * I; ++t) {
        int64_t j = t / I, i = t % I;
        double acc = 0.0;
        for (int64_t n = 0; n < N; ++n)
            acc += dy[n * J + j] * x[n * I + i];
        dw[t] = acc;
    }
    if (db) {
        for (int64_t j = 0; j < J; ++j) {
            double acc = 0.0;
            for (int64_t n = 0; n < N; ++n)
                acc += dy[n * J + j];
            db[j] = acc;
        }
    }
}

/* ---------------------------------------------------------------- pooling */

/* Window o = (p, q) covers rows [p*sh - ph, p*sh - ph + kh) and likewise for
 * columns.  The averaging divisor counts the window after clipping it to the
 * padded extent [-ph, H + ph); the sum runs over the in-bounds cells. */
static int64_t pool_divisor(int64_t H, int64_t W, int64_t kh, int64_t kw,
                            int64_t sh, int64_t sw, int64_t ph, int64_t pw,
                            int64_t p, int64_t q)
{
    int64_t h0 = p * sh - ph, w0 = q * sw - pw;
    int64_t h1 = h0 + kh, w1 = w0 + kw;
    if (h1 > H + ph) h1 = H + ph;
    if (w1 > W + pw) w1 = W + pw;
    return (h1 - h0) * (w1 - w0);
}

void oracle_pool_fwd(int mode, int64_t N, int64_t C, int64_t H, int64_t W,
                     int64_t kh, int64_t kw, int64_t sh, int64_t sw,
                     int64_t ph, int64_t pw, int ceil_mode,
                     const double* x, double* y, uint8_t* argmax)
{
    int64_t P = oracle_pool_out(H, kh, ph, sh, ceil_mode);
    int64_t Q = oracle_pool_out(W, kw, pw, sw, ceil_mode);
    int64_t total = N * C * P * Q;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < total; ++i) {
        int64_t q = i % Q, p = (i / Q) % P, nc = i / (Q * P);
        const double* plane = x + nc * H * W;
        int64_t h0 = p * sh - ph, w0 = q * sw - pw;
        if (mode == 0) {
            int found = 0;
            double best = 0.0;
            int64_t best_cell = 0;
            for (int64_t r = 0; r < kh; ++r) {
                int64_t h = h0 + r;
                if (h < 0 || h >= H)
                    continue;
                for (int64_t s = 0; s < kw; ++s) {
                    int64_t ww = w0 + s;
                    if (ww < 0 || ww >= W)
                        continue;
                    double v = plane[h * W + ww];
                    if (!found || v > best) {
                        best = v;
                        best_cell = r * kw + s;
                        found = 1;
                    }
                }
            }
            y[i] = best;
            if (argmax)
                argmax[i] = (uint8_t)best_cell;
        } else {
            double acc = 0.0;
            for (int64_t r = 0; r < kh; ++r) {
                int64_t h = h0 + r;
                if (h < 0 || h >= H)
                    continue;
                for (int64_t s = 0; s < kw; ++s) {
                    int64_t ww = w0 + s;
                    if (ww < 0 || ww >= W)
                        continue;
                    acc += plane[h * W + ww];
                }
            }
            y[i] = acc / (double)pool_divisor(H, W, kh, kw, sh, sw, ph, pw, p, q);
        }
    }
}

void oracle_pool_bwd(int mode, int64_t N, int64_t C, int64_t H, int64_t W,
                     int64_t kh, int64_t kw, int64_t sh, int64_t sw,
                     int64_t ph, int64_t pw, int ceil_mode,
                     const double* dy, const uint8_t* argmax, double* dx)
{
    int64_t P = oracle_pool_out(H, kh, ph, sh, ceil_mode);
    int64_t Q = oracle_pool_out(W, kw, pw, sw, ceil_mode);
    /* one (n, c) plane per iteration; windows of a plane are visited in order
     * and scatter their gradient, so the sum order is fixed */
#pragma omp parallel for schedule(static)
    for (int64_t nc = 0; nc < N * C; ++nc) {
        double* dplane = dx + nc * H * W;
        memset(dplane, 0, sizeof(double) * (size_t)(H * W));
        for (int64_t p = 0; p < P; ++p) {
            for (int64_t q = 0; q < Q; ++q) {
                int64_t o = (nc * P + p) * Q + q;
                int64_t h0 = p * sh - ph, w0 = q * sw - pw;
                if (mode == 0) {
                    int64_t cell = argmax[o];
                    int64_t h = h0 + cell / kw, ww = w0 + cell % kw;
                    dplane[h * W + ww] += dy[o];
                } else {
                    double g = dy[o] / (double)pool_divisor(H, W, kh, kw, sh, sw, ph, pw, p, q);
                    for (int64_t r = 0; r < kh; ++r) {
                        int64_t h = h0 + r;
                        if (h < 0 || h >= H)
                            continue;
                        for (int64_t s = 0; s < kw; ++s) {
                            int64_t ww = w0 + s;
                            if (ww < 0 || ww >= W)
                                continue;
                            dplane[h * W + ww] += g;
                        }
                    }
                }
            }
        }
    }
}

/* ------------------------------------------------------------------- ReLU */

void oracle_relu_fwd(int64_t n, const double* x, double* y)
{
    for (int64_t i = 0; i < n; ++i)
        y[i] = x[i] > 0.0 ? x[i] : 0.0;
}

void oracle_relu_bwd(int64_t n, const double* y, const double* dy, double* dx)
{
    for (int64_t i = 0; i < n; ++i)
        dx[i] = y[i] > 0.0 ? dy[i] : 0.0;
}

/* ------------------------------------------------- local response norm */

/* Channels c' of the window around c: |c' - c| <= size / 2, inside [0, C). */
static double lrn_scale(const double* x, int64_t C, int64_t HW, int64_t c, int64_t size,
                        double alpha, double k)
{
    int64_t lo = c - size / 2, hi = c + (size - 1) / 2;
    double s = 0.0;
    if (lo < 0) lo = 0;
    if (hi > C - 1) hi = C - 1;
    for (int64_t j = lo; j <= hi; ++j) {
        double v = x[j * HW];
        s += v * v;
    }
    return k + alpha / (double)size * s;
}

void oracle_lrn_fwd(int64_t N, int64_t C, int64_t H, int64_t W, const double* x,
                    int64_t size, double alpha, double beta, double k, double* y)
{
    const int64_t HW = H * W;
    #pragma omp parallel for collapse(2) schedule(static)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t c = 0; c < C; ++c)
            for (int64_t p = 0; p < HW; ++p) {
                const double* xp = x + n * C * HW + p;
                double sc = lrn_scale(xp, C, HW, c, size, alpha, k);
                y[(n * C + c) * HW + p] = xp[c * HW] * pow(sc, -beta);
            }
}

/* dx[c] = dy[c] s[c]^-beta - (2 alpha beta / size) x[c]
 *         * sum over the channels j whose window holds c of dy[j] x[j] s[j]^(-beta-1),
 * the derivative of y[j] = x[j] s[j]^-beta, s[j] = k + alpha/size sum_{i in window(j)} x[i]^2. */
void oracle_lrn_bwd(int64_t N, int64_t C, int64_t H, int64_t W, const double* x, const double* dy,
                    int64_t size, double alpha, double beta, double k, double* dx)
{
    const int64_t HW = H * W;
    #pragma omp parallel for collapse(2) schedule(static)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t c = 0; c < C; ++c)
            for (int64_t p = 0; p < HW; ++p) {
                const double* xp = x + n * C * HW + p;
                const double* dyp = dy + n * C * HW + p;
                double sc = lrn_scale(xp, C, HW, c, size, alpha, k);
                double acc = 0.0;
                /* j's window holds c when j - size/2 <= c <= j + (size-1)/2 */
                int64_t lo = c - (size - 1) / 2, hi = c + size / 2;
                if (lo < 0) lo = 0;
                if (hi > C - 1) hi = C - 1;
                for (int64_t j = lo; j <= hi; ++j) {
                    double sj = lrn_scale(xp, C, HW, j, size, alpha, k);
                    acc += dyp[j * HW] * xp[j * HW] * pow(sj, -beta - 1.0);
                }
                dx[(n * C + c) * HW + p] = dyp[c * HW] * pow(sc, -beta)
                                           - 2.0 * alpha * beta / (double)size * xp[c * HW] * acc;
            }
}

/* ------------------------------------------------------ softmax + x-entropy */

double oracle_softmax_ce(int64_t B, int64_t classes, const double* z,
                         const int32_t* label, double* dz)
{
    double total = 0.0;
    for (int64_t n = 0; n < B; ++n) {
        const double* row = z + n * classes;
        double m = row[0];
        for (int64_t j = 1; j < classes; ++j)
            if (row[j] > m)
                m = row[j];
        double sum = 0.0;
        for (int64_t j = 0; j < classes; ++j)
            sum += exp(row[j] - m);
        double lse = m + log(sum);
        total += lse - row[label[n]];
        for (int64_t j = 0; j < classes; ++j) {
            double prob = exp(row[j] - lse);
            dz[n * classes + j] = (prob - (j == label[n] ? 1.0 : 0.0)) / (double)B;
        }
    }
    return total / (double)B;
}

/* ---------------------------------------------------- bf16 storage rounding */

void oracle_round_bf16(int64_t n, double* x)
{
    for (int64_t i = 0; i < n; ++i) {
        float f = (float)x[i]; /* C's conversion rounds to nearest even */
        uint32_t u;
        memcpy(&u, &f, sizeof u);
        if ((u & 0x7fffffffu) > 0x7f800000u) { /* NaN stays NaN */
            x[i] = (double)f;
            continue;
        }
        /* keep the upper 16 bits, rounding the lower 16 to nearest, ties to even */
        uint32_t lower = u & 0xffffu;
        uint32_t upper = u >> 16;
        if (lower > 0x8000u || (lower == 0x8000u && (upper & 1u)))
            upper += 1u;
        u = upper << 16;
        memcpy(&f, &u, sizeof f);
        x[i] = (double)f;
    }
}

/* ---------------------------------------------------------------- updater */

void oracle_sgd_momentum(int64_t n, double* w, const double* g, double* v,
                         double lr, double momentum, double wd)
{
    for (int64_t i = 0; i < n; ++i) {
        double gi = g[i] + wd * w[i];
        v[i] = momentum * v[i] + lr * gi;
        w[i] = w[i] - v[i];
    }
}

/* AdaGrad (Duchi, Hazan and Singer, JMLR 2011), the diagonal form: the
 * squared gradients accumulate per parameter, and the step divides the
 * learning rate by delta plus the square root of that sum. */
void oracle_adagrad(int64_t n, double* w, const double* g, double* h,
                    double lr, double delta, double wd)
{
    for (int64_t i = 0; i < n; ++i) {
        double gi = g[i] + wd * w[i];
        h[i] = h[i] + gi * gi;
        w[i] = w[i] - lr * gi / (delta + sqrt(h[i]));
    }
}
