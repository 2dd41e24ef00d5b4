/*
 * singa_oracle.h -- CPU reference ("oracle") for the SINGA conv-training hot
 * path (Wang et al., "Deep Learning At Scale and At Ease", arXiv 1603.07846).
 *
 * TEST INFRASTRUCTURE ONLY.  This library is the plain, slow, obviously
 * correct definition that the GPU library is checked against.  It shares no
 * code, header, table or helper with the GPU path, and the product never
 * links or calls it: only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg do.
 *
 * Conventions
 *   - Every tensor is a dense host array of double (fp64), C order.
 *   - Activations are NCHW, filters are KCRS (Caffe order, which SINGA adopts
 *     for its convolution and pooling code, Sec. 6.2.1).
 *   - Each routine evaluates the plain definition output element by output
 *     element, accumulating in fp64 in a fixed loop order.  OpenMP splits the
 *     outer output loop only, so results do not depend on the thread count.
 *   - Sizes are int64; the caller passes consistent sizes (no validation:
 *     the oracle trusts its test harness).
 *
 * Parity status: every routine is pinned by the CPU tests (hand-worked
 * examples, brute-force operator matrices, adjoint identities, finite
 * differences, closed forms and library routines).  The avg-pool divisor on
 * clipped ceil-mode edge windows, where the paper says nothing, follows
 * Caffe's pooling and is pinned by the same rule in torch's avg_pool2d.
 */
#ifndef SINGA_ORACLE_H
#define SINGA_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Output extent of a convolution along one axis: floor((H + 2*pad - R)/stride) + 1. */
int64_t oracle_conv_out(int64_t in, int64_t k, int64_t pad, int64_t stride);

/* Output extent of a pooling window along one axis.  ceil_mode != 0 takes
 * ceil((H + 2*pad - k)/stride) + 1 and drops a last window that would start
 * inside the right padding; ceil_mode == 0 takes the floor. */
int64_t oracle_pool_out(int64_t in, int64_t k, int64_t pad, int64_t stride, int ceil_mode);

/* Convolution layer ComputeFeature (Sec. 4.1.2), cross-correlation:
 *   y[n,k,p,q] = b[k] + sum_{c,r,s} w[k,c,r,s] * x[n,c,p*sh-ph+r, q*sw-pw+s]
 * where taps outside the input read zero.  b may be NULL (no bias).
 * x: N*C*H*W, w: K*C*R*S, y: N*K*P*Q. */
void oracle_conv_fwd(int64_t N, int64_t C, int64_t H, int64_t W,
                     int64_t K, int64_t R, int64_t S,
                     int64_t ph, int64_t pw, int64_t sh, int64_t sw,
                     const double* x, const double* w, const double* b, double* y);

/* Convolution layer ComputeGradient, gradient of the source layer (Sec. 4.1.2):
 *   dx[n,c,h,w] = sum over (k,r,s,p,q) with p*sh-ph+r = h and q*sw-pw+s = w
 *                 of w[k,c,r,s] * dy[n,k,p,q]
 * dy: N*K*P*Q, w: K*C*R*S, dx: N*C*H*W (overwritten). */
void oracle_conv_bwd_data(int64_t N, int64_t C, int64_t H, int64_t W,
                          int64_t K, int64_t R, int64_t S,
                          int64_t ph, int64_t pw, int64_t sh, int64_t sw,
                          const double* dy, const double* w, double* dx);

/* Convolution layer ComputeGradient, parameter gradients (Sec. 4.1.2):
 *   dw[k,c,r,s] = sum_{n,p,q} dy[n,k,p,q] * x[n,c,p*sh-ph+r, q*sw-pw+s]
 *   db[k]       = sum_{n,p,q} dy[n,k,p,q]            (skipped if db == NULL)
 * x: N*C*H*W, dy: N*K*P*Q, dw: K*C*R*S (overwritten), db: K. */
void oracle_conv_bwd_filter(int64_t N, int64_t C, int64_t H, int64_t W,
                            int64_t K, int64_t R, int64_t S,
                            int64_t ph, int64_t pw, int64_t sh, int64_t sw,
                            const double* x, const double* dy, double* dw, double* db);

/* Point evaluators: the same definitions as above, evaluated only at the
 * npts flat output indices idx[] (into y, dx or dw respectively), written to
 * out[0..npts).  Used where a full evaluation would take minutes. */
void oracle_conv_fwd_points(int64_t N, int64_t C, int64_t H, int64_t W,
                            int64_t K, int64_t R, int64_t S,
                            int64_t ph, int64_t pw, int64_t sh, int64_t sw,
                            const double* x, const double* w, const double* b,
                            int64_t npts, const int64_t* idx, double* out);
void oracle_conv_bwd_data_points(int64_t N, int64_t C, int64_t H, int64_t W,
                                 int64_t K, int64_t R, int64_t S,
                                 int64_t ph, int64_t pw, int64_t sh, int64_t sw,
                                 const double* dy, const double* w,
                                 int64_t npts, const int64_t* idx, double* out);
void oracle_conv_bwd_filter_points(int64_t N, int64_t C, int64_t H, int64_t W,
                                   int64_t K, int64_t R, int64_t S,
                                   int64_t ph, int64_t pw, int64_t sh, int64_t sw,
                                   const double* x, const double* dy,
                                   int64_t npts, const int64_t* idx, double* out);

/* Inner-product (fully connected) layer, named in Sec. 4.2.1 and Sec. 4.2.3:
 *   y[n,j] = b[j] + sum_i x[n,i] * w[j,i]; dx = dy * w; dw = dy^T * x; db = sum_n dy.
 * x: N*I, w: J*I, y: N*J.  b and db may be NULL. */
void oracle_fc_fwd(int64_t N, int64_t I, int64_t J,
                   const double* x, const double* w, const double* b, double* y);
void oracle_fc_bwd(int64_t N, int64_t I, int64_t J,
                   const double* x, const double* w, const double* dy,
                   double* dx, double* dw, double* db);

/* Pooling layer (Caffe's pooling, which SINGA adopts, Sec. 6.2.1).
 * mode 0 = MAX: y = maximum over the in-bounds cells of the window, found by a
 *   row-major scan that only replaces on a strictly greater value (the first
 *   maximum wins); argmax[o] = r*kw + s, the window-relative cell of that
 *   maximum (0 .. kh*kw-1).
 * mode 1 = AVG: y = (sum over in-bounds cells) / divisor, where divisor is the
 *   window size after clipping it to [-pad, H+pad) x [-pad, W+pad).
 * argmax may be NULL for AVG.  x: N*C*H*W, y and argmax: N*C*P*Q. */
void oracle_pool_fwd(int mode, int64_t N, int64_t C, int64_t H, int64_t W,
                     int64_t kh, int64_t kw, int64_t sh, int64_t sw,
                     int64_t ph, int64_t pw, int ceil_mode,
                     const double* x, double* y, uint8_t* argmax);

/* Pooling backward: dx (overwritten) receives, from every window o,
 * MAX: dy[o] at the cell argmax[o] names; AVG: dy[o]/divisor(o) at each
 * in-bounds cell.  Contributions of overlapping windows add up. */
void oracle_pool_bwd(int mode, int64_t N, int64_t C, int64_t H, int64_t W,
                     int64_t kh, int64_t kw, int64_t sh, int64_t sw,
                     int64_t ph, int64_t pw, int ceil_mode,
                     const double* dy, const uint8_t* argmax, double* dx);

/* ReLU: y = x if x > 0 else 0;  dx = dy if y > 0 else 0. */
void oracle_relu_fwd(int64_t n, const double* x, double* y);
void oracle_relu_bwd(int64_t n, const double* y, const double* dy, double* dx);

/* Local response normalization across channels (the layer of Sec. 5.4.1
 * that the paper's GPU AlexNet leaves out), with Caffe's conventions as for
 * convolution and pooling (Sec. 6.2.1), NCHW:
 *   s[n,c,h,w] = k + alpha/size * sum_{c' in [c - size/2, c + (size-1)/2] cap [0, C)} x[n,c',h,w]^2
 *   y[n,c,h,w] = x[n,c,h,w] * s[n,c,h,w]^-beta
 * lrn_bwd: dx = the gradient of sum(dy * y) with respect to x. */
void oracle_lrn_fwd(int64_t N, int64_t C, int64_t H, int64_t W, const double* x,
                    int64_t size, double alpha, double beta, double k, double* y);
void oracle_lrn_bwd(int64_t N, int64_t C, int64_t H, int64_t W, const double* x, const double* dy,
                    int64_t size, double alpha, double beta, double k, double* dx);

/* Softmax cross-entropy loss layer (Sec. 2.1, Table 2 and Sec. 4.2.3 name
 * the cross-entropy loss and the softmax loss layer), mean over the batch:
 *   loss = (1/B) sum_n ( log sum_j exp(z[n,j]) - z[n, label[n]] )
 *   dz[n,j] = ( softmax(z[n])_j - [j == label[n]] ) / B
 * z: B*classes, label: B, dz: B*classes.  Returns the loss. */
double oracle_softmax_ce(int64_t B, int64_t classes, const double* z,
                         const int32_t* label, double* dz);

/* Storage rounding of a bf16 layer boundary, in place: each value is rounded
 * to binary32 (round to nearest even) and then to bfloat16 (round to nearest
 * even on the 16 discarded mantissa bits), i.e. the value a bf16 tensor would
 * hold after an fp32 computation.  Used to take the ReLU and max-pooling
 * decisions on the same stored values as a bf16 pipeline. */
void oracle_round_bf16(int64_t n, double* x);

/* Updater (Sec. 4.1.4): one step of SGD with momentum and weight decay,
 * in place on w and v:
 *   g' = g + wd * w;  v = momentum * v + lr * g';  w = w - v. */
void oracle_sgd_momentum(int64_t n, double* w, const double* g, double* v,
                         double lr, double momentum, double wd);

/* Updater (Sec. 4.1.4): one AdaGrad step (the protocol the section names;
 * Duchi, Hazan and Singer 2011, diagonal form), in place on w and the sum of
 * squared gradients h:
 *   g' = g + wd * w;  h = h + g'^2;  w = w - lr * g' / (delta + sqrt(h)). */
void oracle_adagrad(int64_t n, double* w, const double* g, double* h,
                    double lr, double delta, double wd);

#ifdef __cplusplus
}
#endif
#endif
