/*
 * singa_mi.h -- C ABI of the MI355X (gfx950) library for the data-parallel hot
 * path of SINGA's training loop (Wang et al., "Deep Learning At Scale and At
 * Ease", arXiv 1603.07846).
 *
 * The calls follow the paper's layer abstraction (Sec. 4.1.2, Fig. "Layer
 * abstraction"): every layer has a ComputeFeature function, which maps the
 * source layer's feature blob to this layer's blob, and a ComputeGradient
 * function, which computes both the gradients of the layer's Param objects
 * and the gradient of the source layer's blob.  Here
 *     ComputeFeature   -> singa_*_fwd
 *     ComputeGradient  -> singa_conv_bwd_data (source gradient)
 *                       + singa_conv_bwd_filter (Param gradients)
 * and the server-side Updater (Sec. 4.1.4) -> singa_sgd_momentum_update.
 * BPTrainOneBatch (Sec. 4.1.3, Alg. 1) calls them forward over the layers,
 * then backward in reverse order, then updates.
 *
 * General contract (applies to every call below)
 *   - All tensor pointers are DEVICE pointers unless stated otherwise, owned
 *     by the caller.  The library never allocates or frees device memory:
 *     scratch space is passed in as a caller-owned workspace whose size
 *     singa_conv_workspace_bytes() reports.
 *   - Tensors are dense and contiguous in the declared layout.  Activations
 *     are NHWC (SINGA_NHWC, filters KRSC) or NCHW (SINGA_NCHW, filters KCRS).
 *     NHWC is the native layout of the kernels; NCHW calls are carried out by
 *     permuting into the workspace around the same kernels.
 *   - Element types: SINGA_F32 (IEEE binary32) or SINGA_BF16 (bfloat16 bit
 *     patterns, uint16).  bf16 arithmetic accumulates in fp32 and rounds to
 *     nearest even when it stores bf16.  Parameter gradients, biases, master
 *     weights and momentum are always fp32.
 *   - Alignment (SINGA_ERR_ALIGN): tensor pointers must be aligned to their
 *     element size; the ReLU and update calls need 16-byte alignment.  The
 *     convolution and pooling kernels take 16-byte vector paths when the
 *     pointers are 16-byte aligned and the channel count allows, and
 *     element-wise paths otherwise (same results).
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL is the legacy
 *     null stream).  The library never synchronizes.  A kernel fault shows
 *     up at the caller's next synchronization.
 *   - Validation happens before anything is enqueued: a non-zero return means
 *     no work was launched and no output was touched.
 *   - Functions keep no state between calls and may be called from several
 *     threads at once; the only process-wide state is the optional timing
 *     trace (singa_trace_*), a switch the caller sets.  Concurrent calls on
 *     different streams must not share output or workspace buffers.  The
 *     dispatch rules (tile layouts, split counts) depend on the shapes only,
 *     never on the environment.
 */
#ifndef SINGA_MI_H
#define SINGA_MI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------- status codes */
#define SINGA_OK 0
#define SINGA_ERR_NULL (-1)        /* a required pointer argument is NULL */
#define SINGA_ERR_SHAPE (-2)       /* non-positive or inconsistent sizes, empty output */
#define SINGA_ERR_UNSUPPORTED (-3) /* dtype/layout/parameter combination not provided */
#define SINGA_ERR_WORKSPACE (-4)   /* workspace smaller than singa_conv_workspace_bytes() */
#define SINGA_ERR_ALIGN (-5)       /* a device pointer is misaligned (see below) */
#define SINGA_ERR_HIP (-6)         /* the HIP runtime rejected a launch */
#define SINGA_ERR_SCRATCH (-7)     /* needs more than the library's fixed scratch array holds */

typedef enum { SINGA_F32 = 0, SINGA_BF16 = 1 } singa_dtype;
/* SINGA_NHWC_S2D: the input of a strided convolution already in its
 * space-to-depth form (see singa_space_to_depth); accepted as the input
 * layout of singa_conv_fwd, singa_conv_bwd_filter and their workspace
 * queries only, for the convolutions singa_space_to_depth_bytes reports a
 * size for (filters, gradients and outputs then as for SINGA_NHWC). */
typedef enum { SINGA_NCHW = 0, SINGA_NHWC = 1, SINGA_NHWC_S2D = 2 } singa_layout;
typedef enum { SINGA_POOL_MAX = 0, SINGA_POOL_AVG = 1 } singa_pool_mode;
typedef enum {
  SINGA_OP_FWD = 0,
  SINGA_OP_BWD_DATA = 1,
  SINGA_OP_BWD_FILTER = 2,
  SINGA_OP_BWD_FILTER_SGD = 3
} singa_conv_op;

/* Activation extents (batch, channels, height, width), whatever the layout. */
typedef struct { int n, c, h, w; } singa_shape4;
/* Filter extents (filters, channels, rows, cols), whatever the layout. */
typedef struct { int k, c, r, s; } singa_filter4;
/* Zero padding and stride (dilation 1, one group). */
typedef struct { int pad_h, pad_w, stride_h, stride_w; } singa_conv_desc;
/* Pooling window; ceil_mode != 0 rounds the output extent up (Caffe's rule). */
typedef struct { int mode, kh, kw, stride_h, stride_w, pad_h, pad_w, ceil_mode; } singa_pool_desc;
/* Local response normalization across channels: window of `size` channels,
 * s = k + alpha/size * (sum of squares over the window), y = x * s^-beta. */
typedef struct { int size; float alpha, beta, k; } singa_lrn_desc;

typedef void* singa_stream; /* a hipStream_t */

/* Message for a status code (static string). */
const char* singa_strerror(int status);

/* ------------------------------------------------------------ shape helpers */

/* Convolution output extents: P = floor((H + 2*pad_h - R)/stride_h) + 1 and
 * likewise Q; y->c = w->k.  Host-only; no GPU is touched.
 * Errors: NULL, SHAPE (non-positive sizes, channel mismatch, P or Q < 1). */
int singa_conv_out_shape(const singa_shape4* x, const singa_filter4* w,
                         const singa_conv_desc* d, singa_shape4* y);

/* Pooling output extents (Caffe's rule in ceil mode: a last window that would
 * start inside the right padding is dropped).  Host-only.
 * Errors: NULL, SHAPE, UNSUPPORTED (window larger than 255 cells, pad >= window). */
int singa_pool_out_shape(const singa_shape4* x, const singa_pool_desc* d, singa_shape4* y);

/* Workspace bytes that `op` needs for this problem (0 when none).  Host-only.
 * Errors: NULL, SHAPE, UNSUPPORTED. */
int singa_conv_workspace_bytes(int op, singa_dtype dtype, singa_layout layout,
                               const singa_shape4* x, const singa_filter4* w,
                               const singa_conv_desc* d, size_t* bytes);

/* -------------------------------------------------------------- convolution */

/* Convolution ComputeFeature (Sec. 4.1.2; the neuron layer of Table 2),
 * cross-correlation as in Caffe's im2col that SINGA adopts (Sec. 6.2.1):
 *   y[n,k,p,q] = bias[k] + sum_{c,r,s} W[k,c,r,s] * x[n,c,p*sh-ph+r, q*sw-pw+s]
 * with zero padding, then y = max(y, 0) if fuse_relu.
 *   x_ptr : dtype, shape *x in `layout`            (read; with SINGA_NHWC_S2D
 *           the output of singa_space_to_depth for this convolution)
 *   w_ptr : dtype, shape *w (KRSC for NHWC, KCRS for NCHW)   (read)
 *   bias  : fp32[w->k] or NULL                      (read)
 *   y_ptr : dtype, shape singa_conv_out_shape()     (written)
 *   ws    : workspace of singa_conv_workspace_bytes(SINGA_OP_FWD, ...) bytes
 * Implicit GEMM on MFMA (M = N*P*Q output pixels, N = K filters,
 * K = R*S*C taps). */
int singa_conv_fwd(singa_dtype dtype, singa_layout layout,
                   const singa_shape4* x, const void* x_ptr,
                   const singa_filter4* w, const void* w_ptr, const float* bias,
                   const singa_conv_desc* d, void* y_ptr, int fuse_relu,
                   void* ws, size_t ws_bytes, singa_stream stream);

/* Space-to-depth form of a strided convolution's NHWC input, for callers
 * that pass the same input to both singa_conv_fwd and singa_conv_bwd_filter
 * (the first layer of a network): each of those calls otherwise builds this
 * form itself in its workspace.  With stride (sh, sw), padding (ph, pw),
 * R' = ceil(R/sh), S' = ceil(S/sw), P x Q the output extents:
 *   xs[n][h'][w'][(dh*sw + dw)*C + c] = x[n][sh*h' + dh - ph][sw*w' + dw - pw][c]
 *   (0 outside x), h' < P + R' - 1, w' < Q + S' - 1, dh < sh, dw < sw,
 * and the convolution equals the stride-1 unpadded convolution of xs with
 * the filter rearranged the same way (the library rearranges it).
 *   x_ptr  : dtype, shape *x, NHWC                  (read)
 *   xs_ptr : dtype, singa_space_to_depth_bytes() bytes, 16-byte aligned (written)
 * Errors: NULL, SHAPE, ALIGN, UNSUPPORTED (this convolution is not run on
 * the space-to-depth form: singa_space_to_depth_bytes reports 0), HIP. */
int singa_space_to_depth_bytes(singa_dtype dtype, const singa_shape4* x, const singa_filter4* w,
                               const singa_conv_desc* d, size_t* bytes);
int singa_space_to_depth(singa_dtype dtype, const singa_shape4* x, const void* x_ptr,
                         const singa_filter4* w, const singa_conv_desc* d, void* xs_ptr,
                         singa_stream stream);

/* Convolution ComputeGradient, gradient of the source layer (Sec. 4.1.2):
 *   dx[n,c,h,w] = sum over (k,r,s,p,q) with p*sh-ph+r = h, q*sw-pw+s = w
 *                 of W[k,c,r,s] * dy[n,k,p,q]
 *   x      : shape of the layer's input (the shape of dx)
 *   dy_ptr : dtype, shape singa_conv_out_shape()    (read)
 *   relu_y : NULL, or dtype, shape *x (read): the output of a ReLU layer that
 *            is this layer's source.  Then dx is the gradient at that ReLU's
 *            input instead: dx[i] = relu_y[i] > 0 ? (the sum above) : 0, the
 *            ReLU layer's ComputeGradient folded into this call.  NCHW callers
 *            must pass 16-byte aligned relu_y and dx_ptr.
 *   dx_ptr : dtype, shape *x                        (overwritten)
 * Stride 1 (and dense "fully connected" geometry) runs as an implicit GEMM on
 * MFMA over a flipped, transposed copy of W in the workspace; other strides
 * run a gather kernel. */
int singa_conv_bwd_data(singa_dtype dtype, singa_layout layout,
                        const singa_shape4* x, const singa_filter4* w, const void* w_ptr,
                        const singa_conv_desc* d, const void* dy_ptr, const void* relu_y,
                        void* dx_ptr, void* ws, size_t ws_bytes, singa_stream stream);

/* Convolution ComputeGradient, Param gradients (Sec. 4.1.2):
 *   dW[k,c,r,s] = sum_{n,p,q} dy[n,k,p,q] * x[n,c,p*sh-ph+r, q*sw-pw+s]
 *   db[k]       = sum_{n,p,q} dy[n,k,p,q]
 *   x_ptr  : dtype, shape *x (SINGA_NHWC_S2D: its space-to-depth form)  (read)
 *   dy_ptr : dtype, shape singa_conv_out_shape()    (read)
 *   dw     : fp32, shape *w in the filter layout    (written, or added to)
 *   db     : fp32[w->k] or NULL                     (written, or added to)
 *   accumulate != 0 adds into dw/db instead of overwriting them, so a batch
 *   can be processed in shards (dim-0 partitioning, Sec. 5.3).
 * Split-K implicit GEMM on MFMA with a fixed-order reduction of the partial
 * sums (bitwise deterministic; no floating-point atomics). */
int singa_conv_bwd_filter(singa_dtype dtype, singa_layout layout,
                          const singa_shape4* x, const void* x_ptr,
                          const singa_filter4* w, const singa_conv_desc* d,
                          const void* dy_ptr, float* dw, float* db, int accumulate,
                          void* ws, size_t ws_bytes, singa_stream stream);

/* singa_conv_bwd_filter for callers that cannot allocate device memory: code
 * recorded under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  Same arguments, results and kernels, without the
 * workspace: its scratch is a fixed array of SINGA_NOALLOC_SCRATCH_BYTES in
 * device memory that the library holds on each GPU it runs on until the
 * process ends (looked up on a device's first call; nothing is allocated
 * here or later).
 *   Returns SINGA_ERR_SCRATCH (nothing enqueued) when the call would need
 *   more than SINGA_NOALLOC_SCRATCH_BYTES of workspace
 *   (singa_conv_workspace_bytes(SINGA_OP_BWD_FILTER, ...) reports it; every
 *   AlexNet-shaped layer up to batch 256 fits), and SINGA_ERR_UNSUPPORTED
 *   when `stream` belongs to another device than the current one.
 *   Every call on one GPU uses that GPU's one array: calls whose execution
 *   overlaps on the same GPU (different streams, or several host threads)
 *   race on it and give wrong results; serialize them.  Calls on one stream
 *   are serialized by the stream.  Nothing in the array needs clearing. */
#define SINGA_NOALLOC_SCRATCH_BYTES (128u << 20)
int singa_conv_bwd_filter_noalloc(singa_dtype dtype, singa_layout layout,
                                  const singa_shape4* x, const void* x_ptr,
                                  const singa_filter4* w, const singa_conv_desc* d,
                                  const void* dy_ptr, float* dw, float* db, int accumulate,
                                  singa_stream stream);

/* Convolution ComputeGradient for the Params followed at once by the
 * Updater's step on them (Alg. 1 calls Update on a layer's Params right after
 * its ComputeGradient; the Updater of Sec. 4.1.4, as in
 * singa_sgd_momentum_update):
 *   g = dW (and db) exactly as singa_conv_bwd_filter computes them;
 *   v = momentum * v + lr * (g + weight_decay * w);  w = w - v;
 *   w_bf16 = bf16(w) (round to nearest even) when w_bf16 != NULL
 * for the filter (w_master, w_mom: fp32, w_bf16: bf16 bits, shape *w in the
 * filter layout; updated in place) and, when b_master != NULL, for the bias
 * (b_master, b_mom, b_bf16: w->k values).  Every element ends up exactly as
 * singa_sgd_momentum_update leaves it given that gradient.
 *   dw, db : NULL, or fp32 arrays (filter layout / w->k) that also receive
 *            the gradient.
 * The update arrays need 16-byte alignment.  The call reads the filter only
 * through w_master, so a backward-data pass that needs the layer's current
 * bf16 filter must be enqueued before it.
 * singa_conv_workspace_bytes(SINGA_OP_BWD_FILTER_SGD, ...) is 0 exactly when
 * the update is fused into the gradient kernel (bf16, NHWC, K and C multiples
 * of 8, no rewrite of the input, and N*P*Q short enough for a single pass
 * over the reduction, as for fully connected layers): each gradient element
 * is applied where it is complete, without a round trip through memory, and
 * x_ptr and dy_ptr must be 16-byte aligned (SINGA_ERR_ALIGN otherwise).  In
 * every other case the gradient is formed in dw/db or in the workspace and
 * the update follows. */
int singa_conv_bwd_filter_sgd(singa_dtype dtype, singa_layout layout,
                              const singa_shape4* x, const void* x_ptr,
                              const singa_filter4* w, const singa_conv_desc* d,
                              const void* dy_ptr, float* dw, float* db,
                              float* w_master, float* w_mom, uint16_t* w_bf16,
                              float* b_master, float* b_mom, uint16_t* b_bf16,
                              float lr, float momentum, float weight_decay,
                              void* ws, size_t ws_bytes, singa_stream stream);

/* ------------------------------------------------------------------ pooling */

/* Pooling ComputeFeature (Caffe's pooling, adopted in Sec. 6.2.1).
 * MAX: y = largest in-bounds value of the window, scanned row-major with the
 *      first maximum winning; argmax[o] = r*kw + s of that cell (uint8).
 * AVG: y = sum of in-bounds values / (window size after clipping it to
 *      [-pad, H+pad) x [-pad, W+pad)); argmax is ignored and may be NULL.
 *   x_ptr : dtype, shape *x (read);  y_ptr : dtype, singa_pool_out_shape() (written)
 *   argmax: uint8, one per output element (written; required for MAX) */
int singa_pool_fwd(singa_dtype dtype, singa_layout layout,
                   const singa_shape4* x, const void* x_ptr, const singa_pool_desc* d,
                   void* y_ptr, uint8_t* argmax, singa_stream stream);

/* Pooling ComputeGradient: every input cell gathers, from each window that
 * covers it, dy[o] if it is that window's argmax (MAX) or dy[o]/divisor(o)
 * (AVG).  dx_ptr (shape *x) is overwritten; no atomics.
 *   relu_y : NULL, or (MAX only) the pooling's forward output y_ptr, when the
 *            pooling's input is the output of a ReLU layer.  Then dx is the
 *            gradient at that ReLU's input: a window routes dy[o] only when
 *            y[o] > 0.  This is exact: the arg-max cell holds y[o], so it is
 *            the ReLU's output there.  AVG with relu_y is SINGA_ERR_UNSUPPORTED. */
int singa_pool_bwd(singa_dtype dtype, singa_layout layout,
                   const singa_shape4* x, const singa_pool_desc* d,
                   const void* dy_ptr, const uint8_t* argmax, const void* relu_y,
                   void* dx_ptr, singa_stream stream);

/* --------------------------------------------------------------------- ReLU */

/* The rectified linear unit that follows every convolution of the
 * CIFAR-shaped and AlexNet-shaped workloads (the cuda-convnet DCNN of
 * Sec. 6.2.1 and the AlexNet variant of Sec. 6.3.1), as a layer of its own
 * in the layer abstraction of Sec. 4.1.2 (Table 2 lists the neuron layers).
 * ComputeFeature: y = x > 0 ? x : 0 over n elements (in place allowed:
 * y == x).  x, y: dtype arrays of n elements, 16-byte aligned. */
int singa_relu_fwd(singa_dtype dtype, size_t n, const void* x, void* y, singa_stream stream);

/* ComputeGradient of the same layer: dx = y > 0 ? dy : 0 over n elements
 * (the derivative at 0 is taken as 0; in place allowed: dx == dy).  y is the
 * layer's output, dy the gradient at it; 16-byte aligned. */
int singa_relu_bwd(singa_dtype dtype, size_t n, const void* y, const void* dy, void* dx,
                   singa_stream stream);

/* ---------------------------------------------- local response normalization */

/* Local response normalization across channels, the layer Sec. 5.4.1 names
 * beside pooling (the paper's GPU AlexNet leaves it out), in Caffe's form as
 * SINGA's convolution and pooling are (Sec. 6.2.1):
 *   s[n,c,h,w] = k + alpha/size * sum_{c'} x[n,c',h,w]^2 over the channels
 *                c' in [c - size/2, c + (size-1)/2] that exist (in [0, C))
 *   y = x * s^-beta
 * singa_lrn_bwd: dx = the gradient of sum(dy * y) with respect to x,
 *   dx[c] = dy[c] s[c]^-beta - (2 alpha beta / size) x[c]
 *           * sum over the channels j whose window holds c of dy[j] x[j] s[j]^(-beta-1)
 * (s recomputed from x).  fp32 arithmetic for both dtypes.
 *   x_ptr, dy_ptr : dtype, shape *x in `layout` (read);  y_ptr / dx_ptr (written)
 *   d: size >= 1, alpha >= 0, k > 0 (SINGA_ERR_UNSUPPORTED otherwise). */
int singa_lrn_fwd(singa_dtype dtype, singa_layout layout, const singa_shape4* x, const void* x_ptr,
                  const singa_lrn_desc* d, void* y_ptr, singa_stream stream);
int singa_lrn_bwd(singa_dtype dtype, singa_layout layout, const singa_shape4* x, const void* x_ptr,
                  const void* dy_ptr, const singa_lrn_desc* d, void* dx_ptr, singa_stream stream);

/* ------------------------------------------------------------ softmax loss */

/* Softmax cross-entropy loss layer (Sec. 2.1 and Table 2 name the
 * cross-entropy loss; Sec. 4.2.3 the softmax loss layer), mean over the batch:
 *   loss    = (1/B) sum_n ( logsumexp(z[n,:]) - z[n, label[n]] )
 *   dlogits = ( softmax(z[n,:]) - onehot(label[n]) ) / B
 *   logits : dtype [batch][classes] (read);  labels : int32[batch] (read)
 *   loss   : fp32 device array of batch + 1 values (written): loss[0] is the
 *            mean, loss[1 + n] row n's loss
 *   dlogits: dtype [batch][classes] (written)
 * A label outside [0, classes) contributes a zero row loss and its row of
 * dlogits is the plain softmax / B.  The mean is summed in a fixed order. */
int singa_softmax_ce(singa_dtype dtype, int batch, int classes, const void* logits,
                     const int32_t* labels, float* loss, void* dlogits, singa_stream stream);

/* ------------------------------------------------------------------ updater */

/* Updater (Sec. 4.1.4): one fused SGD-with-momentum step over n fp32 values,
 *   g' = g + weight_decay * w;  v = momentum * v + lr * g';  w = w - v
 * and, if w_bf16 != NULL, w_bf16 = bf16(w) (round to nearest even), the
 * compute copy for bf16 layers.  w, v updated in place; g read. */
int singa_sgd_momentum_update(size_t n, float* w, const float* g, float* v, uint16_t* w_bf16,
                              float lr, float momentum, float weight_decay, singa_stream stream);

/* Updater (Sec. 4.1.4), the AdaGrad protocol the section names (Duchi, Hazan
 * and Singer, JMLR 2011, diagonal form): one fused step over n fp32 values,
 *   g' = g + weight_decay * w;  h = h + g'^2;  w = w - lr * g' / (delta + sqrt(h))
 * and, if w_bf16 != NULL, w_bf16 = bf16(w) (round to nearest even).
 *   w, h : updated in place (h, the running sum of squared gradients, starts
 *          at 0);  g : read.  All four pointers 16-byte aligned.
 *   delta > 0 (SINGA_ERR_UNSUPPORTED otherwise: the first step divides by
 *   delta + |g'|), lr >= 0. */
int singa_adagrad_update(size_t n, float* w, const float* g, float* h, uint16_t* w_bf16,
                         float lr, float delta, float weight_decay, singa_stream stream);

/* ------------------------------------------------------ per-kernel timing */

/* Kernel timing trace, a profiling aid for the per-iteration timing protocol
 * of Sec. 6.2.2 (time each step, average over a window of iterations).
 * While enabled, every kernel the library launches is bracketed by two
 * timing events recorded on its own stream and tagged with the kernel's name
 * and algorithmic work (flops for the matrix kernels, bytes moved for the
 * bandwidth-bound ones).  Host-side bookkeeping only; off by default.
 *   singa_trace_enable(on): on != 0 clears the trace and starts recording,
 *                           0 stops recording (the trace is kept).  Returns 0.
 *   singa_trace_count():    number of recorded launches (at most 65536).
 *   singa_trace_get(i, ...): launch i's kernel name (static string), elapsed
 *                           milliseconds, work and unit (0 = flop, 1 = byte).
 *                           The launch's stream must have been synchronized.
 *                           Returns 0, -1 (NULL argument), -2 (i out of
 *                           range) or -6 (the events are not complete). */
int singa_trace_enable(int on);
int singa_trace_count(void);
int singa_trace_get(int i, const char** kernel, double* ms, double* work, int* unit);

#ifdef __cplusplus
}
#endif
#endif /* SINGA_MI_H */
