// internal.h -- launchers shared between the ABI layer and the kernel files.
// Everything here works on NHWC activations and KRSC filters; the ABI layer
// validates arguments before calling in, so launchers assume consistent
// shapes, element-aligned pointers and tensors of fewer than 2^31 bytes (the
// convolution kernels address operands with 32-bit buffer offsets).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace singa {

enum Dt { F32 = 0, BF16 = 1 };

inline size_t dt_size(int dt) { return dt == BF16 ? 2 : 4; }

// Per-kernel timing (trace.cpp): while the trace is enabled, a TraceScope
// brackets one kernel launch with timing events on its stream and tags it with
// the kernel's algorithmic work.
enum { WORK_FLOP = 0, WORK_BYTE = 1 };
class TraceScope {
 public:
  TraceScope(const char* name, hipStream_t st, double work, int unit);
  ~TraceScope();
  TraceScope(const TraceScope&) = delete;
  TraceScope& operator=(const TraceScope&) = delete;

 private:
  hipStream_t st_;
  long idx_;
};

// Geometry of one convolution: input N x H x W x C, K filters R x S x C,
// output N x P x Q x K.
struct ConvShape {
  int N, H, W, C, K, R, S, P, Q, ph, pw, sh, sw;
};

// Implicit-GEMM forward convolution (also used for stride-1 backward-data over
// a flipped filter copy, bwd != 0): y = act(conv(x, w) + bias).  `flops` is
// the algorithmic work of the layer pass this launch carries out.  When the
// output tiles cannot fill the GPU and `partial` (fwd_partial_bytes() of
// workspace) is given, the taps are split across workgroups and a second
// kernel adds the fp32 partial tiles in a fixed order.  `mask` (optional, the
// shape of y) zeroes each output whose mask value is <= 0: the backward of a
// ReLU whose output is `mask`, folded into the store.
hipError_t launch_conv_fwd(int dt, const ConvShape& s, const void* x, const void* w, const float* bias,
                           void* y, int relu, int bwd, double flops, float* partial, const void* mask,
                           hipStream_t st);
size_t fwd_partial_bytes(const ConvShape& s, int dt);

// The same GEMM for a 1x1 geometry (R = S = 1) with the filter given
// transposed, wt[c][k] (the K filter columns contiguous), as the dense
// backward-data needs it: the weight matrix as stored, no transposed copy.
// bf16 only, K % 8 == 0, 16-byte aligned wt; otherwise returns
// hipErrorNotSupported and launches nothing.  No bias, no ReLU.
hipError_t launch_conv_fwd_wt(int dt, const ConvShape& s, const void* x, const void* wt, void* y, int bwd,
                              double flops, float* partial, const void* mask, hipStream_t st);

// Split-K implicit-GEMM filter gradient, dw (K, R, S, C) and, with db, the
// bias gradient from one more GEMM column against ones.  With one split the
// kernel writes (or, with acc_dw / acc_db, adds into) dw and db directly;
// otherwise it writes partial tiles into `partial` (wgrad_partial_bytes() of
// workspace; NULL when that is 0) and a second kernel adds them in a fixed
// order.  `flops` is the algorithmic work of the layer pass this launch
// carries out (s may be a rewritten geometry with zero taps).
size_t wgrad_partial_bytes(const ConvShape& s, int dt, bool bias);
hipError_t launch_conv_wgrad(int dt, const ConvShape& s, const void* x, const void* dy, float* partial, float* dw,
                             float* db, int acc_dw, int acc_db, double flops, hipStream_t st);

// Parameters the filter-gradient kernel updates in place once a gradient
// element is complete (SGD with momentum, one step per element): the fp32
// master filter w (K, R, S, C), its momentum v and its bf16 compute copy wb
// (NULL: none); the same for the bias (b NULL: no bias).
struct SgdTargets {
  float* w;
  float* v;
  uint16_t* wb;
  float* b;
  float* vb;
  uint16_t* bb;
  float lr, mom, wd;
};

// True when the filter gradient of s runs as one pass of the 128 x 256 kernel
// writing each element once (bf16, K % 8 == 0, C % 8 == 0, one split), the
// case in which the update is fused into it.
bool wgrad_update_fusable(const ConvShape& s, int dt, bool bias);

// The filter gradient with the update fused: every complete element g of dw
// (and db) is applied to the targets and, when dw (db) is not NULL, also
// stored there.  x and dy must be 16-byte aligned and wgrad_update_fusable()
// true; otherwise returns hipErrorNotSupported and launches nothing.
hipError_t launch_conv_wgrad_sgd(int dt, const ConvShape& s, const void* x, const void* dy, float* dw, float* db,
                                 const SgdTargets& u, hipStream_t st);

// The filter gradient with the update applied by its split-K reduction: the
// GEMM writes partial tiles into `partial` (wgrad_partial_bytes() of
// workspace) and the fixed-order reduction applies the step to each summed
// element (w, v, wb, and b, vb, bb with a bias), storing the gradient in dw
// (db) too when not NULL.  When the kernel that runs s would use a single
// split and cannot take the update itself, returns hipErrorNotSupported and
// launches nothing.
hipError_t launch_conv_wgrad_reduce_sgd(int dt, const ConvShape& s, const void* x, const void* dy, float* partial,
                                        float* dw, float* db, const SgdTargets& u, double flops, hipStream_t st);

// Batched 2-D transpose: for b in [0, batch): out(b)[c][r] = in(b)[r][c] with
// in(b) = in + in_base(b), out(b) = out + out_base(b), where
// in_base(b) = b * in_bstride and out_base(b) = (flip ? batch-1-b : b) * out_bstride.
hipError_t launch_transpose(int dt, const void* in, void* out, int batch, int rows, int cols,
                            long in_bstride, long in_rstride, long out_bstride, long out_rstride,
                            int flip, hipStream_t st);

// Direct (gather) backward-data for any stride: dx = conv^T(dy, w).
hipError_t launch_conv_bwd_data_direct(int dt, const ConvShape& s, const void* dy, const void* w, void* dx,
                                       const void* mask, hipStream_t st);

// Zero-pad the innermost (channel) dimension: in [rows][C] -> out [rows][Cp],
// Cp a multiple of the 16-byte vector width.
hipError_t launch_pad_channels(int dt, const void* in, void* out, long rows, int C, int Cp, hipStream_t st);
// Space-to-depth rewrite of the strided convolution s as the stride-1,
// unpadded convolution g (H, W, C, R, S of g are the rewritten ones): input,
// filter, filter gradient (fp32, optionally accumulated) and input gradient
// (optionally masked by a ReLU output).
hipError_t launch_space_to_depth(int dt, const ConvShape& s, const ConvShape& g, const void* x, void* xs,
                                 hipStream_t st);
hipError_t launch_filter_to_s2d(int dt, const ConvShape& s, const ConvShape& g, const void* w, void* ws,
                                hipStream_t st);
hipError_t launch_s2d_to_filter_f32(const ConvShape& s, const ConvShape& g, const float* dws, float* dw,
                                    int accumulate, hipStream_t st);
hipError_t launch_depth_to_space(int dt, const ConvShape& s, const ConvShape& g, const void* dxs, const void* mask,
                                 void* dx, hipStream_t st);
hipError_t launch_unpad_channels_f32(const float* in, float* out, long rows, int Cp, int C, int accumulate,
                                     hipStream_t st);

// NCHW <-> NHWC permutations for the NCHW entry points.
hipError_t launch_nchw_to_nhwc(int dt, const void* in, void* out, int N, int C, int H, int W, hipStream_t st);
hipError_t launch_nhwc_to_nchw(int dt, const void* in, void* out, int N, int C, int H, int W, hipStream_t st);
// fp32 filter gradient KRSC -> KCRS, with optional accumulation into out.
hipError_t launch_krsc_to_kcrs_f32(const float* in, float* out, int K, int C, int R, int S, int accumulate,
                                   hipStream_t st);

// Pooling, ReLU, softmax-CE, SGD.
hipError_t launch_pool_fwd(int dt, int mode, int N, int C, int H, int W, int P, int Q, int kh, int kw, int sh,
                           int sw, int ph, int pw, const void* x, void* y, uint8_t* argmax, int nchw,
                           hipStream_t st);
// ymask (MAX only, optional): the pooling's forward output; a window routes
// its gradient only when its maximum is > 0 (ReLU backward on the pooling's
// input folded in: the input equals the maximum at the arg-max cell).
hipError_t launch_pool_bwd(int dt, int mode, int N, int C, int H, int W, int P, int Q, int kh, int kw, int sh,
                           int sw, int ph, int pw, const void* dy, const uint8_t* argmax, const void* ymask,
                           void* dx, int nchw, hipStream_t st);
hipError_t launch_relu_fwd(int dt, size_t n, const void* x, void* y, hipStream_t st);
hipError_t launch_relu_bwd(int dt, size_t n, const void* y, const void* dy, void* dx, hipStream_t st);

// Local response normalization across channels (bwd = 0: y = lrn(x) into
// out; bwd = 1: dx into out from x and dy), N x C x HW elements, NHWC or NCHW.
hipError_t launch_lrn(int dt, int bwd, int N, int C, int HW, int size, float alpha, float beta, float k,
                      const void* x, const void* dy, void* out, int nchw, hipStream_t st);
hipError_t launch_softmax_ce(int dt, int B, int classes, const void* z, const int32_t* labels, float* loss,
                             void* dz, hipStream_t st);
hipError_t launch_adagrad(size_t n, float* w, const float* g, float* h, uint16_t* wb, float lr, float delta,
                          float wd, hipStream_t st);
hipError_t launch_sgd(size_t n, float* w, const float* g, float* v, uint16_t* wb, float lr, float mom, float wd,
                      hipStream_t st);

}  // namespace singa
