// abi.cpp -- the C entry points declared in include/singa_mi.h: argument
// validation, workspace carving, NCHW <-> NHWC staging and kernel dispatch.
// Nothing is enqueued unless every check passes.
#include "singa_mi.h"

#include <hip/hip_runtime.h>

#include <climits>
#include <cstdint>

#include "internal.h"

using namespace singa;

namespace {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

inline bool aligned_to(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

inline int hip_status(hipError_t e) { return e == hipSuccess ? SINGA_OK : SINGA_ERR_HIP; }

bool dtype_ok(int dt) { return dt == SINGA_F32 || dt == SINGA_BF16; }
bool layout_ok(int l) { return l == SINGA_NCHW || l == SINGA_NHWC; }

bool fits_i32(long long v) { return v > 0 && v < (long long)INT_MAX; }

// Shape checks shared by the convolution calls; fills s on success.
int conv_geometry(const singa_shape4* x, const singa_filter4* w, const singa_conv_desc* d, ConvShape* s) {
  if (!x || !w || !d) return SINGA_ERR_NULL;
  if (x->n <= 0 || x->c <= 0 || x->h <= 0 || x->w <= 0) return SINGA_ERR_SHAPE;
  if (w->k <= 0 || w->c <= 0 || w->r <= 0 || w->s <= 0) return SINGA_ERR_SHAPE;
  if (w->c != x->c) return SINGA_ERR_SHAPE;
  if (d->pad_h < 0 || d->pad_w < 0 || d->stride_h < 1 || d->stride_w < 1) return SINGA_ERR_SHAPE;
  const long long hs = (long long)x->h + 2LL * d->pad_h - w->r;
  const long long ws = (long long)x->w + 2LL * d->pad_w - w->s;
  if (hs < 0 || ws < 0) return SINGA_ERR_SHAPE;
  const long long P = hs / d->stride_h + 1, Q = ws / d->stride_w + 1;
  // every index the kernels form must fit a signed 32-bit integer
  // every operand must stay below 2^31 bytes in fp32 (32-bit buffer offsets)
  if (!fits_i32(4LL * x->n * x->h * x->w * x->c) || !fits_i32(4LL * x->n * P * Q * w->k) ||
      !fits_i32(4LL * w->k * w->r * w->s * w->c))
    return SINGA_ERR_UNSUPPORTED;
  s->N = x->n; s->H = x->h; s->W = x->w; s->C = x->c;
  s->K = w->k; s->R = w->r; s->S = w->s;
  s->P = (int)P; s->Q = (int)Q;
  s->ph = d->pad_h; s->pw = d->pad_w; s->sh = d->stride_h; s->sw = d->stride_w;
  return SINGA_OK;
}

inline size_t act_bytes(const ConvShape& s, int dt) { return (size_t)s.N * s.H * s.W * s.C * dt_size(dt); }
inline size_t out_bytes(const ConvShape& s, int dt) { return (size_t)s.N * s.P * s.Q * s.K * dt_size(dt); }
inline size_t filt_bytes(const ConvShape& s, int dt) { return (size_t)s.K * s.R * s.S * s.C * dt_size(dt); }
// Algorithmic flops of one pass of a convolution layer: 2 x the multiply-adds
// of the direct definition, padded taps included (the same for all 3 passes).
inline double conv_flops(const ConvShape& s) {
  return 2.0 * s.N * (double)s.P * s.Q * s.K * (double)s.C * s.R * s.S;
}

// Backward-data through the forward GEMM needs a transposed filter copy:
// dense "fully connected" geometry, or unit stride (flipped filter).
bool bwd_data_fc(const ConvShape& s) {
  return s.P == 1 && s.Q == 1 && s.ph == 0 && s.pw == 0 && s.R == s.H && s.S == s.W;
}
bool bwd_data_gemm(const ConvShape& s) { return bwd_data_fc(s) || (s.sh == 1 && s.sw == 1); }

// The forward convolution that carries out a GEMM-style backward-data:
// dense FC geometry: dx[n][(r,s,c)] = sum_k dy[n][k] w[k][(r,s,c)], a 1x1
//   "convolution" of dy (N x 1 x 1 x K) with wt[(r,s,c)][k];
// unit stride: dx = conv(dy, wt) with wt[c][r'][s'][k] = w[k][R-1-r'][S-1-s'][c]
//   and padding R-1-ph, S-1-pw.
ConvShape bwd_data_inner(const ConvShape& s) {
  if (bwd_data_fc(s)) return ConvShape{s.N, 1, 1, s.K, s.R * s.S * s.C, 1, 1, 1, 1, 0, 0, 1, 1};
  return ConvShape{s.N, s.P, s.Q, s.K, s.C, s.R, s.S, s.H, s.W, s.R - 1 - s.ph, s.S - 1 - s.pw, 1, 1};
}

// Workspace carving: a list of sub-buffers, each 256-byte aligned.
struct Carve {
  char* base;
  size_t used = 0;
  explicit Carve(void* b) : base((char*)b) {}
  void* take(size_t bytes) {
    void* p = base ? base + used : nullptr;
    used += align_up(bytes);
    return p;
  }
};

// Convolutions whose channel count is not a multiple of 4 (the first layer's
// 3 colour channels) run their forward and filter-gradient passes on copies of
// the input (and, forward, the filter) zero-padded to a multiple of 4
// channels, so that every tap load is a vector: 16 bytes for fp32, two 8-byte
// halves for bf16 (16-byte loads need 8 bf16 channels).  The padded taps are
// zeros: 4/3 of the layer's multiply-adds for C = 3.
inline int padded_channels(const ConvShape& s, int dt) {
  (void)dt;
  if (s.C % 4 == 0) return 0;
  const int cp = (s.C + 3) / 4 * 4;
  return cp <= 2 * s.C ? cp : 0;
}

// Space-to-depth geometry of the strided convolution s: blocks of sh x sw
// input pixels become channels, the filter shrinks to ceil(R/sh) x ceil(S/sw)
// and the layer becomes a stride-1 convolution without padding with the same
// output (the transforms are in conv_aux.hip).
ConvShape s2d_shape(const ConvShape& s) {
  ConvShape g = s;
  g.R = (s.R + s.sh - 1) / s.sh;
  g.S = (s.S + s.sw - 1) / s.sw;
  g.C = s.C * s.sh * s.sw;
  g.H = s.P + g.R - 1;
  g.W = s.Q + g.S - 1;
  g.ph = g.pw = 0;
  g.sh = g.sw = 1;
  return g;
}
bool s2d_fits(const ConvShape& g) {
  return fits_i32(4LL * g.N * g.H * g.W * g.C) && fits_i32(4LL * g.K * g.R * g.S * g.C);
}

// Input rewrite of the forward and filter-gradient GEMMs, and the GEMM's
// geometry g.  A strided layer whose channel count gives no 16-byte tap
// vectors but whose space-to-depth channel count does is rewritten as that
// stride-1 layer (the first layer, 11x11/4 on 3 channels, becomes 3x3/1 on
// 48 channels: 432 taps instead of 484 padded ones, all vector loads); other
// channel counts that are not a multiple of 4 are zero-padded.
enum Rewrite { RW_NONE, RW_PAD, RW_S2D };
Rewrite input_rewrite(const ConvShape& s, int dt, ConvShape* g) {
  const int vec = dt == BF16 ? 8 : 4;
  *g = s;
  if (s.C % vec != 0 && (s.sh > 1 || s.sw > 1) && !bwd_data_fc(s)) {
    const ConvShape t = s2d_shape(s);
    if (t.C % vec == 0 && s2d_fits(t)) {
      *g = t;
      return RW_S2D;
    }
  }
  const int cp = padded_channels(s, dt);
  if (cp) {
    g->C = cp;
    return RW_PAD;
  }
  return RW_NONE;
}

// Backward-data of a strided, non-dense layer: the stride-1 GEMM on the
// space-to-depth layer g, whose input gradient is then scattered back.
bool bwd_data_s2d(const ConvShape& s, ConvShape* g) {
  if (bwd_data_gemm(s)) return false;
  *g = s2d_shape(s);
  return s2d_fits(*g);
}

// A convolution whose input may be given in the space-to-depth layout: the
// ones input_rewrite runs on that form.
bool s2d_input_ok(const ConvShape& s, int dt) {
  ConvShape g;
  return input_rewrite(s, dt, &g) == RW_S2D;
}

// One function computes both the size and the layout of every workspace, so
// the two can never disagree.
struct FwdWs { void *x, *w, *y, *xp, *wp; float* partial; };
struct BwdDataWs { void *dy, *w, *wt, *dx, *ws, *dxs; float* partial; };
struct BwdFilterWs { void *x, *dy, *xp; float *dw, *dwp, *partial; };

size_t carve_fwd(const ConvShape& s, int dt, int layout, void* ws, FwdWs* o) {
  Carve c(ws);
  o->x = o->w = o->y = o->xp = o->wp = nullptr;
  o->partial = nullptr;
  if (layout == SINGA_NCHW) {
    o->x = c.take(act_bytes(s, dt));
    o->w = c.take(filt_bytes(s, dt));
    o->y = c.take(out_bytes(s, dt));
  }
  ConvShape g;
  if (input_rewrite(s, dt, &g) != RW_NONE) {
    // an input given in the space-to-depth layout is the rewritten input
    if (layout != SINGA_NHWC_S2D) o->xp = c.take((size_t)g.N * g.H * g.W * g.C * dt_size(dt));
    o->wp = c.take((size_t)g.K * g.R * g.S * g.C * dt_size(dt));
  }
  const size_t pb = fwd_partial_bytes(g, dt);
  if (pb) o->partial = (float*)c.take(pb);
  return c.used;
}

// NHWC forward on (x, w): through the rewritten input and filter when
// input_rewrite says so (x_s2d: x is already the space-to-depth input).
hipError_t conv_fwd_nhwc(int dt, const ConvShape& s, const void* x, const void* w, const float* bias, void* y,
                         int relu, const FwdWs& o, hipStream_t st, bool x_s2d = false) {
  ConvShape g;
  const Rewrite rw = input_rewrite(s, dt, &g);
  if (rw == RW_NONE) return launch_conv_fwd(dt, s, x, w, bias, y, relu, 0, conv_flops(s), o.partial, nullptr, st);
  hipError_t e;
  if (rw == RW_PAD) {
    e = launch_pad_channels(dt, x, o.xp, (long)s.N * s.H * s.W, s.C, g.C, st);
    if (e == hipSuccess) e = launch_pad_channels(dt, w, o.wp, (long)s.K * s.R * s.S, s.C, g.C, st);
  } else {
    e = x_s2d ? hipSuccess : launch_space_to_depth(dt, s, g, x, o.xp, st);
    if (e == hipSuccess) e = launch_filter_to_s2d(dt, s, g, w, o.wp, st);
  }
  if (e == hipSuccess)
    e = launch_conv_fwd(dt, g, x_s2d ? x : o.xp, o.wp, bias, y, relu, 0, conv_flops(s), o.partial, nullptr, st);
  return e;
}

size_t carve_bwd_data(const ConvShape& s, int dt, int layout, void* ws, BwdDataWs* o) {
  Carve c(ws);
  o->dy = o->w = o->wt = o->dx = o->ws = o->dxs = nullptr;
  o->partial = nullptr;
  if (layout == SINGA_NCHW) {
    o->dy = c.take(out_bytes(s, dt));
    o->w = c.take(filt_bytes(s, dt));
    o->dx = c.take(act_bytes(s, dt));
  }
  ConvShape g;
  if (bwd_data_gemm(s)) {
    o->wt = c.take(filt_bytes(s, dt));
    const size_t pb = fwd_partial_bytes(bwd_data_inner(s), dt);
    if (pb) o->partial = (float*)c.take(pb);
  } else if (bwd_data_s2d(s, &g)) {
    o->ws = c.take(filt_bytes(g, dt));
    o->wt = c.take(filt_bytes(g, dt));
    o->dxs = c.take(act_bytes(g, dt));
    const size_t pb = fwd_partial_bytes(bwd_data_inner(g), dt);
    if (pb) o->partial = (float*)c.take(pb);
  }
  return c.used;
}

size_t carve_bwd_filter(const ConvShape& s, int dt, int layout, bool bias, void* ws, BwdFilterWs* o) {
  Carve c(ws);
  o->x = o->dy = o->xp = nullptr;
  o->dw = o->dwp = nullptr;
  if (layout == SINGA_NCHW) {
    o->x = c.take(act_bytes(s, dt));
    o->dy = c.take(out_bytes(s, dt));
    o->dw = (float*)c.take((size_t)s.K * s.R * s.S * s.C * sizeof(float));
  }
  ConvShape g;
  if (input_rewrite(s, dt, &g) != RW_NONE) {
    if (layout != SINGA_NHWC_S2D) o->xp = c.take((size_t)g.N * g.H * g.W * g.C * dt_size(dt));
    o->dwp = (float*)c.take((size_t)g.K * g.R * g.S * g.C * sizeof(float));
  }
  const size_t pb = wgrad_partial_bytes(g, dt, bias);
  o->partial = pb ? (float*)c.take(pb) : nullptr;
  return c.used;
}

// Filter gradient with the update: nothing when the update is fused into the
// gradient kernel; otherwise fp32 staging for the gradient (used when the
// caller passes no dw / db) and the filter gradient's own workspace.
struct BwdFilterSgdWs {
  bool fused;
  float* g;
  float* gb;
  void* inner;
  size_t inner_bytes;
};

bool bwd_filter_sgd_fused(const ConvShape& s, int dt, int layout, bool bias) {
  ConvShape g;
  return layout == SINGA_NHWC && input_rewrite(s, dt, &g) == RW_NONE && wgrad_update_fusable(s, dt, bias);
}

size_t carve_bwd_filter_sgd(const ConvShape& s, int dt, int layout, bool bias, void* ws, BwdFilterSgdWs* o) {
  Carve c(ws);
  o->fused = bwd_filter_sgd_fused(s, dt, layout, bias);
  o->g = o->gb = nullptr;
  o->inner = nullptr;
  o->inner_bytes = 0;
  if (o->fused) return 0;
  o->g = (float*)c.take((size_t)s.K * s.R * s.S * s.C * sizeof(float));
  if (bias) o->gb = (float*)c.take((size_t)s.K * sizeof(float));
  BwdFilterWs f;
  o->inner_bytes = carve_bwd_filter(s, dt, layout, bias, nullptr, &f);
  o->inner = o->inner_bytes ? c.take(o->inner_bytes) : nullptr;
  return c.used;
}

// Filter KCRS (NCHW callers) -> KRSC.
hipError_t kcrs_to_krsc(int dt, const ConvShape& s, const void* in, void* out, hipStream_t st) {
  const int RS = s.R * s.S;
  return launch_transpose(dt, in, out, s.K, s.C, RS, (long)s.C * RS, RS, (long)RS * s.C, s.C, 0, st);
}

}  // namespace

extern "C" {

const char* singa_strerror(int status) {
  switch (status) {
    case SINGA_OK: return "ok";
    case SINGA_ERR_NULL: return "a required pointer argument is NULL";
    case SINGA_ERR_SHAPE: return "non-positive or inconsistent sizes";
    case SINGA_ERR_UNSUPPORTED: return "unsupported dtype, layout or parameter combination";
    case SINGA_ERR_WORKSPACE: return "workspace too small";
    case SINGA_ERR_ALIGN: return "device pointer not aligned";
    case SINGA_ERR_HIP: return "HIP runtime error at launch";
    case SINGA_ERR_SCRATCH: return "needs more scratch than the library's fixed scratch array holds";
    default: return "unknown status";
  }
}

int singa_conv_out_shape(const singa_shape4* x, const singa_filter4* w, const singa_conv_desc* d, singa_shape4* y) {
  if (!y) return SINGA_ERR_NULL;
  ConvShape s;
  int rc = conv_geometry(x, w, d, &s);
  if (rc != SINGA_OK) return rc;
  y->n = s.N; y->c = s.K; y->h = s.P; y->w = s.Q;
  return SINGA_OK;
}

int singa_pool_out_shape(const singa_shape4* x, const singa_pool_desc* d, singa_shape4* y) {
  if (!x || !d || !y) return SINGA_ERR_NULL;
  if (x->n <= 0 || x->c <= 0 || x->h <= 0 || x->w <= 0) return SINGA_ERR_SHAPE;
  if (d->mode != SINGA_POOL_MAX && d->mode != SINGA_POOL_AVG) return SINGA_ERR_UNSUPPORTED;
  if (d->kh <= 0 || d->kw <= 0 || d->stride_h < 1 || d->stride_w < 1 || d->pad_h < 0 || d->pad_w < 0)
    return SINGA_ERR_SHAPE;
  if (d->kh * d->kw > 256 || d->pad_h >= d->kh || d->pad_w >= d->kw) return SINGA_ERR_UNSUPPORTED;
  long long out[2];
  const long long in[2] = {x->h, x->w}, k[2] = {d->kh, d->kw}, p[2] = {d->pad_h, d->pad_w},
                  st[2] = {d->stride_h, d->stride_w};
  for (int a = 0; a < 2; ++a) {
    const long long span = in[a] + 2 * p[a] - k[a];
    if (span < 0) return SINGA_ERR_SHAPE;
    if (d->ceil_mode) {
      out[a] = (span + st[a] - 1) / st[a] + 1;
      if (p[a] > 0 && (out[a] - 1) * st[a] >= in[a] + p[a]) out[a] -= 1;
    } else {
      out[a] = span / st[a] + 1;
    }
  }
  if (!fits_i32((long long)x->n * x->c * x->h * x->w) || !fits_i32((long long)x->n * x->c * out[0] * out[1]))
    return SINGA_ERR_UNSUPPORTED;
  y->n = x->n; y->c = x->c; y->h = (int)out[0]; y->w = (int)out[1];
  return SINGA_OK;
}

int singa_conv_workspace_bytes(int op, singa_dtype dtype, singa_layout layout, const singa_shape4* x,
                               const singa_filter4* w, const singa_conv_desc* d, size_t* bytes) {
  if (!bytes) return SINGA_ERR_NULL;
  if (!dtype_ok(dtype) || !(layout_ok(layout) || layout == SINGA_NHWC_S2D)) return SINGA_ERR_UNSUPPORTED;
  ConvShape s;
  int rc = conv_geometry(x, w, d, &s);
  if (rc != SINGA_OK) return rc;
  if (layout == SINGA_NHWC_S2D && !(s2d_input_ok(s, dtype) && (op == SINGA_OP_FWD || op == SINGA_OP_BWD_FILTER)))
    return SINGA_ERR_UNSUPPORTED;
  switch (op) {
    case SINGA_OP_FWD: { FwdWs o; *bytes = carve_fwd(s, dtype, layout, nullptr, &o); break; }
    case SINGA_OP_BWD_DATA: { BwdDataWs o; *bytes = carve_bwd_data(s, dtype, layout, nullptr, &o); break; }
    case SINGA_OP_BWD_FILTER: { BwdFilterWs o; *bytes = carve_bwd_filter(s, dtype, layout, true, nullptr, &o); break; }
    case SINGA_OP_BWD_FILTER_SGD: {
      BwdFilterSgdWs o;
      *bytes = carve_bwd_filter_sgd(s, dtype, layout, true, nullptr, &o);
      break;
    }
    default: return SINGA_ERR_UNSUPPORTED;
  }
  return SINGA_OK;
}

int singa_space_to_depth_bytes(singa_dtype dtype, const singa_shape4* x, const singa_filter4* w,
                               const singa_conv_desc* d, size_t* bytes) {
  if (!bytes) return SINGA_ERR_NULL;
  if (!dtype_ok(dtype)) return SINGA_ERR_UNSUPPORTED;
  ConvShape s;
  int rc = conv_geometry(x, w, d, &s);
  if (rc != SINGA_OK) return rc;
  ConvShape g;
  *bytes = input_rewrite(s, dtype, &g) == RW_S2D ? (size_t)g.N * g.H * g.W * g.C * dt_size(dtype) : 0;
  return SINGA_OK;
}

int singa_space_to_depth(singa_dtype dtype, const singa_shape4* x, const void* x_ptr, const singa_filter4* w,
                         const singa_conv_desc* d, void* xs_ptr, singa_stream stream) {
  if (!dtype_ok(dtype)) return SINGA_ERR_UNSUPPORTED;
  ConvShape s;
  int rc = conv_geometry(x, w, d, &s);
  if (rc != SINGA_OK) return rc;
  ConvShape g;
  if (input_rewrite(s, dtype, &g) != RW_S2D) return SINGA_ERR_UNSUPPORTED;
  if (!x_ptr || !xs_ptr) return SINGA_ERR_NULL;
  if (!aligned_to(x_ptr, dt_size(dtype)) || !aligned_to(xs_ptr, 16)) return SINGA_ERR_ALIGN;
  return hip_status(launch_space_to_depth(dtype, s, g, x_ptr, xs_ptr, (hipStream_t)stream));
}

int singa_conv_fwd(singa_dtype dtype, singa_layout layout, const singa_shape4* x, const void* x_ptr,
                   const singa_filter4* w, const void* w_ptr, const float* bias, const singa_conv_desc* d,
                   void* y_ptr, int fuse_relu, void* ws, size_t ws_bytes, singa_stream stream) {
  if (!dtype_ok(dtype) || !(layout_ok(layout) || layout == SINGA_NHWC_S2D)) return SINGA_ERR_UNSUPPORTED;
  ConvShape s;
  int rc = conv_geometry(x, w, d, &s);
  if (rc != SINGA_OK) return rc;
  if (layout == SINGA_NHWC_S2D && !s2d_input_ok(s, dtype)) return SINGA_ERR_UNSUPPORTED;
  if (!x_ptr || !w_ptr || !y_ptr) return SINGA_ERR_NULL;
  const size_t es = dt_size(dtype);
  if (!aligned_to(x_ptr, es) || !aligned_to(w_ptr, es) || !aligned_to(y_ptr, es) || !aligned_to(bias, 4) ||
      !aligned_to(ws, 16))
    return SINGA_ERR_ALIGN;
  FwdWs o;
  const size_t need = carve_fwd(s, dtype, layout, nullptr, &o);
  if (need > 0 && (!ws || ws_bytes < need)) return SINGA_ERR_WORKSPACE;
  carve_fwd(s, dtype, layout, ws, &o);
  hipStream_t st = (hipStream_t)stream;
  if (layout != SINGA_NCHW)
    return hip_status(conv_fwd_nhwc(dtype, s, x_ptr, w_ptr, bias, y_ptr, fuse_relu, o, st, layout == SINGA_NHWC_S2D));
  hipError_t e = launch_nchw_to_nhwc(dtype, x_ptr, o.x, s.N, s.C, s.H, s.W, st);
  if (e == hipSuccess) e = kcrs_to_krsc(dtype, s, w_ptr, o.w, st);
  if (e == hipSuccess) e = conv_fwd_nhwc(dtype, s, o.x, o.w, bias, o.y, fuse_relu, o, st);
  if (e == hipSuccess) e = launch_nhwc_to_nchw(dtype, o.y, y_ptr, s.N, s.K, s.P, s.Q, st);
  return hip_status(e);
}

int singa_conv_bwd_data(singa_dtype dtype, singa_layout layout, const singa_shape4* x, const singa_filter4* w,
                        const void* w_ptr, const singa_conv_desc* d, const void* dy_ptr, const void* relu_y,
                        void* dx_ptr, void* ws, size_t ws_bytes, singa_stream stream) {
  if (!dtype_ok(dtype) || !layout_ok(layout)) return SINGA_ERR_UNSUPPORTED;
  ConvShape s;
  int rc = conv_geometry(x, w, d, &s);
  if (rc != SINGA_OK) return rc;
  if (!w_ptr || !dy_ptr || !dx_ptr) return SINGA_ERR_NULL;
  const size_t es = dt_size(dtype);
  if (!aligned_to(w_ptr, es) || !aligned_to(dy_ptr, es) || !aligned_to(dx_ptr, es) || !aligned_to(ws, 16) ||
      !aligned_to(relu_y, es))
    return SINGA_ERR_ALIGN;
  // NCHW applies the ReLU mask with the vectorized ReLU-backward kernel
  if (relu_y && layout == SINGA_NCHW && (!aligned_to(relu_y, 16) || !aligned_to(dx_ptr, 16)))
    return SINGA_ERR_ALIGN;
  BwdDataWs o;
  const size_t need = carve_bwd_data(s, dtype, layout, nullptr, &o);
  if (need > 0 && (!ws || ws_bytes < need)) return SINGA_ERR_WORKSPACE;
  carve_bwd_data(s, dtype, layout, ws, &o);
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = hipSuccess;
  const void* dy = dy_ptr;
  const void* wk = w_ptr;  // KRSC filter
  void* dx = dx_ptr;
  const void* nhwc_mask = layout == SINGA_NHWC ? relu_y : nullptr;  // folded into the producing kernel
  if (layout == SINGA_NCHW) {
    e = launch_nchw_to_nhwc(dtype, dy_ptr, o.dy, s.N, s.K, s.P, s.Q, st);
    if (e == hipSuccess) e = kcrs_to_krsc(dtype, s, w_ptr, o.w, st);
    dy = o.dy;
    wk = o.w;
    dx = o.dx;
  }
  const int RS = s.R * s.S;
  ConvShape g;
  if (e == hipSuccess) {
    if (!bwd_data_gemm(s) && bwd_data_s2d(s, &g)) {
      // wt[c'][r'][s'][k] = w'[k][R'-1-r'][S'-1-s'][c'] of the space-to-depth layer g
      const int RSg = g.R * g.S;
      e = launch_filter_to_s2d(dtype, s, g, wk, o.ws, st);
      if (e == hipSuccess)
        e = launch_transpose(dtype, o.ws, o.wt, RSg, g.K, g.C, g.C, (long)RSg * g.C, g.K, (long)RSg * g.K, 1, st);
      if (e == hipSuccess)
        e = launch_conv_fwd(dtype, bwd_data_inner(g), dy, o.wt, nullptr, o.dxs, 0, 1, conv_flops(s), o.partial,
                            nullptr, st);
      if (e == hipSuccess) e = launch_depth_to_space(dtype, s, g, o.dxs, nhwc_mask, dx, st);
    } else if (bwd_data_gemm(s)) {
      // dense geometry: the GEMM reads w itself as the transposed filter when it can
      e = bwd_data_fc(s) ? launch_conv_fwd_wt(dtype, bwd_data_inner(s), dy, wk, dx, 1, conv_flops(s), o.partial,
                                              nhwc_mask, st)
                         : hipErrorNotSupported;
      if (e == hipErrorNotSupported) {
        if (bwd_data_fc(s)) {
          const int J = RS * s.C;  // wt[(r,s,c)][k] = w[k][(r,s,c)]
          e = launch_transpose(dtype, wk, o.wt, 1, s.K, J, 0, J, 0, s.K, 0, st);
        } else {  // wt[c][r'][s'][k] = w[k][R-1-r'][S-1-s'][c]
          e = launch_transpose(dtype, wk, o.wt, RS, s.K, s.C, s.C, (long)RS * s.C, s.K, (long)RS * s.K, 1, st);
        }
        if (e == hipSuccess)
          e = launch_conv_fwd(dtype, bwd_data_inner(s), dy, o.wt, nullptr, dx, 0, 1, conv_flops(s), o.partial,
                              nhwc_mask, st);
      }
    } else {
      e = launch_conv_bwd_data_direct(dtype, s, dy, wk, dx, nhwc_mask, st);
    }
  }
  if (e == hipSuccess && layout == SINGA_NCHW) {
    e = launch_nhwc_to_nchw(dtype, dx, dx_ptr, s.N, s.C, s.H, s.W, st);
    if (e == hipSuccess && relu_y) e = launch_relu_bwd(dtype, act_bytes(s, dtype) / es, relu_y, dx_ptr, dx_ptr, st);
  }
  return hip_status(e);
}

int singa_conv_bwd_filter(singa_dtype dtype, singa_layout layout, const singa_shape4* x, const void* x_ptr,
                          const singa_filter4* w, const singa_conv_desc* d, const void* dy_ptr, float* dw,
                          float* db, int accumulate, void* ws, size_t ws_bytes, singa_stream stream) {
  if (!dtype_ok(dtype) || !(layout_ok(layout) || layout == SINGA_NHWC_S2D)) return SINGA_ERR_UNSUPPORTED;
  ConvShape s;
  int rc = conv_geometry(x, w, d, &s);
  if (rc != SINGA_OK) return rc;
  if (layout == SINGA_NHWC_S2D && !s2d_input_ok(s, dtype)) return SINGA_ERR_UNSUPPORTED;
  if (!x_ptr || !dy_ptr || !dw) return SINGA_ERR_NULL;
  const size_t es = dt_size(dtype);
  if (!aligned_to(x_ptr, es) || !aligned_to(dy_ptr, es) || !aligned_to(dw, 4) || !aligned_to(db, 4) ||
      !aligned_to(ws, 16))
    return SINGA_ERR_ALIGN;
  BwdFilterWs o;
  const bool bias = db != nullptr;
  const size_t need = carve_bwd_filter(s, dtype, layout, bias, nullptr, &o);
  if (need > 0 && (!ws || ws_bytes < need)) return SINGA_ERR_WORKSPACE;
  carve_bwd_filter(s, dtype, layout, bias, ws, &o);
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = hipSuccess;
  const void* xx = x_ptr;
  const void* dy = dy_ptr;
  if (layout == SINGA_NCHW) {
    e = launch_nchw_to_nhwc(dtype, x_ptr, o.x, s.N, s.C, s.H, s.W, st);
    if (e == hipSuccess) e = launch_nchw_to_nhwc(dtype, dy_ptr, o.dy, s.N, s.K, s.P, s.Q, st);
    xx = o.x;
    dy = o.dy;
  }
  // g: the GEMM's geometry (input rewritten when input_rewrite says so)
  ConvShape g;
  const Rewrite rw = input_rewrite(s, dtype, &g);
  if (rw == RW_PAD && e == hipSuccess) e = launch_pad_channels(dtype, xx, o.xp, (long)s.N * s.H * s.W, s.C, g.C, st);
  if (rw == RW_S2D && e == hipSuccess && layout != SINGA_NHWC_S2D) e = launch_space_to_depth(dtype, s, g, xx, o.xp, st);
  if (rw != RW_NONE && layout != SINGA_NHWC_S2D) xx = o.xp;
  float* krsc = layout != SINGA_NCHW ? dw : o.dw;  // KRSC result
  const int acc = layout != SINGA_NCHW ? accumulate : 0;
  float* target = rw != RW_NONE ? o.dwp : krsc;  // the GEMM's (K, g.R, g.S, g.C) result
  const int tacc = rw != RW_NONE ? 0 : acc;
  // db is written in place by the GEMM's bias column, with the caller's accumulate
  if (e == hipSuccess)
    e = launch_conv_wgrad(dtype, g, xx, dy, o.partial, target, db, tacc, accumulate, conv_flops(s), st);
  if (e == hipSuccess && rw == RW_PAD)
    e = launch_unpad_channels_f32(o.dwp, krsc, (long)s.K * s.R * s.S, g.C, s.C, acc, st);
  if (e == hipSuccess && rw == RW_S2D) e = launch_s2d_to_filter_f32(s, g, o.dwp, krsc, acc, st);
  if (e == hipSuccess && layout == SINGA_NCHW) e = launch_krsc_to_kcrs_f32(o.dw, dw, s.K, s.C, s.R, s.S, accumulate, st);
  return hip_status(e);
}

int singa_conv_bwd_filter_sgd(singa_dtype dtype, singa_layout layout, const singa_shape4* x, const void* x_ptr,
                              const singa_filter4* w, const singa_conv_desc* d, const void* dy_ptr, float* dw,
                              float* db, float* w_master, float* w_mom, uint16_t* w_bf16, float* b_master,
                              float* b_mom, uint16_t* b_bf16, float lr, float momentum, float weight_decay,
                              void* ws, size_t ws_bytes, singa_stream stream) {
  if (!dtype_ok(dtype) || !layout_ok(layout)) return SINGA_ERR_UNSUPPORTED;
  ConvShape s;
  int rc = conv_geometry(x, w, d, &s);
  if (rc != SINGA_OK) return rc;
  if (!x_ptr || !dy_ptr || !w_master || !w_mom || (b_master == nullptr) != (b_mom == nullptr)) return SINGA_ERR_NULL;
  if (b_bf16 && !b_master) return SINGA_ERR_NULL;
  const size_t es = dt_size(dtype);
  if (!aligned_to(x_ptr, es) || !aligned_to(dy_ptr, es) || !aligned_to(dw, 4) || !aligned_to(db, 4) ||
      !aligned_to(w_master, 16) || !aligned_to(w_mom, 16) || !aligned_to(w_bf16, 16) || !aligned_to(b_master, 16) ||
      !aligned_to(b_mom, 16) || !aligned_to(b_bf16, 16) || !aligned_to(ws, 16))
    return SINGA_ERR_ALIGN;
  const bool bias = b_master != nullptr;
  BwdFilterSgdWs o;
  const size_t need = carve_bwd_filter_sgd(s, dtype, layout, bias, nullptr, &o);
  if (need > 0 && (!ws || ws_bytes < need)) return SINGA_ERR_WORKSPACE;
  carve_bwd_filter_sgd(s, dtype, layout, bias, ws, &o);
  hipStream_t st = (hipStream_t)stream;
  if (o.fused) {
    if (!aligned_to(x_ptr, 16) || !aligned_to(dy_ptr, 16)) return SINGA_ERR_ALIGN;
    const SgdTargets u{w_master, w_mom, w_bf16, b_master, b_mom, b_bf16, lr, momentum, weight_decay};
    return hip_status(launch_conv_wgrad_sgd(dtype, s, x_ptr, dy_ptr, dw, db, u, st));
  }
  // a split reduction applies the step to each summed element (NHWC input
  // taken as it is); otherwise the gradient, then the flat update
  ConvShape g0;
  if (layout == SINGA_NHWC && input_rewrite(s, dtype, &g0) == RW_NONE) {
    BwdFilterWs f;
    carve_bwd_filter(s, dtype, layout, bias, o.inner, &f);
    const SgdTargets u{w_master, w_mom, w_bf16, b_master, b_mom, b_bf16, lr, momentum, weight_decay};
    const hipError_t e = launch_conv_wgrad_reduce_sgd(dtype, s, x_ptr, dy_ptr, f.partial, dw, db, u, conv_flops(s), st);
    if (e != hipErrorNotSupported) return hip_status(e);
  }
  float* g = dw ? dw : o.g;
  float* gb = bias ? (db ? db : o.gb) : nullptr;
  rc = singa_conv_bwd_filter(dtype, layout, x, x_ptr, w, d, dy_ptr, g, gb, 0, o.inner, o.inner_bytes, stream);
  if (rc != SINGA_OK) return rc;
  hipError_t e = launch_sgd((size_t)s.K * s.R * s.S * s.C, w_master, g, w_mom, w_bf16, lr, momentum, weight_decay, st);
  if (e == hipSuccess && bias) e = launch_sgd((size_t)s.K, b_master, gb, b_mom, b_bf16, lr, momentum, weight_decay, st);
  return hip_status(e);
}

int singa_pool_fwd(singa_dtype dtype, singa_layout layout, const singa_shape4* x, const void* x_ptr,
                   const singa_pool_desc* d, void* y_ptr, uint8_t* argmax, singa_stream stream) {
  if (!dtype_ok(dtype) || !layout_ok(layout)) return SINGA_ERR_UNSUPPORTED;
  singa_shape4 y;
  int rc = singa_pool_out_shape(x, d, &y);
  if (rc != SINGA_OK) return rc;
  if (!x_ptr || !y_ptr || (d->mode == SINGA_POOL_MAX && !argmax)) return SINGA_ERR_NULL;
  const size_t es = dt_size(dtype);
  if (!aligned_to(x_ptr, es) || !aligned_to(y_ptr, es)) return SINGA_ERR_ALIGN;
  uint8_t* am = d->mode == SINGA_POOL_MAX ? argmax : nullptr;
  return hip_status(launch_pool_fwd(dtype, d->mode, x->n, x->c, x->h, x->w, y.h, y.w, d->kh, d->kw, d->stride_h,
                                    d->stride_w, d->pad_h, d->pad_w, x_ptr, y_ptr, am, layout == SINGA_NCHW,
                                    (hipStream_t)stream));
}

int singa_pool_bwd(singa_dtype dtype, singa_layout layout, const singa_shape4* x, const singa_pool_desc* d,
                   const void* dy_ptr, const uint8_t* argmax, const void* relu_y, void* dx_ptr,
                   singa_stream stream) {
  if (!dtype_ok(dtype) || !layout_ok(layout)) return SINGA_ERR_UNSUPPORTED;
  singa_shape4 y;
  int rc = singa_pool_out_shape(x, d, &y);
  if (rc != SINGA_OK) return rc;
  if (!dy_ptr || !dx_ptr || (d->mode == SINGA_POOL_MAX && !argmax)) return SINGA_ERR_NULL;
  if (relu_y && d->mode != SINGA_POOL_MAX) return SINGA_ERR_UNSUPPORTED;
  const size_t es = dt_size(dtype);
  if (!aligned_to(dy_ptr, es) || !aligned_to(dx_ptr, es) || !aligned_to(relu_y, es)) return SINGA_ERR_ALIGN;
  return hip_status(launch_pool_bwd(dtype, d->mode, x->n, x->c, x->h, x->w, y.h, y.w, d->kh, d->kw, d->stride_h,
                                    d->stride_w, d->pad_h, d->pad_w, dy_ptr, argmax, relu_y, dx_ptr,
                                    layout == SINGA_NCHW, (hipStream_t)stream));
}

int singa_relu_fwd(singa_dtype dtype, size_t n, const void* x, void* y, singa_stream stream) {
  if (!dtype_ok(dtype)) return SINGA_ERR_UNSUPPORTED;
  if (n == 0) return SINGA_OK;
  if (!x || !y) return SINGA_ERR_NULL;
  if (!aligned_to(x, 16) || !aligned_to(y, 16)) return SINGA_ERR_ALIGN;
  return hip_status(launch_relu_fwd(dtype, n, x, y, (hipStream_t)stream));
}

int singa_relu_bwd(singa_dtype dtype, size_t n, const void* y, const void* dy, void* dx, singa_stream stream) {
  if (!dtype_ok(dtype)) return SINGA_ERR_UNSUPPORTED;
  if (n == 0) return SINGA_OK;
  if (!y || !dy || !dx) return SINGA_ERR_NULL;
  if (!aligned_to(y, 16) || !aligned_to(dy, 16) || !aligned_to(dx, 16)) return SINGA_ERR_ALIGN;
  return hip_status(launch_relu_bwd(dtype, n, y, dy, dx, (hipStream_t)stream));
}

int singa_softmax_ce(singa_dtype dtype, int batch, int classes, const void* logits, const int32_t* labels,
                     float* loss, void* dlogits, singa_stream stream) {
  if (!dtype_ok(dtype)) return SINGA_ERR_UNSUPPORTED;
  if (batch <= 0 || classes <= 0 || !fits_i32((long long)batch * classes)) return SINGA_ERR_SHAPE;
  if (!logits || !labels || !loss || !dlogits) return SINGA_ERR_NULL;
  const size_t es = dt_size(dtype);
  if (!aligned_to(logits, es) || !aligned_to(dlogits, es) || !aligned_to(labels, 4) || !aligned_to(loss, 4))
    return SINGA_ERR_ALIGN;
  return hip_status(launch_softmax_ce(dtype, batch, classes, logits, labels, loss, dlogits, (hipStream_t)stream));
}

static int lrn_check(singa_dtype dtype, singa_layout layout, const singa_shape4* x, const singa_lrn_desc* d) {
  if (!x || !d) return SINGA_ERR_NULL;
  if (!dtype_ok(dtype) || !layout_ok(layout)) return SINGA_ERR_UNSUPPORTED;
  if (x->n <= 0 || x->c <= 0 || x->h <= 0 || x->w <= 0) return SINGA_ERR_SHAPE;
  if (!fits_i32((long long)x->n * x->c * x->h * x->w)) return SINGA_ERR_UNSUPPORTED;
  if (d->size < 1 || !(d->alpha >= 0.f) || !(d->k > 0.f) || !(d->beta == d->beta)) return SINGA_ERR_UNSUPPORTED;
  return SINGA_OK;
}

int singa_lrn_fwd(singa_dtype dtype, singa_layout layout, const singa_shape4* x, const void* x_ptr,
                  const singa_lrn_desc* d, void* y_ptr, singa_stream stream) {
  int rc = lrn_check(dtype, layout, x, d);
  if (rc != SINGA_OK) return rc;
  if (!x_ptr || !y_ptr) return SINGA_ERR_NULL;
  const size_t es = dt_size(dtype);
  if (!aligned_to(x_ptr, es) || !aligned_to(y_ptr, es)) return SINGA_ERR_ALIGN;
  return hip_status(launch_lrn(dtype, 0, x->n, x->c, x->h * x->w, d->size, d->alpha, d->beta, d->k, x_ptr, nullptr,
                               y_ptr, layout == SINGA_NCHW, (hipStream_t)stream));
}

int singa_lrn_bwd(singa_dtype dtype, singa_layout layout, const singa_shape4* x, const void* x_ptr,
                  const void* dy_ptr, const singa_lrn_desc* d, void* dx_ptr, singa_stream stream) {
  int rc = lrn_check(dtype, layout, x, d);
  if (rc != SINGA_OK) return rc;
  if (!x_ptr || !dy_ptr || !dx_ptr) return SINGA_ERR_NULL;
  const size_t es = dt_size(dtype);
  if (!aligned_to(x_ptr, es) || !aligned_to(dy_ptr, es) || !aligned_to(dx_ptr, es)) return SINGA_ERR_ALIGN;
  return hip_status(launch_lrn(dtype, 1, x->n, x->c, x->h * x->w, d->size, d->alpha, d->beta, d->k, x_ptr, dy_ptr,
                               dx_ptr, layout == SINGA_NCHW, (hipStream_t)stream));
}

int singa_adagrad_update(size_t n, float* w, const float* g, float* h, uint16_t* w_bf16, float lr, float delta,
                         float weight_decay, singa_stream stream) {
  if (n == 0) return SINGA_OK;
  if (!w || !g || !h) return SINGA_ERR_NULL;
  if (!aligned_to(w, 16) || !aligned_to(g, 16) || !aligned_to(h, 16) || !aligned_to(w_bf16, 16))
    return SINGA_ERR_ALIGN;
  if (!(delta > 0.f) || !(lr >= 0.f)) return SINGA_ERR_UNSUPPORTED;
  return hip_status(launch_adagrad(n, w, g, h, w_bf16, lr, delta, weight_decay, (hipStream_t)stream));
}

int singa_sgd_momentum_update(size_t n, float* w, const float* g, float* v, uint16_t* w_bf16, float lr,
                              float momentum, float weight_decay, singa_stream stream) {
  if (n == 0) return SINGA_OK;
  if (!w || !g || !v) return SINGA_ERR_NULL;
  if (!aligned_to(w, 16) || !aligned_to(g, 16) || !aligned_to(v, 16) || !aligned_to(w_bf16, 16))
    return SINGA_ERR_ALIGN;
  return hip_status(launch_sgd(n, w, g, v, w_bf16, lr, momentum, weight_decay, (hipStream_t)stream));
}

}  // extern "C"
