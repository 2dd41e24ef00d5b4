// eltwise.hip -- bandwidth-bound layers of the hot path: pooling (max/avg,
// forward and gather-style backward), ReLU, softmax cross-entropy and the
// fused SGD-momentum Updater.
#include "common.h"
#include "internal.h"

namespace singa {

namespace {

template <typename T> __device__ __forceinline__ float ld_f(const T* p);
template <> __device__ __forceinline__ float ld_f<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float ld_f<bf16_t>(const bf16_t* p) { return bf16_to_f32(*p); }

template <typename T> __device__ __forceinline__ void st_f(T* p, float v);
template <> __device__ __forceinline__ void st_f<float>(float* p, float v) { *p = v; }
template <> __device__ __forceinline__ void st_f<bf16_t>(bf16_t* p, float v) { *p = f32_to_bf16(v); }

// 16 bytes <-> VEC floats (bf16: 8, fp32: 4) without taking a local's address
template <typename T> __device__ __forceinline__ void unpack16(const uint4& u, float* f);
template <> __device__ __forceinline__ void unpack16<bf16_t>(const uint4& u, float* f) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
template <> __device__ __forceinline__ void unpack16<float>(const uint4& u, float* f) {
  f[0] = __uint_as_float(u.x); f[1] = __uint_as_float(u.y); f[2] = __uint_as_float(u.z); f[3] = __uint_as_float(u.w);
}
template <typename T> __device__ __forceinline__ uint4 pack16(const float* f);
template <> __device__ __forceinline__ uint4 pack16<bf16_t>(const float* f) {
  return make_uint4(f32x2_to_bf16x2(f[0], f[1]), f32x2_to_bf16x2(f[2], f[3]), f32x2_to_bf16x2(f[4], f[5]),
                    f32x2_to_bf16x2(f[6], f[7]));
}
template <> __device__ __forceinline__ uint4 pack16<float>(const float* f) {
  return make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]), __float_as_uint(f[3]));
}

unsigned grid_for(size_t total, int block = 256, size_t cap = 1 << 20) {
  size_t g = (total + block - 1) / block;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return (unsigned)g;
}

struct PoolGeom {
  int N, C, H, W, P, Q, kh, kw, sh, sw, ph, pw;
};

// Element offset of (n, c, h, w) in either layout.
template <bool NCHW>
__device__ __forceinline__ long off4(const PoolGeom& g, int n, int c, int h, int w, int HH, int WW) {
  if (NCHW) return (((long)n * g.C + c) * HH + h) * WW + w;
  return (((long)n * HH + h) * WW + w) * g.C + c;
}

// Window size after clipping it to the padded extent [-pad, H+pad).
__device__ __forceinline__ int pool_divisor(const PoolGeom& g, int p, int q) {
  const int h0 = p * g.sh - g.ph, w0 = q * g.sw - g.pw;
  const int h1 = min(h0 + g.kh, g.H + g.ph), w1 = min(w0 + g.kw, g.W + g.pw);
  return (h1 - h0) * (w1 - w0);
}

template <typename T, bool NCHW>
__global__ __launch_bounds__(256) void pool_fwd_kernel(PoolGeom g, int mode, const T* __restrict__ x,
                                                       T* __restrict__ y, uint8_t* __restrict__ argmax, long total) {
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (long)gridDim.x * blockDim.x) {
    int n, c, p, q;
    if (NCHW) {
      q = (int)(i % g.Q);
      long t = i / g.Q;
      p = (int)(t % g.P);
      t /= g.P;
      c = (int)(t % g.C);
      n = (int)(t / g.C);
    } else {
      c = (int)(i % g.C);
      long t = i / g.C;
      q = (int)(t % g.Q);
      t /= g.Q;
      p = (int)(t % g.P);
      n = (int)(t / g.P);
    }
    const int h0 = p * g.sh - g.ph, w0 = q * g.sw - g.pw;
    if (mode == 0) {
      float best = 0.f;
      int cell = 0;
      bool found = false;
      for (int r = 0; r < g.kh; ++r) {
        const int h = h0 + r;
        if ((unsigned)h >= (unsigned)g.H) continue;
        for (int s = 0; s < g.kw; ++s) {
          const int w = w0 + s;
          if ((unsigned)w >= (unsigned)g.W) continue;
          const float v = ld_f<T>(x + off4<NCHW>(g, n, c, h, w, g.H, g.W));
          if (!found || v > best) {
            best = v;
            cell = r * g.kw + s;
            found = true;
          }
        }
      }
      st_f<T>(y + i, best);
      argmax[i] = (uint8_t)cell;
    } else {
      float acc = 0.f;
      for (int r = 0; r < g.kh; ++r) {
        const int h = h0 + r;
        if ((unsigned)h >= (unsigned)g.H) continue;
        for (int s = 0; s < g.kw; ++s) {
          const int w = w0 + s;
          if ((unsigned)w >= (unsigned)g.W) continue;
          acc += ld_f<T>(x + off4<NCHW>(g, n, c, h, w, g.H, g.W));
        }
      }
      st_f<T>(y + i, acc / (float)pool_divisor(g, p, q));
    }
  }
}

// Gather form of the pooling gradient: each input cell visits the windows
// that cover it (in window order) and takes what they route to it.
template <typename T, bool NCHW>
__global__ __launch_bounds__(256) void pool_bwd_kernel(PoolGeom g, int mode, const T* __restrict__ dy,
                                                       const uint8_t* __restrict__ argmax,
                                                       const T* __restrict__ ymask, T* __restrict__ dx,
                                                       long total) {
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (long)gridDim.x * blockDim.x) {
    int n, c, h, w;
    if (NCHW) {
      w = (int)(i % g.W);
      long t = i / g.W;
      h = (int)(t % g.H);
      t /= g.H;
      c = (int)(t % g.C);
      n = (int)(t / g.C);
    } else {
      c = (int)(i % g.C);
      long t = i / g.C;
      w = (int)(t % g.W);
      t /= g.W;
      h = (int)(t % g.H);
      n = (int)(t / g.H);
    }
    // windows p with p*sh - ph <= h < p*sh - ph + kh
    const int hn = h + g.ph - g.kh + 1, wn = w + g.pw - g.kw + 1;
    const int p_lo = hn <= 0 ? 0 : (hn + g.sh - 1) / g.sh;
    const int q_lo = wn <= 0 ? 0 : (wn + g.sw - 1) / g.sw;
    const int p_hi = min(g.P - 1, (h + g.ph) / g.sh);
    const int q_hi = min(g.Q - 1, (w + g.pw) / g.sw);
    float acc = 0.f;
    for (int p = p_lo; p <= p_hi; ++p) {
      for (int q = q_lo; q <= q_hi; ++q) {
        const long o = off4<NCHW>(g, n, c, p, q, g.P, g.Q);
        if (mode == 0) {
          const int cell = (h - (p * g.sh - g.ph)) * g.kw + (w - (q * g.sw - g.pw));
          if (argmax[o] == cell && (!ymask || ld_f<T>(ymask + o) > 0.f)) acc += ld_f<T>(dy + o);
        } else {
          acc += ld_f<T>(dy + o) / (float)pool_divisor(g, p, q);
        }
      }
    }
    st_f<T>(dx + i, acc);
  }
}

// NHWC pooling over 16-byte channel vectors: one thread per (output pixel,
// VEC consecutive channels).  Same window scan and first-maximum rule as the
// scalar kernel, applied per channel; the VEC argmax bytes are stored together.
// KS > 0: a KS x KS window known at compile time, whose KS^2 loads are all
// issued before the scan (cells outside the input load a clamped, in-bounds
// pixel and are skipped by the scan, which keeps the generic order); a max
// window wholly inside the input (every window of an unpadded floor-size
// pooling) takes cell 0 as its first maximum and compares the rest with no
// bounds or first-cell tests.  MODE: 0 max, 1 average.  A max output is one
// of the inputs, so bf16 results are repacked exactly from the high halves.
template <typename T, int VEC, int KS, int MODE>
__global__ __launch_bounds__(256) void pool_fwd_nhwc_vec_kernel(PoolGeom g, FastDiv dCV, FastDiv dQ, FastDiv dP,
                                                                const T* __restrict__ x, T* __restrict__ y,
                                                                uint8_t* __restrict__ argmax, int total) {
  const int CV = g.C / VEC;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    const int t1 = (int)fdiv((uint32_t)i, dCV);
    const int cv = i - t1 * CV;
    const int t2 = (int)fdiv((uint32_t)t1, dQ);
    const int q = t1 - t2 * g.Q;
    const int n = (int)fdiv((uint32_t)t2, dP);
    const int p = t2 - n * g.P;
    const int h0 = p * g.sh - g.ph, w0 = q * g.sw - g.pw;
    float best[VEC];
    int cell[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
      best[j] = 0.f;
      cell[j] = 0;
    }
    bool found = false;
    auto scan = [&](const uint4& u, int c) {
      float f[VEC];
      unpack16<T>(u, f);
#pragma unroll
      for (int j = 0; j < VEC; ++j) {
        if constexpr (MODE == 0) {
          if (!found || f[j] > best[j]) {
            best[j] = f[j];
            cell[j] = c;
          }
        } else {
          best[j] += f[j];
        }
      }
      found = true;
    };
    if constexpr (KS > 0) {
      uint4 v[KS * KS];
#pragma unroll
      for (int r = 0; r < KS; ++r)
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const int h = min(max(h0 + r, 0), g.H - 1), w = min(max(w0 + s, 0), g.W - 1);
          v[r * KS + s] = *(const uint4*)(x + ((n * g.H + h) * g.W + w) * g.C + cv * VEC);
        }
      const bool inside = h0 >= 0 && w0 >= 0 && h0 + KS <= g.H && w0 + KS <= g.W;
      if (MODE == 0 && inside) {
        unpack16<T>(v[0], best);
#pragma unroll
        for (int c = 1; c < KS * KS; ++c) {
          float f[VEC];
          unpack16<T>(v[c], f);
#pragma unroll
          for (int j = 0; j < VEC; ++j)
            if (f[j] > best[j]) {
              best[j] = f[j];
              cell[j] = c;
            }
        }
      } else {
#pragma unroll
        for (int r = 0; r < KS; ++r)
#pragma unroll
          for (int s = 0; s < KS; ++s)
            if ((unsigned)(h0 + r) < (unsigned)g.H && (unsigned)(w0 + s) < (unsigned)g.W) scan(v[r * KS + s], r * KS + s);
      }
    } else {
      for (int r = 0; r < g.kh; ++r) {
        const int h = h0 + r;
        if ((unsigned)h >= (unsigned)g.H) continue;
        for (int s = 0; s < g.kw; ++s) {
          const int w = w0 + s;
          if ((unsigned)w >= (unsigned)g.W) continue;
          scan(*(const uint4*)(x + ((n * g.H + h) * g.W + w) * g.C + cv * VEC), r * g.kw + s);
        }
      }
    }
    uint4 o;
    if constexpr (MODE == 0) {
      if constexpr (VEC == 8) {
        uint32_t d[4];
#pragma unroll
        for (int k = 0; k < 4; ++k)
          d[k] = (__float_as_uint(best[2 * k]) >> 16) | (__float_as_uint(best[2 * k + 1]) & 0xffff0000u);
        o = make_uint4(d[0], d[1], d[2], d[3]);
      } else {
        o = pack16<T>(best);
      }
    } else {
      const float inv = 1.f / (float)pool_divisor(g, p, q);
#pragma unroll
      for (int j = 0; j < VEC; ++j) best[j] *= inv;
      o = pack16<T>(best);
    }
    *(uint4*)(y + (size_t)i * VEC) = o;
    if constexpr (MODE == 0) {
      const uint32_t a0 = (uint32_t)cell[0] | (cell[1] << 8) | (cell[2] << 16) | ((uint32_t)cell[3] << 24);
      if constexpr (VEC == 8) {
        const uint32_t a1 = (uint32_t)cell[4] | (cell[5] << 8) | (cell[6] << 16) | ((uint32_t)cell[7] << 24);
        *(uint2*)(argmax + (size_t)i * VEC) = make_uint2(a0, a1);
      } else {
        *(uint32_t*)(argmax + (size_t)i * VEC) = a0;
      }
    }
  }
}

// One thread per (input pixel, VEC consecutive channels), 32-bit index math
// (every pooled tensor has fewer than 2^31 elements).
template <typename T, int VEC, bool MASK>
__global__ __launch_bounds__(256) void pool_bwd_nhwc_vec_kernel(PoolGeom g, FastDiv dCV, FastDiv dW, FastDiv dH,
                                                                int mode, const T* __restrict__ dy,
                                                                const uint8_t* __restrict__ argmax,
                                                                const T* __restrict__ ymask, T* __restrict__ dx,
                                                                int total) {
  const int CV = g.C / VEC;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    const int t1 = (int)fdiv((uint32_t)i, dCV);
    const int cv = i - t1 * CV;
    const int t2 = (int)fdiv((uint32_t)t1, dW);
    const int w = t1 - t2 * g.W;
    const int n = (int)fdiv((uint32_t)t2, dH);
    const int h = t2 - n * g.H;
    const int hn = h + g.ph - g.kh + 1, wn = w + g.pw - g.kw + 1;
    const int p_lo = hn <= 0 ? 0 : (hn + g.sh - 1) / g.sh;
    const int q_lo = wn <= 0 ? 0 : (wn + g.sw - 1) / g.sw;
    const int p_hi = min(g.P - 1, (h + g.ph) / g.sh);
    const int q_hi = min(g.Q - 1, (w + g.pw) / g.sw);
    float acc[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) acc[j] = 0.f;
    for (int p = p_lo; p <= p_hi; ++p) {
      for (int q = q_lo; q <= q_hi; ++q) {
        const int o = ((n * g.P + p) * g.Q + q) * g.C + cv * VEC;
        union { uint4 u; T e[VEC]; } v;
        v.u = *(const uint4*)(dy + o);
        if (mode == 0) {
          const int cell = (h - (p * g.sh - g.ph)) * g.kw + (w - (q * g.sw - g.pw));
          uint8_t am[VEC];
          if constexpr (VEC == 8) {
            const uint2 a = *(const uint2*)(argmax + o);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              am[j] = (uint8_t)(a.x >> (8 * j));
              am[4 + j] = (uint8_t)(a.y >> (8 * j));
            }
          } else {
            const uint32_t a = *(const uint32_t*)(argmax + o);
#pragma unroll
            for (int j = 0; j < 4; ++j) am[j] = (uint8_t)(a >> (8 * j));
          }
          union { uint4 u; T e[VEC]; } ym;
          if constexpr (MASK) ym.u = *(const uint4*)(ymask + o);
#pragma unroll
          for (int j = 0; j < VEC; ++j) {
            bool take = am[j] == cell;
            if constexpr (MASK) take = take && ld_f<T>(&ym.e[j]) > 0.f;
            if (take) acc[j] += ld_f<T>(&v.e[j]);
          }
        } else {
          const float inv = 1.f / (float)pool_divisor(g, p, q);
#pragma unroll
          for (int j = 0; j < VEC; ++j) acc[j] += ld_f<T>(&v.e[j]) * inv;
        }
      }
    }
    union { uint4 u; T e[VEC]; } out;
#pragma unroll
    for (int j = 0; j < VEC; ++j) st_f<T>(&out.e[j], acc[j]);
    *(uint4*)(dx + (size_t)i * VEC) = out.u;
  }
}

// Max pooling backward for 3x3 windows, stride 2, no padding (NHWC, VEC
// channels per thread): a thread owns the 2 x 2 input block (2 hb + dh,
// 2 wb + dw), which windows (hb - 1 .. hb) x (wb - 1 .. wb) cover, so each
// window's dy / arg-max / mask vectors are read once for four input pixels
// instead of once per pixel.  Same window order per pixel as the generic
// kernel: windows p ascending, then q ascending.
template <typename T, int VEC, bool MASK>
__global__ __launch_bounds__(256) void pool_bwd_k3s2_kernel(PoolGeom g, FastDiv dCV, FastDiv dWB, FastDiv dHB,
                                                            int HB, int WB, const T* __restrict__ dy,
                                                            const uint8_t* __restrict__ argmax,
                                                            const T* __restrict__ ymask, T* __restrict__ dx,
                                                            int total) {
  const int CV = g.C / VEC;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    const int t1 = (int)fdiv((uint32_t)i, dCV);
    const int cv = i - t1 * CV;
    const int t2 = (int)fdiv((uint32_t)t1, dWB);
    const int wb = t1 - t2 * WB;
    const int n = (int)fdiv((uint32_t)t2, dHB);
    const int hb = t2 - n * HB;
    // the four windows' vectors, all loaded before any is used; a window
    // outside the output gets arg-max cells 0xff, which match no input.  The
    // folded ReLU mask zeroes a window's gradient once per window (a value
    // that goes nowhere cannot change a sum), then each input pixel sums the
    // windows whose arg-max names it.
    float d[2][2][VEC];
    uint32_t am[2][2][VEC / 4];
#pragma unroll
    for (int pi = 0; pi < 2; ++pi)
#pragma unroll
      for (int qi = 0; qi < 2; ++qi) {
        const int p = hb - 1 + pi, q = wb - 1 + qi;
        const bool ok = p >= 0 && p < g.P && q >= 0 && q < g.Q;
        const int o = ok ? ((n * g.P + p) * g.Q + q) * g.C + cv * VEC : 0;
        uint4 vu = make_uint4(0u, 0u, 0u, 0u), mu = make_uint4(0u, 0u, 0u, 0u);
        if (ok) vu = *(const uint4*)(dy + o);
        if constexpr (MASK) {
          if (ok) mu = *(const uint4*)(ymask + o);
        }
        if constexpr (VEC == 8) {
          uint2 a2 = make_uint2(~0u, ~0u);
          if (ok) a2 = *(const uint2*)(argmax + o);
          am[pi][qi][0] = a2.x;
          am[pi][qi][VEC / 4 - 1] = a2.y;
        } else {
          uint32_t a1 = ~0u;
          if (ok) a1 = *(const uint32_t*)(argmax + o);
          am[pi][qi][0] = a1;
        }
        unpack16<T>(vu, d[pi][qi]);
        if constexpr (MASK) {
          float m[VEC];
          unpack16<T>(mu, m);
#pragma unroll
          for (int j = 0; j < VEC; ++j) d[pi][qi][j] = m[j] > 0.f ? d[pi][qi][j] : 0.f;
        }
      }
    float acc[2][2][VEC];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int j = 0; j < VEC; ++j) acc[a][b][j] = 0.f;
#pragma unroll
    for (int pi = 0; pi < 2; ++pi) {
#pragma unroll
      for (int qi = 0; qi < 2; ++qi) {
        // input (2 hb + dh, 2 wb + dw) sits at cell (2 hb + dh - 2 p) * 3 + (2 wb + dw - 2 q) of this window;
        // window p = hb - 1 covers only dh = 0 (cell row 2), p = hb covers dh = 0, 1 (rows 0, 1)
#pragma unroll
        for (int dh = 0; dh < 2; ++dh) {
          if (pi == 0 && dh == 1) continue;
#pragma unroll
          for (int dw = 0; dw < 2; ++dw) {
            if (qi == 0 && dw == 1) continue;
            const uint32_t cell = (2 * (1 - pi) + dh) * 3 + (2 * (1 - qi) + dw);
#pragma unroll
            for (int j = 0; j < VEC; ++j) {
              const uint32_t aj = (am[pi][qi][j / 4] >> (8 * (j % 4))) & 0xffu;
              acc[dh][dw][j] += aj == cell ? d[pi][qi][j] : 0.f;
            }
          }
        }
      }
    }
#pragma unroll
    for (int dh = 0; dh < 2; ++dh) {
      const int h = 2 * hb + dh;
      if (h >= g.H) continue;
#pragma unroll
      for (int dw = 0; dw < 2; ++dw) {
        const int w = 2 * wb + dw;
        if (w >= g.W) continue;
        *(uint4*)(dx + (size_t)((n * g.H + h) * g.W + w) * g.C + cv * VEC) = pack16<T>(acc[dh][dw]);
      }
    }
  }
}

// ReLU over 16-byte vectors; the scalar tail goes to the first threads.
template <typename T>
__global__ __launch_bounds__(256) void relu_fwd_kernel(const T* x, T* y, size_t n) {
  constexpr int VEC = 16 / sizeof(T);
  const size_t nv = n / VEC;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < nv; i += stride) {
    union { uint4 u; T e[VEC]; } v;
    v.u = ((const uint4*)x)[i];
#pragma unroll
    for (int j = 0; j < VEC; ++j)
      if (!(ld_f<T>(&v.e[j]) > 0.f)) v.e[j] = (T)0;
    ((uint4*)y)[i] = v.u;
  }
  const size_t t = nv * VEC + (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t < n) y[t] = ld_f<T>(x + t) > 0.f ? x[t] : (T)0;
}

template <typename T>
__global__ __launch_bounds__(256) void relu_bwd_kernel(const T* y, const T* dy, T* dx, size_t n) {
  constexpr int VEC = 16 / sizeof(T);
  const size_t nv = n / VEC;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < nv; i += stride) {
    union { uint4 u; T e[VEC]; } vy, vg;
    vy.u = ((const uint4*)y)[i];
    vg.u = ((const uint4*)dy)[i];
#pragma unroll
    for (int j = 0; j < VEC; ++j)
      if (!(ld_f<T>(&vy.e[j]) > 0.f)) vg.e[j] = (T)0;
    ((uint4*)dx)[i] = vg.u;
  }
  const size_t t = nv * VEC + (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t < n) dx[t] = ld_f<T>(y + t) > 0.f ? dy[t] : (T)0;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// One wave per row.  The row's maximum and the sum of exp(z - max) are
// built in one pass with the running-max rescaling of the sum, in chunks of
// 16 values per lane whose loads are all issued before any is used; a second
// pass, chunked the same way, writes the gradient.  The row's loss goes to
// loss[1 + row].
template <typename T>
__global__ __launch_bounds__(256) void softmax_ce_rows_kernel(int B, int classes, const T* __restrict__ z,
                                                              const int32_t* __restrict__ labels,
                                                              float* __restrict__ loss, T* __restrict__ dz) {
  constexpr int U = 16;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= B) return;
  const T* zr = z + (size_t)row * classes;
  float m = -INFINITY, s = 0.f;
  for (int base = 0; base < classes; base += 64 * U) {
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = base + 64 * u + lane;
      v[u] = j < classes ? ld_f<T>(zr + j) : -INFINITY;
    }
    float mc = m;
#pragma unroll
    for (int u = 0; u < U; ++u) mc = fmaxf(mc, v[u]);
    if (mc == -INFINITY) continue;  // nothing in this chunk for this lane
    s *= expf(m - mc);              // m = -inf: s is 0 and stays 0
#pragma unroll
    for (int u = 0; u < U; ++u) s += expf(v[u] - mc);
    m = mc;
  }
  // combine the lanes' (max, sum) pairs
  const float mw = wave_max(m);
  s = (m == -INFINITY) ? 0.f : s * expf(m - mw);
  s = wave_sum(s);
  const float lse = mw + logf(s);
  const int lab = labels[row];
  const float invB = 1.f / (float)B;
  T* dr = dz + (size_t)row * classes;
  for (int base = 0; base < classes; base += 64 * U) {
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = base + 64 * u + lane;
      v[u] = j < classes ? ld_f<T>(zr + j) : 0.f;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = base + 64 * u + lane;
      if (j < classes) st_f<T>(dr + j, (expf(v[u] - lse) - (j == lab ? 1.f : 0.f)) * invB);
    }
  }
  if (lane == 0) loss[1 + row] = (lab >= 0 && lab < classes) ? lse - ld_f<T>(zr + lab) : 0.f;
}

// loss[0] = mean of loss[1..B]: thread t adds rows t, t + 256, ... in order,
// then a fixed-shape tree adds the thread sums.
__global__ __launch_bounds__(256) void softmax_ce_mean_kernel(int B, float* __restrict__ loss) {
  __shared__ float red[256];
  float s = 0.f;
  for (int r = threadIdx.x; r < B; r += 256) s += loss[1 + r];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) loss[0] = red[0] / (float)B;
}

// Fused SGD with momentum, and AdaGrad, over a flat parameter buffer (the
// Updater), with the bf16 shadow written in the same pass.  The Updaters stream w, g and the state (momentum v, or AdaGrad's h) once:
// a thread owns UPD_U float4 vectors of each array, UPD_U x 256 apart so that
// each load instruction of a workgroup covers 4 KB of contiguous memory, and
// issues all its loads before any arithmetic.  Loads and stores are
// non-temporal (the buffers are read once and written once per step, larger
// than the caches): with 16 parameters per thread this measured 6.1 TB/s on
// the 62.4M-parameter buffer, against 5.3-5.5 with cached accesses, 8
// parameters per thread or either kind of access alone non-temporal.
constexpr int UPD_U = 4;
typedef float f4v __attribute__((ext_vector_type(4)));
typedef uint32_t u2v __attribute__((ext_vector_type(2)));

__device__ __forceinline__ u2v bf16x4_bits(const f4v& w) {
  return u2v{f32x2_to_bf16x2(w.x, w.y), f32x2_to_bf16x2(w.z, w.w)};
}

// STEP(w, state, g): one Updater step on one parameter (sgd_step or adagrad_step).
template <typename Step>
__device__ __forceinline__ void update_stream(size_t n, float* __restrict__ w, const float* __restrict__ g,
                                              float* __restrict__ s, uint16_t* __restrict__ wb, Step step) {
  const size_t n4 = n / 4;
  const size_t base = (size_t)blockIdx.x * blockDim.x * UPD_U + threadIdx.x;
  f4v W[UPD_U], G[UPD_U], S[UPD_U];
#pragma unroll
  for (int u = 0; u < UPD_U; ++u) {
    const size_t i = base + (size_t)u * blockDim.x;
    if (i < n4) {
      W[u] = __builtin_nontemporal_load((const f4v*)w + i);
      G[u] = __builtin_nontemporal_load((const f4v*)g + i);
      S[u] = __builtin_nontemporal_load((const f4v*)s + i);
    }
  }
#pragma unroll
  for (int u = 0; u < UPD_U; ++u) {
    const size_t i = base + (size_t)u * blockDim.x;
    if (i < n4) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float we = W[u][e], se = S[u][e];
        step(we, se, G[u][e]);
        W[u][e] = we;
        S[u][e] = se;
      }
      __builtin_nontemporal_store(S[u], (f4v*)s + i);
      __builtin_nontemporal_store(W[u], (f4v*)w + i);
      if (wb) __builtin_nontemporal_store(bf16x4_bits(W[u]), (u2v*)wb + i);
    }
  }
  // the last n % 4 parameters: one thread each in the first workgroup
  const size_t t = n4 * 4 + threadIdx.x;
  if (blockIdx.x == 0 && t < n) {
    float wt = w[t], st = s[t];
    step(wt, st, g[t]);
    s[t] = st;
    w[t] = wt;
    if (wb) wb[t] = f32_to_bf16(wt);
  }
}

__global__ __launch_bounds__(256) void sgd_kernel(size_t n, float* __restrict__ w, const float* __restrict__ g,
                                                  float* __restrict__ v, uint16_t* __restrict__ wb, float lr,
                                                  float mom, float wd) {
  update_stream(n, w, g, v, wb, [=](float& we, float& ve, float ge) { sgd_step(we, ve, ge, lr, mom, wd); });
}

// AdaGrad over a flat parameter buffer, laid out like sgd_kernel.
__global__ __launch_bounds__(256) void adagrad_kernel(size_t n, float* __restrict__ w, const float* __restrict__ g,
                                                      float* __restrict__ h, uint16_t* __restrict__ wb, float lr,
                                                      float delta, float wd) {
  update_stream(n, w, g, h, wb, [=](float& we, float& he, float ge) { adagrad_step(we, he, ge, lr, delta, wd); });
}

// ------------------------------------------------- local response norm
//
// Across channels, Caffe's form: s = k + alpha/size * (sum of x^2 over the
// channels [c - size/2, c + (size-1)/2] that exist), y = x s^-beta;
// backward dx[c] = dy[c] s[c]^-beta - (2 alpha beta / size) x[c] *
// sum over the channels j whose window holds c of dy[j] x[j] s[j]^(-beta-1),
// with s recomputed from x.  All in fp32.
struct LrnGeom {
  int N, C, HW, size;
  float alpha, beta, k;
};

__device__ __forceinline__ float pow_neg(float s, float e) { return exp2f(-e * log2f(s)); }  // s^-e, s > 0
// The same for a normal s (s >= 2^-126: the vector kernel's s >= k, which the
// launcher checks): the hardware log2 / exp2 without the library's
// subnormal handling, and the reciprocal, each within an ulp or two.
__device__ __forceinline__ float pow_neg_n(float s, float e) {
  return __builtin_amdgcn_exp2f(-e * __builtin_amdgcn_logf(s));
}
__device__ __forceinline__ float rcp_n(float s) { return __builtin_amdgcn_rcpf(s); }

// One element per thread, any layout: channel stride cs (1 for NHWC, HW for NCHW).
template <typename T, bool NCHW, bool BWD>
__global__ __launch_bounds__(256) void lrn_kernel(LrnGeom g, const T* __restrict__ x, const T* __restrict__ dy,
                                                  T* __restrict__ out, long total) {
  const long cs = NCHW ? g.HW : 1;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (long)gridDim.x * blockDim.x) {
    int c;
    long base;  // element (n, channel 0, p)
    if (NCHW) {
      const long n = i / ((long)g.C * g.HW), r = i - n * g.C * g.HW;
      c = (int)(r / g.HW);
      base = n * g.C * g.HW + (r - (long)c * g.HW);
    } else {
      c = (int)(i % g.C);
      base = i - c;
    }
    auto scale = [&](int j) {
      const int lo = max(j - g.size / 2, 0), hi = min(j + (g.size - 1) / 2, g.C - 1);
      float acc = 0.f;
      for (int t = lo; t <= hi; ++t) {
        const float v = ld_f<T>(x + base + t * cs);
        acc = fmaf(v, v, acc);
      }
      return fmaf(g.alpha / (float)g.size, acc, g.k);
    };
    const float xc = ld_f<T>(x + base + c * cs);
    if (!BWD) {
      st_f<T>(out + i, xc * pow_neg(scale(c), g.beta));
    } else {
      const int lo = max(c - (g.size - 1) / 2, 0), hi = min(c + g.size / 2, g.C - 1);
      float acc = 0.f;
      for (int j = lo; j <= hi; ++j)
        acc += ld_f<T>(dy + base + j * cs) * ld_f<T>(x + base + j * cs) * pow_neg(scale(j), g.beta + 1.f);
      const float r = ld_f<T>(dy + i) * pow_neg(scale(c), g.beta) - 2.f * g.alpha * g.beta / (float)g.size * xc * acc;
      st_f<T>(out + i, r);
    }
  }
}

// NHWC, VEC channels (16 bytes) per thread.  A workgroup stages 256
// consecutive chunks of x (and dy) plus one chunk on either side in LDS, so
// every element is read from memory once; each thread takes its chunk and its
// two neighbours from LDS (zeros past the ends of the pixel's channel axis,
// which add nothing to a sum of squares), so every window of its channels is
// in registers.  Backward: each thread computes s^-beta and
// q = dy x s^(-beta-1) = dy x s^-beta / s for its own channels only (one
// power per channel) and leaves q in LDS, where the neighbouring threads
// take the (SIZE-1)/2 and SIZE/2 values their windows reach into; the kernel
// is bound by its transcendental arithmetic, not its bytes.  The window
// SIZE is a compile-time constant (3 or 5), so all register indices are
// static.
template <typename T, int VEC, bool BWD, int SIZE>
__global__ __launch_bounds__(256) void lrn_vec_kernel(LrnGeom g, const T* __restrict__ x, const T* __restrict__ dy,
                                                      T* __restrict__ out, long chunks) {
  const int CV = g.C / VEC;
  __shared__ uint4 xs[258];
  __shared__ float qs[BWD ? 256 * VEC : 1];
  const uint4* __restrict__ x4 = (const uint4*)x;
  const uint4* __restrict__ d4 = (const uint4*)dy;
  const int tid = threadIdx.x;
  // 16 bytes at p, or zeros when !ok, by value (a reference to a local
  // constant would put the constant in scratch memory)
  auto ld0 = [](bool ok, const uint4* p) {
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (ok) v = *p;
    return v;
  };
  // s of channel c sums x^2 over [c - HI, c + LO]; dx of c sums q over [c - LO, c + HI]
  constexpr int LO = (SIZE - 1) / 2, HI = SIZE / 2;
  for (long b0 = (long)blockIdx.x * 256; b0 < chunks; b0 += (long)gridDim.x * 256) {
    const long t = b0 + tid;
    xs[1 + tid] = ld0(t < chunks, x4 + t);
    float dv[VEC];
    unpack16<T>(ld0(BWD && t < chunks, d4 + t), dv);
    if (tid < 2) {  // the chunks just before and just after the workgroup's range
      const long h = tid == 0 ? b0 - 1 : b0 + 256;
      xs[tid == 0 ? 0 : 257] = ld0(h >= 0 && h < chunks, x4 + h);
    }
    __syncthreads();
    const int cv = (int)(t % CV);
    float xv[3 * VEC];
#pragma unroll
    for (int h = 0; h < 3; ++h) {
      const bool in = (h == 0 && cv > 0) || h == 1 || (h == 2 && cv < CV - 1);  // same pixel
      unpack16<T>(ld0(in, xs + tid + h), xv + h * VEC);
    }
    const float an = g.alpha / (float)SIZE;
    // window sums of x^2 as a running sum over the chunk (the kernel is bound
    // by its arithmetic): squares of channels -HI .. VEC + LO - 1
    float sq[HI + VEC + LO];
#pragma unroll
    for (int r = 0; r < HI + VEC + LO; ++r) sq[r] = xv[VEC - HI + r] * xv[VEC - HI + r];
    float sc[VEC], p[VEC];
    float win = 0.f;
#pragma unroll
    for (int r = 0; r <= HI + LO; ++r) win += sq[r];
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
      if (j > 0) win += sq[j + HI + LO] - sq[j - 1];
      sc[j] = fmaf(an, win, g.k);
      p[j] = pow_neg_n(sc[j], g.beta);  // s^-beta
    }
    float o[VEC];
    if (!BWD) {
#pragma unroll
      for (int j = 0; j < VEC; ++j) o[j] = xv[VEC + j] * p[j];
    } else {
#pragma unroll
      for (int j = 0; j < VEC; ++j) qs[tid * VEC + j] = dv[j] * xv[VEC + j] * p[j] * rcp_n(sc[j]);
      __syncthreads();
      // q of the own chunk (at LO + j) and of the LO channels before it and the
      // HI channels after it that the windows reach into (same pixel only)
      float q[LO + VEC + HI];
#pragma unroll
      for (int j = 0; j < VEC; ++j) q[LO + j] = qs[tid * VEC + j];
#pragma unroll
      for (int e = 0; e < LO; ++e) q[e] = (cv > 0 && tid > 0) ? qs[(tid - 1) * VEC + VEC - LO + e] : 0.f;
#pragma unroll
      for (int e = 0; e < HI; ++e) q[LO + VEC + e] = (cv < CV - 1 && tid < 255) ? qs[(tid + 1) * VEC + e] : 0.f;
      // a neighbour chunk outside this workgroup's range: its q from its own
      // values; the window sums of its channels needed here only reach into
      // this chunk (VEC >= LO + HI)
      static_assert(VEC >= LO + HI, "window wider than a chunk");
      const bool left = tid == 0 && cv > 0, right = tid == 255 && cv < CV - 1 && t + 1 < chunks;
      if (left || right) {
        const long nb = left ? t - 1 : t + 1;
        float dnf[VEC], xnf[VEC];
        unpack16<T>(d4[nb], dnf);
        unpack16<T>(x4[nb], xnf);
        if (left) {  // channels VEC - LO .. VEC - 1 of chunk t - 1; their windows reach into this chunk
#pragma unroll
          for (int e = 0; e < LO; ++e) {
            const int j = VEC - LO + e;
            float acc = 0.f;
#pragma unroll
            for (int f = -HI; f <= LO; ++f) {
              const float v = j + f < VEC ? xnf[j + f] : xv[VEC + j + f - VEC];
              acc = fmaf(v, v, acc);
            }
            const float sn = fmaf(an, acc, g.k);
            q[e] = dnf[j] * xnf[j] * pow_neg_n(sn, g.beta) * rcp_n(sn);
          }
        } else {  // channels 0 .. HI - 1 of chunk t + 1; their windows reach back into this chunk
#pragma unroll
          for (int e = 0; e < HI; ++e) {
            float acc = 0.f;
#pragma unroll
            for (int f = -HI; f <= LO; ++f) {
              const float v = e + f >= 0 ? xnf[e + f] : xv[VEC + VEC + e + f];
              acc = fmaf(v, v, acc);
            }
            const float sn = fmaf(an, acc, g.k);
            q[LO + VEC + e] = dnf[e] * xnf[e] * pow_neg_n(sn, g.beta) * rcp_n(sn);
          }
        }
      }
      const float c2 = 2.f * g.alpha * g.beta / (float)SIZE;
      float qw = 0.f;  // running sum of q over [j - LO, j + HI]
#pragma unroll
      for (int r = 0; r <= LO + HI; ++r) qw += q[r];
#pragma unroll
      for (int j = 0; j < VEC; ++j) {
        if (j > 0) qw += q[j + LO + HI] - q[j - 1];
        o[j] = dv[j] * p[j] - c2 * xv[VEC + j] * qw;
      }
    }
    if (t < chunks) ((uint4*)out)[t] = pack16<T>(o);
    __syncthreads();  // the LDS tiles are reused by the next range
  }
}

}  // namespace

hipError_t launch_lrn(int dt, int bwd, int N, int C, int HW, int size, float alpha, float beta, float k,
                      const void* x, const void* dy, void* out, int nchw, hipStream_t st) {
  LrnGeom g{N, C, HW, size, alpha, beta, k};
  const long total = (long)N * C * HW;
  const int vec = dt == BF16 ? 8 : 4;
  // (the vector kernel's arithmetic assumes a normal k, hence a normal s)
  const bool v = !nchw && C % vec == 0 && (uintptr_t)x % 16 == 0 && (uintptr_t)out % 16 == 0 &&
                 (uintptr_t)dy % 16 == 0 && (size == 3 || size == 5) && k >= 1.17549435e-38f;
  TraceScope ts(bwd ? "lrn_bwd_kernel" : "lrn_fwd_kernel", st, (double)total * dt_size(dt) * (bwd ? 3 : 2),
                WORK_BYTE);
  if (v) {
    const long chunks = total / vec;
    const unsigned grid = grid_for((size_t)chunks);
#define LRN_VEC(T, VV, B, Z)                                                                                   \
  hipLaunchKernelGGL((lrn_vec_kernel<T, VV, B, Z>), dim3(grid), dim3(256), 0, st, g, (const T*)x, (const T*)dy, \
                     (T*)out, chunks)
#define LRN_VEC_SIZE(T, VV, B) \
  if (size == 5) LRN_VEC(T, VV, B, 5); else LRN_VEC(T, VV, B, 3);
    if (dt == BF16) { if (bwd) { LRN_VEC_SIZE(bf16_t, 8, true) } else { LRN_VEC_SIZE(bf16_t, 8, false) } }
    else { if (bwd) { LRN_VEC_SIZE(float, 4, true) } else { LRN_VEC_SIZE(float, 4, false) } }
#undef LRN_VEC_SIZE
#undef LRN_VEC
    return hipGetLastError();
  }
  const unsigned grid = grid_for((size_t)total);
#define LRN_EL(T, L, B) \
  hipLaunchKernelGGL((lrn_kernel<T, L, B>), dim3(grid), dim3(256), 0, st, g, (const T*)x, (const T*)dy, (T*)out, total)
  if (dt == BF16) {
    if (nchw) { if (bwd) LRN_EL(bf16_t, true, true); else LRN_EL(bf16_t, true, false); }
    else { if (bwd) LRN_EL(bf16_t, false, true); else LRN_EL(bf16_t, false, false); }
  } else {
    if (nchw) { if (bwd) LRN_EL(float, true, true); else LRN_EL(float, true, false); }
    else { if (bwd) LRN_EL(float, false, true); else LRN_EL(float, false, false); }
  }
#undef LRN_EL
  return hipGetLastError();
}

hipError_t launch_adagrad(size_t n, float* w, const float* g, float* h, uint16_t* wb, float lr, float delta,
                          float wd, hipStream_t st) {
  const unsigned grid = grid_for(n / 4 / UPD_U + 1, 256, 1u << 30);
  TraceScope ts("adagrad_kernel", st, (double)n * (20.0 + (wb ? 2.0 : 0.0)), WORK_BYTE);
  hipLaunchKernelGGL(adagrad_kernel, dim3(grid), dim3(256), 0, st, n, w, g, h, wb, lr, delta, wd);
  return hipGetLastError();
}

hipError_t launch_pool_fwd(int dt, int mode, int N, int C, int H, int W, int P, int Q, int kh, int kw, int sh, int sw,
                           int ph, int pw, const void* x, void* y, uint8_t* argmax, int nchw, hipStream_t st) {
  PoolGeom g{N, C, H, W, P, Q, kh, kw, sh, sw, ph, pw};
  const long total = (long)N * C * P * Q;
  const int vec = dt == BF16 ? 8 : 4;
  const bool v = !nchw && C % vec == 0 && (uintptr_t)x % 16 == 0 && (uintptr_t)y % 16 == 0 &&
                 (mode != 0 || (uintptr_t)argmax % vec == 0);
  TraceScope ts(mode == 0 ? "pool_fwd_kernel<max>" : "pool_fwd_kernel<avg>", st,
                (double)N * C * H * W * dt_size(dt) + (double)total * (dt_size(dt) + (mode == 0 ? 1 : 0)), WORK_BYTE);
  if (v) {
    const int tv = (int)(total / vec);
    const unsigned grid = grid_for((size_t)tv);
    const FastDiv dCV = make_fastdiv((uint32_t)(C / vec)), dQ = make_fastdiv((uint32_t)Q),
                  dP = make_fastdiv((uint32_t)P);
    const bool k3 = kh == 3 && kw == 3;
#define POOL_FWD_VEC(T, V, KS, M)                                                                        \
  hipLaunchKernelGGL((pool_fwd_nhwc_vec_kernel<T, V, KS, M>), dim3(grid), dim3(256), 0, st, g, dCV, dQ, dP, \
                     (const T*)x, (T*)y, argmax, tv)
#define POOL_FWD_VEC_M(T, V, KS) \
  if (mode == 0) POOL_FWD_VEC(T, V, KS, 0); else POOL_FWD_VEC(T, V, KS, 1)
    if (dt == BF16) {
      if (k3) { POOL_FWD_VEC_M(bf16_t, 8, 3); } else { POOL_FWD_VEC_M(bf16_t, 8, 0); }
    } else {
      if (k3) { POOL_FWD_VEC_M(float, 4, 3); } else { POOL_FWD_VEC_M(float, 4, 0); }
    }
#undef POOL_FWD_VEC_M
#undef POOL_FWD_VEC
    return hipGetLastError();
  }
  const unsigned grid = grid_for((size_t)total);
#define POOL_FWD(T, L) \
  hipLaunchKernelGGL((pool_fwd_kernel<T, L>), dim3(grid), dim3(256), 0, st, g, mode, (const T*)x, (T*)y, argmax, total)
  if (dt == BF16) {
    if (nchw) POOL_FWD(bf16_t, true); else POOL_FWD(bf16_t, false);
  } else {
    if (nchw) POOL_FWD(float, true); else POOL_FWD(float, false);
  }
#undef POOL_FWD
  return hipGetLastError();
}

hipError_t launch_pool_bwd(int dt, int mode, int N, int C, int H, int W, int P, int Q, int kh, int kw, int sh, int sw,
                           int ph, int pw, const void* dy, const uint8_t* argmax, const void* ymask, void* dx,
                           int nchw, hipStream_t st) {
  PoolGeom g{N, C, H, W, P, Q, kh, kw, sh, sw, ph, pw};
  const long total = (long)N * C * H * W;
  const int vec = dt == BF16 ? 8 : 4;
  if (mode != 0) ymask = nullptr;
  const bool v = !nchw && C % vec == 0 && (uintptr_t)dy % 16 == 0 && (uintptr_t)dx % 16 == 0 &&
                 (mode != 0 || (uintptr_t)argmax % vec == 0) && (uintptr_t)ymask % 16 == 0;
  TraceScope ts(mode == 0 ? "pool_bwd_kernel<max>" : "pool_bwd_kernel<avg>", st,
                (double)N * C * P * Q * (dt_size(dt) * (ymask ? 2 : 1) + (mode == 0 ? 1 : 0)) +
                    (double)total * dt_size(dt),
                WORK_BYTE);
  if (v && mode == 0 && kh == 3 && kw == 3 && sh == 2 && sw == 2 && ph == 0 && pw == 0) {
    const int HB = (H + 1) / 2, WB = (W + 1) / 2;
    const int tb = N * HB * WB * (C / vec);
    const unsigned grid = grid_for((size_t)tb);
    const FastDiv dCV = make_fastdiv((uint32_t)(C / vec)), dWB = make_fastdiv((uint32_t)WB),
                  dHB = make_fastdiv((uint32_t)HB);
#define POOL_BWD_K3S2(T, VV, M)                                                                                  \
  hipLaunchKernelGGL((pool_bwd_k3s2_kernel<T, VV, M>), dim3(grid), dim3(256), 0, st, g, dCV, dWB, dHB, HB, WB,   \
                     (const T*)dy, argmax, (const T*)ymask, (T*)dx, tb)
    if (dt == BF16) {
      if (ymask) POOL_BWD_K3S2(bf16_t, 8, true); else POOL_BWD_K3S2(bf16_t, 8, false);
    } else {
      if (ymask) POOL_BWD_K3S2(float, 4, true); else POOL_BWD_K3S2(float, 4, false);
    }
#undef POOL_BWD_K3S2
    return hipGetLastError();
  }
  if (v) {
    const int tv = (int)(total / vec);
    const unsigned grid = grid_for((size_t)tv);
    const FastDiv dCV = make_fastdiv((uint32_t)(C / vec)), dW = make_fastdiv((uint32_t)W),
                  dH = make_fastdiv((uint32_t)H);
#define POOL_BWD_VEC(T, VV, M)                                                                                   \
  hipLaunchKernelGGL((pool_bwd_nhwc_vec_kernel<T, VV, M>), dim3(grid), dim3(256), 0, st, g, dCV, dW, dH, mode, \
                     (const T*)dy, argmax, (const T*)ymask, (T*)dx, tv)
    if (dt == BF16) {
      if (ymask) POOL_BWD_VEC(bf16_t, 8, true); else POOL_BWD_VEC(bf16_t, 8, false);
    } else {
      if (ymask) POOL_BWD_VEC(float, 4, true); else POOL_BWD_VEC(float, 4, false);
    }
#undef POOL_BWD_VEC
    return hipGetLastError();
  }
  const unsigned grid = grid_for((size_t)total);
#define POOL_BWD(T, L)                                                                                           \
  hipLaunchKernelGGL((pool_bwd_kernel<T, L>), dim3(grid), dim3(256), 0, st, g, mode, (const T*)dy, argmax,      \
                     (const T*)ymask, (T*)dx, total)
  if (dt == BF16) {
    if (nchw) POOL_BWD(bf16_t, true); else POOL_BWD(bf16_t, false);
  } else {
    if (nchw) POOL_BWD(float, true); else POOL_BWD(float, false);
  }
#undef POOL_BWD
  return hipGetLastError();
}

hipError_t launch_relu_fwd(int dt, size_t n, const void* x, void* y, hipStream_t st) {
  const size_t vec = dt == BF16 ? 8 : 4;
  const unsigned grid = grid_for(n / vec + 1, 256, 8192);
  TraceScope ts("relu_fwd_kernel", st, 2.0 * n * dt_size(dt), WORK_BYTE);
  if (dt == BF16)
    hipLaunchKernelGGL(relu_fwd_kernel<bf16_t>, dim3(grid), dim3(256), 0, st, (const bf16_t*)x, (bf16_t*)y, n);
  else
    hipLaunchKernelGGL(relu_fwd_kernel<float>, dim3(grid), dim3(256), 0, st, (const float*)x, (float*)y, n);
  return hipGetLastError();
}

hipError_t launch_relu_bwd(int dt, size_t n, const void* y, const void* dy, void* dx, hipStream_t st) {
  const size_t vec = dt == BF16 ? 8 : 4;
  const unsigned grid = grid_for(n / vec + 1, 256, 8192);
  TraceScope ts("relu_bwd_kernel", st, 3.0 * n * dt_size(dt), WORK_BYTE);
  if (dt == BF16)
    hipLaunchKernelGGL(relu_bwd_kernel<bf16_t>, dim3(grid), dim3(256), 0, st, (const bf16_t*)y, (const bf16_t*)dy,
                       (bf16_t*)dx, n);
  else
    hipLaunchKernelGGL(relu_bwd_kernel<float>, dim3(grid), dim3(256), 0, st, (const float*)y, (const float*)dy,
                       (float*)dx, n);
  return hipGetLastError();
}

hipError_t launch_softmax_ce(int dt, int B, int classes, const void* z, const int32_t* labels, float* loss, void* dz,
                             hipStream_t st) {
  {
    TraceScope ts("softmax_ce_rows_kernel", st, 2.0 * B * (double)classes * dt_size(dt) + 8.0 * B, WORK_BYTE);
    const unsigned grid = (unsigned)((B + 3) / 4);
    if (dt == BF16)
      hipLaunchKernelGGL(softmax_ce_rows_kernel<bf16_t>, dim3(grid), dim3(256), 0, st, B, classes, (const bf16_t*)z,
                         labels, loss, (bf16_t*)dz);
    else
      hipLaunchKernelGGL(softmax_ce_rows_kernel<float>, dim3(grid), dim3(256), 0, st, B, classes, (const float*)z,
                         labels, loss, (float*)dz);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  TraceScope ts("softmax_ce_mean_kernel", st, 4.0 * B + 4.0, WORK_BYTE);
  hipLaunchKernelGGL(softmax_ce_mean_kernel, dim3(1), dim3(256), 0, st, B, loss);
  return hipGetLastError();
}

hipError_t launch_sgd(size_t n, float* w, const float* g, float* v, uint16_t* wb, float lr, float mom, float wd,
                      hipStream_t st) {
  const unsigned grid = grid_for(n / 4 / UPD_U + 1, 256, 1u << 30);
  TraceScope ts("sgd_kernel", st, (double)n * (20.0 + (wb ? 2.0 : 0.0)), WORK_BYTE);
  hipLaunchKernelGGL(sgd_kernel, dim3(grid), dim3(256), 0, st, n, w, g, v, wb, lr, mom, wd);
  return hipGetLastError();
}

}  // namespace singa
