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
                                                       const uint8_t* __restrict__ argmax, T* __restrict__ dx,
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
          if (argmax[o] == cell) acc += ld_f<T>(dy + o);
        } else {
          acc += ld_f<T>(dy + o) / (float)pool_divisor(g, p, q);
        }
      }
    }
    st_f<T>(dx + i, acc);
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

// One workgroup of 16 waves; wave w takes rows w, w+16, ...  Each wave keeps
// its rows' losses in row order and the waves are summed in wave order, so
// the loss does not depend on timing.
constexpr int CE_WAVES = 16;
template <typename T>
__global__ __launch_bounds__(64 * CE_WAVES) void softmax_ce_kernel(int B, int classes, const T* __restrict__ z,
                                                                   const int32_t* __restrict__ labels,
                                                                   float* __restrict__ loss, T* __restrict__ dz) {
  __shared__ float wave_loss[CE_WAVES];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float invB = 1.f / (float)B;
  float my_loss = 0.f;
  for (int row = wave; row < B; row += CE_WAVES) {
    const T* zr = z + (size_t)row * classes;
    float m = -INFINITY;
    for (int j = lane; j < classes; j += 64) m = fmaxf(m, ld_f<T>(zr + j));
    m = wave_max(m);
    float s = 0.f;
    for (int j = lane; j < classes; j += 64) s += expf(ld_f<T>(zr + j) - m);
    s = wave_sum(s);
    const float lse = m + logf(s);
    const int lab = labels[row];
    const bool lab_ok = lab >= 0 && lab < classes;
    if (lab_ok) my_loss += lse - ld_f<T>(zr + lab);
    T* dr = dz + (size_t)row * classes;
    for (int j = lane; j < classes; j += 64) {
      const float prob = expf(ld_f<T>(zr + j) - lse);
      st_f<T>(dr + j, (prob - (j == lab ? 1.f : 0.f)) * invB);
    }
  }
  if (lane == 0) wave_loss[wave] = my_loss;
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = 0.f;
    for (int w = 0; w < CE_WAVES; ++w) t += wave_loss[w];
    *loss = t * invB;
  }
}

__global__ __launch_bounds__(256) void sgd_kernel(size_t n, float* __restrict__ w, const float* __restrict__ g,
                                                  float* __restrict__ v, uint16_t* __restrict__ wb, float lr,
                                                  float mom, float wd) {
  const size_t nv = n / 4;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < nv; i += stride) {
    float4 wv = ((const float4*)w)[i];
    const float4 gv = ((const float4*)g)[i];
    float4 vv = ((const float4*)v)[i];
    vv.x = mom * vv.x + lr * (gv.x + wd * wv.x);
    vv.y = mom * vv.y + lr * (gv.y + wd * wv.y);
    vv.z = mom * vv.z + lr * (gv.z + wd * wv.z);
    vv.w = mom * vv.w + lr * (gv.w + wd * wv.w);
    wv.x -= vv.x;
    wv.y -= vv.y;
    wv.z -= vv.z;
    wv.w -= vv.w;
    ((float4*)v)[i] = vv;
    ((float4*)w)[i] = wv;
    if (wb) {
      uint2 b;
      b.x = (uint32_t)f32_to_bf16(wv.x) | ((uint32_t)f32_to_bf16(wv.y) << 16);
      b.y = (uint32_t)f32_to_bf16(wv.z) | ((uint32_t)f32_to_bf16(wv.w) << 16);
      ((uint2*)wb)[i] = b;
    }
  }
  const size_t t = nv * 4 + (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t < n) {
    const float vt = mom * v[t] + lr * (g[t] + wd * w[t]);
    const float wt = w[t] - vt;
    v[t] = vt;
    w[t] = wt;
    if (wb) wb[t] = f32_to_bf16(wt);
  }
}

}  // namespace

hipError_t launch_pool_fwd(int dt, int mode, int N, int C, int H, int W, int P, int Q, int kh, int kw, int sh, int sw,
                           int ph, int pw, const void* x, void* y, uint8_t* argmax, int nchw, hipStream_t st) {
  PoolGeom g{N, C, H, W, P, Q, kh, kw, sh, sw, ph, pw};
  const long total = (long)N * C * P * Q;
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
                           int ph, int pw, const void* dy, const uint8_t* argmax, void* dx, int nchw, hipStream_t st) {
  PoolGeom g{N, C, H, W, P, Q, kh, kw, sh, sw, ph, pw};
  const long total = (long)N * C * H * W;
  const unsigned grid = grid_for((size_t)total);
#define POOL_BWD(T, L) \
  hipLaunchKernelGGL((pool_bwd_kernel<T, L>), dim3(grid), dim3(256), 0, st, g, mode, (const T*)dy, argmax, (T*)dx, total)
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
  if (dt == BF16)
    hipLaunchKernelGGL(relu_fwd_kernel<bf16_t>, dim3(grid), dim3(256), 0, st, (const bf16_t*)x, (bf16_t*)y, n);
  else
    hipLaunchKernelGGL(relu_fwd_kernel<float>, dim3(grid), dim3(256), 0, st, (const float*)x, (float*)y, n);
  return hipGetLastError();
}

hipError_t launch_relu_bwd(int dt, size_t n, const void* y, const void* dy, void* dx, hipStream_t st) {
  const size_t vec = dt == BF16 ? 8 : 4;
  const unsigned grid = grid_for(n / vec + 1, 256, 8192);
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
  if (dt == BF16)
    hipLaunchKernelGGL(softmax_ce_kernel<bf16_t>, dim3(1), dim3(64 * CE_WAVES), 0, st, B, classes, (const bf16_t*)z,
                       labels, loss, (bf16_t*)dz);
  else
    hipLaunchKernelGGL(softmax_ce_kernel<float>, dim3(1), dim3(64 * CE_WAVES), 0, st, B, classes, (const float*)z,
                       labels, loss, (float*)dz);
  return hipGetLastError();
}

hipError_t launch_sgd(size_t n, float* w, const float* g, float* v, uint16_t* wb, float lr, float mom, float wd,
                      hipStream_t st) {
  const unsigned grid = grid_for(n / 4 + 1, 256, 8192);
  hipLaunchKernelGGL(sgd_kernel, dim3(grid), dim3(256), 0, st, n, w, g, v, wb, lr, mom, wd);
  return hipGetLastError();
}

}  // namespace singa
