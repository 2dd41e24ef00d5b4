// conv_aux.hip -- the bandwidth-bound helpers around the convolution GEMMs:
//   * batched tiled transpose (flipped filter copies for backward-data, and the
//     filter transpose of a dense "fully connected" layer),
//   * direct gather backward-data for strides above one,
//   * bias-gradient column sums in a fixed order,
//   * NCHW <-> NHWC permutations for the NCHW entry points.
#include <type_traits>

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

// 32 x 32 tile through LDS: reads are coalesced along cols, writes along rows.
template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const T* __restrict__ in, T* __restrict__ out, int batch,
                                                        int rows, int cols, long in_bstride, long in_rstride,
                                                        long out_bstride, long out_rstride, int flip) {
  __shared__ T tile[32][33];
  const int b = blockIdx.z;
  const int r0 = blockIdx.y * 32, c0 = blockIdx.x * 32;
  const T* src = in + (long)b * in_bstride;
  T* dst = out + (long)(flip ? batch - 1 - b : b) * out_bstride;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 32 x 8
#pragma unroll
  for (int k = 0; k < 32; k += 8) {
    int r = r0 + ty + k, c = c0 + tx;
    if (r < rows && c < cols) tile[ty + k][tx] = src[(long)r * in_rstride + c];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 32; k += 8) {
    int c = c0 + ty + k, r = r0 + tx;
    if (r < rows && c < cols) dst[(long)c * out_rstride + r] = tile[tx][ty + k];
  }
}

// Vector form for 16-byte aligned rows: a 64 x 64 tile, read as 16-byte row
// vectors into LDS and written as 16-byte vectors of the transposed rows
// (every stride, size and base a multiple of the vector width).
template <typename T>
__global__ __launch_bounds__(256) void transpose_vec_kernel(const T* __restrict__ in, T* __restrict__ out, int batch,
                                                            int rows, int cols, long in_bstride, long in_rstride,
                                                            long out_bstride, long out_rstride, int flip) {
  constexpr int VEC = 16 / (int)sizeof(T);
  constexpr int TPR = 64 / VEC;   // threads per 64-element row
  constexpr int RPP = 256 / TPR;  // rows per pass
  __shared__ T tile[64][64 + 2];
  const int b = blockIdx.z;
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const T* src = in + (long)b * in_bstride;
  T* dst = out + (long)(flip ? batch - 1 - b : b) * out_bstride;
  const int tc = threadIdx.x % TPR, tr = threadIdx.x / TPR;
#pragma unroll
  for (int k = 0; k < 64; k += RPP) {
    const int r = r0 + tr + k, c = c0 + tc * VEC;
    union { uint4 u; T e[VEC]; } v;
    if (r < rows && c < cols) v.u = *(const uint4*)(src + (long)r * in_rstride + c);
    else v.u = make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int j = 0; j < VEC; ++j) tile[tr + k][tc * VEC + j] = v.e[j];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 64; k += RPP) {
    const int c = c0 + tr + k, r = r0 + tc * VEC;  // output row c, output columns r .. r + VEC - 1
    if (c < cols && r < rows) {
      union { uint4 u; T e[VEC]; } v;
#pragma unroll
      for (int j = 0; j < VEC; ++j) v.e[j] = tile[tc * VEC + j][tr + k];
      *(uint4*)(dst + (long)c * out_rstride + r) = v.u;
    }
  }
}

// dx[n,h,w,c] = sum over taps (r,s) whose output pixel (p,q) lands on a whole
// multiple of the stride, and over k, of w[k,r,s,c] * dy[n,p,q,k].
template <typename T>
__global__ __launch_bounds__(256) void bwd_data_direct_kernel(ConvShape s, const T* __restrict__ dy,
                                                              const T* __restrict__ w,
                                                              const T* __restrict__ mask, T* __restrict__ dx,
                                                              long total) {
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (long)gridDim.x * blockDim.x) {
    const int c = (int)(i % s.C);
    long t = i / s.C;
    const int x = (int)(t % s.W);
    t /= s.W;
    const int h = (int)(t % s.H);
    const int n = (int)(t / s.H);
    float acc = 0.f;
    for (int r = 0; r < s.R; ++r) {
      const int pn = h + s.ph - r;
      if (pn < 0 || pn % s.sh) continue;
      const int p = pn / s.sh;
      if (p >= s.P) continue;
      for (int q_s = 0; q_s < s.S; ++q_s) {
        const int qn = x + s.pw - q_s;
        if (qn < 0 || qn % s.sw) continue;
        const int q = qn / s.sw;
        if (q >= s.Q) continue;
        const T* dyr = dy + (((long)n * s.P + p) * s.Q + q) * s.K;
        const T* wr = w + ((long)r * s.S + q_s) * s.C + c;
        const long wk = (long)s.R * s.S * s.C;
        for (int k = 0; k < s.K; ++k) acc += ld_f<T>(wr + k * wk) * ld_f<T>(dyr + k);
      }
    }
    if (mask && !(ld_f<T>(mask + i) > 0.f)) acc = 0.f;
    st_f<T>(dx + i, acc);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void nchw_to_nhwc_kernel(const T* __restrict__ in, T* __restrict__ out, int C,
                                                           int HW) {
  // one (n) image per blockIdx.z; transpose [C][HW] -> [HW][C] with 32x32 tiles
  __shared__ T tile[32][33];
  const long base = (long)blockIdx.z * C * HW;
  const int c0 = blockIdx.y * 32, s0 = blockIdx.x * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
#pragma unroll
  for (int k = 0; k < 32; k += 8) {
    int c = c0 + ty + k, sp = s0 + tx;
    if (c < C && sp < HW) tile[ty + k][tx] = in[base + (long)c * HW + sp];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 32; k += 8) {
    int sp = s0 + ty + k, c = c0 + tx;
    if (c < C && sp < HW) out[base + (long)sp * C + c] = tile[tx][ty + k];
  }
}

template <typename T>
__global__ __launch_bounds__(256) void nhwc_to_nchw_kernel(const T* __restrict__ in, T* __restrict__ out, int C,
                                                           int HW) {
  __shared__ T tile[32][33];
  const long base = (long)blockIdx.z * C * HW;
  const int s0 = blockIdx.y * 32, c0 = blockIdx.x * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
#pragma unroll
  for (int k = 0; k < 32; k += 8) {
    int sp = s0 + ty + k, c = c0 + tx;
    if (c < C && sp < HW) tile[ty + k][tx] = in[base + (long)sp * C + c];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 32; k += 8) {
    int c = c0 + ty + k, sp = s0 + tx;
    if (c < C && sp < HW) out[base + (long)c * HW + sp] = tile[tx][ty + k];
  }
}

__global__ __launch_bounds__(256) void krsc_to_kcrs_kernel(const float* __restrict__ in, float* __restrict__ out,
                                                           int K, int C, int RS, int accumulate) {
  const long total = (long)K * C * RS;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (long)gridDim.x * blockDim.x) {
    // i indexes the KCRS output
    const int rs = (int)(i % RS);
    const long kc = i / RS;
    const int c = (int)(kc % C);
    const int k = (int)(kc / C);
    const float v = in[((long)k * RS + rs) * C + c];
    out[i] = accumulate ? out[i] + v : v;
  }
}

// out[r][c] = in[r][c] for c < C, 0 for C <= c < Cp (Cp % 4 == 0): one
// thread per 4-channel chunk of an output row, stored as one vector.
template <typename T>
__global__ __launch_bounds__(256) void pad_channels_kernel(const T* __restrict__ in, T* __restrict__ out, long rows,
                                                           int C, int Cp) {
  typedef typename std::conditional<sizeof(T) == 2, uint2, uint4>::type V4;
  const int nv = Cp / 4;
  const long total = rows * nv;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (long)gridDim.x * blockDim.x) {
    const long r = i / nv;
    const int c0 = (int)(i - r * nv) * 4;
    union { V4 u; T e[4]; } v;
#pragma unroll
    for (int j = 0; j < 4; ++j) v.e[j] = (c0 + j < C) ? in[r * C + c0 + j] : (T)0;
    *(V4*)(out + r * Cp + c0) = v.u;
  }
}

// The same for C = 3, Cp = 4 (colour images): one thread per 8 rows, read as
// 3 (bf16) / 6 (fp32) 16-byte vectors and written as 4 / 8.
template <typename T>
__global__ __launch_bounds__(256) void pad_3to4_kernel(const T* __restrict__ in, T* __restrict__ out, long groups) {
  constexpr int NI = 24 * (int)sizeof(T) / 16, NO = 32 * (int)sizeof(T) / 16;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < groups; i += (long)gridDim.x * blockDim.x) {
    union { uint4 u[NI]; T e[24]; } a;
    union { uint4 u[NO]; T e[32]; } b;
    const uint4* src = (const uint4*)(in + i * 24);
#pragma unroll
    for (int k = 0; k < NI; ++k) a.u[k] = src[k];
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      b.e[4 * p] = a.e[3 * p];
      b.e[4 * p + 1] = a.e[3 * p + 1];
      b.e[4 * p + 2] = a.e[3 * p + 2];
      b.e[4 * p + 3] = T(0);
    }
    uint4* dst = (uint4*)(out + i * 32);
#pragma unroll
    for (int k = 0; k < NO; ++k) dst[k] = b.u[k];
  }
}

// Space-to-depth rewrite of a strided convolution (stride sh x sw, padding
// ph, pw) as a stride-1 convolution without padding:
//   x'[n][h'][w'][(dh*sw + dw)*C + c] = x[n][sh*h' + dh - ph][sw*w' + dw - pw][c]  (0 outside x)
//   w'[k][r'][s'][(dh*sw + dw)*C + c] = w[k][sh*r' + dh][sw*s' + dw][c]           (0 past R, S)
// so that y[n][p][q][k] = sum over (r', s', c') of w'[k][r'][s'][c'] x'[n][p + r'][q + s'][c'].
// One thread per 16-byte chunk of x' (VEC channels of one rewritten pixel),
// 32-bit index math with precomputed divisors.
template <typename T>
__global__ __launch_bounds__(256) void space_to_depth_kernel(const T* __restrict__ x, T* __restrict__ xs, int H,
                                                             int W, int C, int Hs, int Ws, int sh, int sw, int ph,
                                                             int pw, FastDiv dJ, FastDiv dWs, FastDiv dHs, FastDiv dC,
                                                             FastDiv dSw, int total) {
  constexpr int VEC = 16 / (int)sizeof(T);
  const int J = (int)dJ.d;  // chunks per rewritten pixel
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    const int pix = (int)fdiv((uint32_t)i, dJ);
    const int j = i - pix * J;
    const int t = (int)fdiv((uint32_t)pix, dWs);
    const int wq = pix - t * Ws;
    const int n = (int)fdiv((uint32_t)t, dHs);
    const int hq = t - n * Hs;
    union { uint4 u; T e[VEC]; } v;
#pragma unroll
    for (int u = 0; u < VEC; ++u) {
      const int e = j * VEC + u;
      const int d = (int)fdiv((uint32_t)e, dC);
      const int c = e - d * C;
      const int dh = (int)fdiv((uint32_t)d, dSw);
      const int dw = d - dh * sw;
      const int h = sh * hq + dh - ph, w = sw * wq + dw - pw;
      const bool ok = (unsigned)h < (unsigned)H && (unsigned)w < (unsigned)W;
      v.e[u] = ok ? x[((n * H + h) * W + w) * C + c] : T(0);
    }
    *(uint4*)(xs + (size_t)i * VEC) = v.u;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void filter_to_s2d_kernel(const T* __restrict__ w, T* __restrict__ ws, int R,
                                                            int S, int C, int Rs, int Ss, int sh, int sw,
                                                            int total) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    const int Cs = sh * sw * C;
    const int cs = i % Cs;
    int t = i / Cs;
    const int ss = t % Ss;
    t /= Ss;
    const int rs = t % Rs;
    const int k = t / Rs;
    const int c = cs % C, d = cs / C, dh = d / sw, dw = d % sw;
    const int r = sh * rs + dh, s = sw * ss + dw;
    ws[i] = (r < R && s < S) ? w[((k * R + r) * S + s) * C + c] : T(0);
  }
}

// dw[k][r][s][c] (+)= dws[k][r / sh][s / sw][((r % sh)*sw + s % sw)*C + c] (fp32 filter gradients).
__global__ __launch_bounds__(256) void s2d_to_filter_f32_kernel(const float* __restrict__ dws, float* __restrict__ dw,
                                                                int R, int S, int C, int Rs, int Ss, int sh, int sw,
                                                                int accumulate, int total) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    const int c = i % C;
    int t = i / C;
    const int s = t % S;
    t /= S;
    const int r = t % R;
    const int k = t / R;
    const int Cs = sh * sw * C;
    const float v = dws[((k * Rs + r / sh) * Ss + s / sw) * Cs + ((r % sh) * sw + s % sw) * C + c];
    dw[i] = accumulate ? dw[i] + v : v;
  }
}

// dx[n][h][w][c] = dxs[n][(h + ph) / sh][(w + pw) / sw][(((h + ph) % sh)*sw + (w + pw) % sw)*C + c]
// (0 where that position lies outside dxs: no output window reads it), then
// zeroed where mask <= 0 when a ReLU's output is given.
template <typename T>
__global__ __launch_bounds__(256) void depth_to_space_kernel(const T* __restrict__ dxs, const T* __restrict__ mask,
                                                             T* __restrict__ dx, FastDiv dC, FastDiv dW, FastDiv dH,
                                                             int H, int W, int C, int Hs, int Ws, int sh, int sw,
                                                             int ph, int pw, int total) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    const int t1 = (int)fdiv((uint32_t)i, dC);
    const int c = i - t1 * C;
    const int t2 = (int)fdiv((uint32_t)t1, dW);
    const int w = t1 - t2 * W;
    const int n = (int)fdiv((uint32_t)t2, dH);
    const int h = t2 - n * H;
    const int hq = (h + ph) / sh, wq = (w + pw) / sw;
    float v = 0.f;
    if (hq < Hs && wq < Ws) {
      const int Cs = sh * sw * C;
      v = ld_f<T>(dxs + ((n * Hs + hq) * Ws + wq) * Cs + (((h + ph) % sh) * sw + (w + pw) % sw) * C + c);
    }
    if (mask && !(ld_f<T>(mask + i) > 0.f)) v = 0.f;
    st_f<T>(dx + i, v);
  }
}

// out[r][c] (+)= in[r][c] for c < C: drops the zero-padded channels of an
// fp32 filter gradient computed on a channel-padded input.
__global__ __launch_bounds__(256) void unpad_channels_f32_kernel(const float* __restrict__ in,
                                                                 float* __restrict__ out, long rows, int Cp, int C,
                                                                 int accumulate) {
  const long total = rows * C;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (long)gridDim.x * blockDim.x) {
    const long r = i / C;
    const int c = (int)(i - r * C);
    const float v = in[r * Cp + c];
    out[i] = accumulate ? out[i] + v : v;
  }
}

unsigned grid_for(long total, int block = 256, long cap = 65536) {
  long g = (total + block - 1) / block;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return (unsigned)g;
}

}  // namespace

hipError_t launch_transpose(int dt, const void* in, void* out, int batch, int rows, int cols, long in_bstride,
                            long in_rstride, long out_bstride, long out_rstride, int flip, hipStream_t st) {
  TraceScope ts("transpose_kernel", st, 2.0 * batch * (double)rows * cols * dt_size(dt), WORK_BYTE);
  const long vec = 16 / (long)dt_size(dt);
  if (rows % vec == 0 && cols % vec == 0 && in_rstride % vec == 0 && out_rstride % vec == 0 &&
      in_bstride % vec == 0 && out_bstride % vec == 0 && (uintptr_t)in % 16 == 0 && (uintptr_t)out % 16 == 0) {
    dim3 g64((cols + 63) / 64, (rows + 63) / 64, batch);
    if (dt == BF16)
      hipLaunchKernelGGL(transpose_vec_kernel<bf16_t>, g64, dim3(256), 0, st, (const bf16_t*)in, (bf16_t*)out, batch,
                         rows, cols, in_bstride, in_rstride, out_bstride, out_rstride, flip);
    else
      hipLaunchKernelGGL(transpose_vec_kernel<float>, g64, dim3(256), 0, st, (const float*)in, (float*)out, batch,
                         rows, cols, in_bstride, in_rstride, out_bstride, out_rstride, flip);
    return hipGetLastError();
  }
  dim3 grid((cols + 31) / 32, (rows + 31) / 32, batch), block(256);
  if (dt == BF16)
    hipLaunchKernelGGL(transpose_kernel<bf16_t>, grid, block, 0, st, (const bf16_t*)in, (bf16_t*)out, batch, rows,
                       cols, in_bstride, in_rstride, out_bstride, out_rstride, flip);
  else
    hipLaunchKernelGGL(transpose_kernel<float>, grid, block, 0, st, (const float*)in, (float*)out, batch, rows,
                       cols, in_bstride, in_rstride, out_bstride, out_rstride, flip);
  return hipGetLastError();
}

hipError_t launch_conv_bwd_data_direct(int dt, const ConvShape& s, const void* dy, const void* w, void* dx,
                                       const void* mask, hipStream_t st) {
  const long total = (long)s.N * s.H * s.W * s.C;
  const unsigned g = grid_for(total);
  TraceScope ts("bwd_data_direct_kernel", st,
                2.0 * s.N * (double)s.P * s.Q * s.K * (double)s.C * s.R * s.S, WORK_FLOP);
  if (dt == BF16)
    hipLaunchKernelGGL(bwd_data_direct_kernel<bf16_t>, dim3(g), dim3(256), 0, st, s, (const bf16_t*)dy,
                       (const bf16_t*)w, (const bf16_t*)mask, (bf16_t*)dx, total);
  else
    hipLaunchKernelGGL(bwd_data_direct_kernel<float>, dim3(g), dim3(256), 0, st, s, (const float*)dy,
                       (const float*)w, (const float*)mask, (float*)dx, total);
  return hipGetLastError();
}

hipError_t launch_pad_channels(int dt, const void* in, void* out, long rows, int C, int Cp, hipStream_t st) {
  if (Cp % 4 != 0 || C > Cp) return hipErrorInvalidValue;
  TraceScope ts("pad_channels_kernel", st, (double)rows * (C + Cp) * dt_size(dt), WORK_BYTE);
  const long groups = rows / 8;
  if (C == 3 && Cp == 4 && groups > 0 && (uintptr_t)in % 16 == 0 && (uintptr_t)out % 16 == 0) {
    // vector body over whole groups of 8 rows, generic kernel for the tail
    if (dt == BF16)
      hipLaunchKernelGGL(pad_3to4_kernel<bf16_t>, dim3(grid_for(groups)), dim3(256), 0, st, (const bf16_t*)in,
                         (bf16_t*)out, groups);
    else
      hipLaunchKernelGGL(pad_3to4_kernel<float>, dim3(grid_for(groups)), dim3(256), 0, st, (const float*)in,
                         (float*)out, groups);
    const long done = groups * 8;
    if (done == rows) return hipGetLastError();
    const size_t es = dt_size(dt);
    in = (const char*)in + done * C * es;
    out = (char*)out + done * Cp * es;
    rows -= done;
  }
  const long total = rows * (Cp / 4);
  if (dt == BF16)
    hipLaunchKernelGGL(pad_channels_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, st, (const bf16_t*)in,
                       (bf16_t*)out, rows, C, Cp);
  else
    hipLaunchKernelGGL(pad_channels_kernel<float>, dim3(grid_for(total)), dim3(256), 0, st, (const float*)in,
                       (float*)out, rows, C, Cp);
  return hipGetLastError();
}

hipError_t launch_unpad_channels_f32(const float* in, float* out, long rows, int Cp, int C, int accumulate,
                                     hipStream_t st) {
  const long total = rows * C;
  TraceScope ts("unpad_channels_f32_kernel", st, (double)rows * (C * (accumulate ? 12.0 : 8.0)), WORK_BYTE);
  hipLaunchKernelGGL(unpad_channels_f32_kernel, dim3(grid_for(total)), dim3(256), 0, st, in, out, rows, Cp, C,
                     accumulate);
  return hipGetLastError();
}

hipError_t launch_space_to_depth(int dt, const ConvShape& s, const ConvShape& g, const void* x, void* xs,
                                 hipStream_t st) {
  const int vec = 16 / (int)dt_size(dt);
  if (g.C % vec != 0 || (uintptr_t)xs % 16 != 0) return hipErrorInvalidValue;  // callers guarantee both
  const int J = g.C / vec;
  const int total = g.N * g.H * g.W * J;
  TraceScope ts("space_to_depth_kernel", st,
                ((double)s.N * s.H * s.W * s.C + (double)g.N * g.H * g.W * g.C) * dt_size(dt), WORK_BYTE);
  const FastDiv dJ = make_fastdiv((uint32_t)J), dWs = make_fastdiv((uint32_t)g.W), dHs = make_fastdiv((uint32_t)g.H),
                dC = make_fastdiv((uint32_t)s.C), dSw = make_fastdiv((uint32_t)s.sw);
  if (dt == BF16)
    hipLaunchKernelGGL(space_to_depth_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, st, (const bf16_t*)x,
                       (bf16_t*)xs, s.H, s.W, s.C, g.H, g.W, s.sh, s.sw, s.ph, s.pw, dJ, dWs, dHs, dC, dSw, total);
  else
    hipLaunchKernelGGL(space_to_depth_kernel<float>, dim3(grid_for(total)), dim3(256), 0, st, (const float*)x,
                       (float*)xs, s.H, s.W, s.C, g.H, g.W, s.sh, s.sw, s.ph, s.pw, dJ, dWs, dHs, dC, dSw, total);
  return hipGetLastError();
}

hipError_t launch_filter_to_s2d(int dt, const ConvShape& s, const ConvShape& g, const void* w, void* ws,
                                hipStream_t st) {
  const int total = g.K * g.R * g.S * g.C;
  TraceScope ts("filter_to_s2d_kernel", st, (double)total * 2 * dt_size(dt), WORK_BYTE);
  if (dt == BF16)
    hipLaunchKernelGGL(filter_to_s2d_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, st, (const bf16_t*)w,
                       (bf16_t*)ws, s.R, s.S, s.C, g.R, g.S, s.sh, s.sw, total);
  else
    hipLaunchKernelGGL(filter_to_s2d_kernel<float>, dim3(grid_for(total)), dim3(256), 0, st, (const float*)w,
                       (float*)ws, s.R, s.S, s.C, g.R, g.S, s.sh, s.sw, total);
  return hipGetLastError();
}

hipError_t launch_s2d_to_filter_f32(const ConvShape& s, const ConvShape& g, const float* dws, float* dw,
                                    int accumulate, hipStream_t st) {
  const int total = s.K * s.R * s.S * s.C;
  TraceScope ts("s2d_to_filter_f32_kernel", st, (double)total * (accumulate ? 12.0 : 8.0), WORK_BYTE);
  hipLaunchKernelGGL(s2d_to_filter_f32_kernel, dim3(grid_for(total)), dim3(256), 0, st, dws, dw, s.R, s.S, s.C, g.R,
                     g.S, s.sh, s.sw, accumulate, total);
  return hipGetLastError();
}

hipError_t launch_depth_to_space(int dt, const ConvShape& s, const ConvShape& g, const void* dxs, const void* mask,
                                 void* dx, hipStream_t st) {
  const int total = s.N * s.H * s.W * s.C;
  TraceScope ts("depth_to_space_kernel", st, (double)total * (mask ? 3 : 2) * dt_size(dt), WORK_BYTE);
  const FastDiv dC = make_fastdiv((uint32_t)s.C), dW = make_fastdiv((uint32_t)s.W), dH = make_fastdiv((uint32_t)s.H);
  if (dt == BF16)
    hipLaunchKernelGGL(depth_to_space_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, st, (const bf16_t*)dxs,
                       (const bf16_t*)mask, (bf16_t*)dx, dC, dW, dH, s.H, s.W, s.C, g.H, g.W, s.sh, s.sw, s.ph, s.pw,
                       total);
  else
    hipLaunchKernelGGL(depth_to_space_kernel<float>, dim3(grid_for(total)), dim3(256), 0, st, (const float*)dxs,
                       (const float*)mask, (float*)dx, dC, dW, dH, s.H, s.W, s.C, g.H, g.W, s.sh, s.sw, s.ph, s.pw,
                       total);
  return hipGetLastError();
}

hipError_t launch_nchw_to_nhwc(int dt, const void* in, void* out, int N, int C, int H, int W, hipStream_t st) {
  const int HW = H * W;
  dim3 grid((HW + 31) / 32, (C + 31) / 32, N), block(256);
  TraceScope ts("nchw_to_nhwc_kernel", st, 2.0 * N * (double)C * HW * dt_size(dt), WORK_BYTE);
  if (dt == BF16)
    hipLaunchKernelGGL(nchw_to_nhwc_kernel<bf16_t>, grid, block, 0, st, (const bf16_t*)in, (bf16_t*)out, C, HW);
  else
    hipLaunchKernelGGL(nchw_to_nhwc_kernel<float>, grid, block, 0, st, (const float*)in, (float*)out, C, HW);
  return hipGetLastError();
}

hipError_t launch_nhwc_to_nchw(int dt, const void* in, void* out, int N, int C, int H, int W, hipStream_t st) {
  const int HW = H * W;
  dim3 grid((C + 31) / 32, (HW + 31) / 32, N), block(256);
  TraceScope ts("nhwc_to_nchw_kernel", st, 2.0 * N * (double)C * HW * dt_size(dt), WORK_BYTE);
  if (dt == BF16)
    hipLaunchKernelGGL(nhwc_to_nchw_kernel<bf16_t>, grid, block, 0, st, (const bf16_t*)in, (bf16_t*)out, C, HW);
  else
    hipLaunchKernelGGL(nhwc_to_nchw_kernel<float>, grid, block, 0, st, (const float*)in, (float*)out, C, HW);
  return hipGetLastError();
}

hipError_t launch_krsc_to_kcrs_f32(const float* in, float* out, int K, int C, int R, int S, int accumulate,
                                   hipStream_t st) {
  const long total = (long)K * C * R * S;
  TraceScope ts("krsc_to_kcrs_kernel", st, 4.0 * total * (accumulate ? 3 : 2), WORK_BYTE);
  hipLaunchKernelGGL(krsc_to_kcrs_kernel, dim3(grid_for(total)), dim3(256), 0, st, in, out, K, C, R * S,
                     accumulate);
  return hipGetLastError();
}

}  // namespace singa
