// conv_igemm.hip -- convolution as implicit GEMM on gfx950 matrix cores.
//
// Forward (ComputeFeature of the convolution layer, Sec. 4.1.2):
//   GEMM rows    m = (n, p, q) output pixels      (M = N*P*Q)
//   GEMM columns j = k output channels            (Nn = K)
//   reduction    t = (r, s, c) filter taps        (Kg = R*S*C)
//   A[m][t] = x[n, p*sh-ph+r, q*sw-pw+s, c] (zero outside), B[j][t] = w[k][r][s][c]
// Both operands are contiguous along t in NHWC/KRSC, so 16-byte vectors of
// consecutive taps are read straight from HBM into LDS rows.
//
// Filter gradient (ComputeGradient, Param gradients):
//   rows i = k, columns j = (r, s, c), reduction t = (n, p, q)
//   A[i][t] = dy[n,p,q,k], B[j][t] = x[n, p*sh-ph+r, q*sw-pw+s, c]
// Here both operands are contiguous along i/j instead of t, so each thread
// loads a small (t x 4) block and transposes it in registers before writing
// the LDS rows.  The t range is split across workgroups (split-K); partial
// sums go to a buffer that a second kernel reduces in a fixed order.
//
// Tiling: 256 threads (4 wave64) per workgroup, a 128 x 128 output tile,
// each wave a 64 x 64 quadrant made of 2 x 2 blocks of 32 x 32 MFMA
// (v_mfma_f32_32x32x2_f32 for fp32, v_mfma_f32_32x32x16_bf16 for bf16).
// A K-tile is 128 bytes of every operand row (32 fp32 or 64 bf16 taps); LDS
// rows are padded to 144 bytes so the 16-byte fragment reads of 16
// consecutive rows hit distinct banks.  Two LDS stages: global loads of tile
// k+1 are in flight while tile k is multiplied.
#include "common.h"
#include "internal.h"

namespace singa {

namespace {

constexpr int NT = 256;
constexpr int BM = 128;
constexpr int BN = 128;
constexpr int ROWB = 128;               // bytes of one operand row per K-tile
constexpr int PITCH = ROWB + 16;        // padded LDS row pitch
constexpr int TILE = BM * PITCH;        // bytes of one operand tile
constexpr int SMEM = 2 * 2 * TILE;      // 2 stages x (A, B)

template <typename T> struct KT {
  static constexpr int VEC = 16 / (int)sizeof(T);  // elements per 16 bytes
  static constexpr int BK = ROWB / (int)sizeof(T); // taps per K-tile
};

union V16 {
  uint4 u;
  float f[4];
  bf16_t h[8];
};

template <typename T> __device__ __forceinline__ void set_elem(V16& v, int j, T e);
template <> __device__ __forceinline__ void set_elem<float>(V16& v, int j, float e) { v.f[j] = e; }
template <> __device__ __forceinline__ void set_elem<bf16_t>(V16& v, int j, bf16_t e) { v.h[j] = e; }

template <typename T> __device__ __forceinline__ T zero_elem();
template <> __device__ __forceinline__ float zero_elem<float>() { return 0.f; }
template <> __device__ __forceinline__ bf16_t zero_elem<bf16_t>() { return (bf16_t)0; }

template <typename T> __device__ __forceinline__ void store_out(T* p, float v);
template <> __device__ __forceinline__ void store_out<float>(float* p, float v) { *p = v; }
template <> __device__ __forceinline__ void store_out<bf16_t>(bf16_t* p, float v) { *p = f32_to_bf16(v); }

// Multiply one K-tile held in LDS: acc[bm][bn] += A(rows) * B(cols)^T.
template <typename T>
__device__ __forceinline__ void mma_tile(const char* As, const char* Bs, f32x16 (&acc)[2][2], int wm, int wn,
                                         int lane) {
  typedef typename Frag<T>::type FragT;
  const int li = lane & 31, lh = lane >> 5;
  const char* ab = As + (wm * 64 + li) * PITCH + lh * 16;
  const char* bb = Bs + (wn * 64 + li) * PITCH + lh * 16;
#pragma unroll
  for (int kc = 0; kc < ROWB / 32; ++kc) {
    FragT a0 = *(const FragT*)(ab + kc * 32);
    FragT a1 = *(const FragT*)(ab + 32 * PITCH + kc * 32);
    FragT b0 = *(const FragT*)(bb + kc * 32);
    FragT b1 = *(const FragT*)(bb + 32 * PITCH + kc * 32);
    if constexpr (sizeof(T) == 2) {
      acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b1, acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, acc[1][1], 0, 0, 0);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[j], b0[j], acc[0][0], 0, 0, 0);
        acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[j], b1[j], acc[0][1], 0, 0, 0);
        acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[j], b0[j], acc[1][0], 0, 0, 0);
        acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[j], b1[j], acc[1][1], 0, 0, 0);
      }
    }
  }
}

// ------------------------------------------------------------------ forward

struct FwdArgs {
  const void* x;
  const void* w;
  const float* bias;
  void* y;
  int M, Nn, Kg;
  int H, W, C, S, P, Q;
  int sh, sw, ph, pw;
  FastDiv dPQ, dQ, dC, dS;
  int relu;
  int tiles_n;
};

// VA: A taps are loaded as 16-byte vectors (C % VEC == 0); otherwise element
// by element.  VB: likewise for the filter rows (Kg % VEC == 0).  BWD only
// names the instance that serves backward-data, so profiles tell them apart.
template <typename T, bool VA, bool VB, bool BWD>
__global__ __launch_bounds__(NT) void conv_fwd_kernel(FwdArgs a) {
  constexpr int VEC = KT<T>::VEC;
  constexpr int BK = KT<T>::BK;
  __shared__ __attribute__((aligned(16))) char smem[SMEM];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int tm = blockIdx.x / a.tiles_n, tn = blockIdx.x - tm * a.tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  const T* __restrict__ xp = (const T*)a.x;
  const T* __restrict__ wp = (const T*)a.w;

  // Each thread fills one 16-byte column (cv) of 4 rows (rl + 32 i) of each operand.
  const int cv = tid & 7, rl = tid >> 3;
  int abase[4], ah0[4], aw0[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int m = m0 + rl + 32 * i;
    if (m < a.M) {
      int n = (int)fdiv((uint32_t)m, a.dPQ);
      int pq = m - n * a.P * a.Q;
      int p = (int)fdiv((uint32_t)pq, a.dQ);
      int q = pq - p * a.Q;
      abase[i] = n * a.H * a.W * a.C;
      ah0[i] = p * a.sh - a.ph;
      aw0[i] = q * a.sw - a.pw;
    } else {
      abase[i] = 0;
      ah0[i] = -(1 << 28);  // fails every bounds check
      aw0[i] = 0;
    }
  }
  int brow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int n = n0 + rl + 32 * i;
    brow[i] = n < a.Nn ? n : -1;
  }

  V16 ra[4], rb[4];
  auto load_tile = [&](int k0) {
    const int kk = k0 + cv * VEC;
    if constexpr (VA) {
      const bool kin = kk < a.Kg;
      int rs = (int)fdiv((uint32_t)kk, a.dC);
      int c = kk - rs * a.C;
      int r = (int)fdiv((uint32_t)rs, a.dS);
      int s = rs - r * a.S;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int h = ah0[i] + r, w = aw0[i] + s;
        bool ok = kin && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
        ra[i].u = ok ? *(const uint4*)(xp + abase[i] + (h * a.W + w) * a.C + c) : make_uint4(0, 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int j = 0; j < VEC; ++j) {
        int kj = kk + j;
        const bool kin = kj < a.Kg;
        int rs = (int)fdiv((uint32_t)kj, a.dC);
        int c = kj - rs * a.C;
        int r = (int)fdiv((uint32_t)rs, a.dS);
        int s = rs - r * a.S;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          int h = ah0[i] + r, w = aw0[i] + s;
          bool ok = kin && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
          set_elem<T>(ra[i], j, ok ? xp[abase[i] + (h * a.W + w) * a.C + c] : zero_elem<T>());
        }
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if constexpr (VB) {
        bool ok = brow[i] >= 0 && kk < a.Kg;
        rb[i].u = ok ? *(const uint4*)(wp + (size_t)brow[i] * a.Kg + kk) : make_uint4(0, 0, 0, 0);
      } else {
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
          bool ok = brow[i] >= 0 && kk + j < a.Kg;
          set_elem<T>(rb[i], j, ok ? wp[(size_t)brow[i] * a.Kg + kk + j] : zero_elem<T>());
        }
      }
    }
  };
  auto store_tile = [&](int stage) {
    char* As = smem + stage * 2 * TILE;
    char* Bs = As + TILE;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *(uint4*)(As + (rl + 32 * i) * PITCH + cv * 16) = ra[i].u;
      *(uint4*)(Bs + (rl + 32 * i) * PITCH + cv * 16) = rb[i].u;
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int wm = wave >> 1, wn = wave & 1;
  const int nkt = (a.Kg + BK - 1) / BK;
  load_tile(0);
  store_tile(0);
  __syncthreads();
  for (int kt = 0; kt < nkt; ++kt) {
    const bool more = kt + 1 < nkt;
    if (more) load_tile((kt + 1) * BK);
    const char* As = smem + (kt & 1) * 2 * TILE;
    mma_tile<T>(As, As + TILE, acc, wm, wn, lane);
    if (more) store_tile((kt + 1) & 1);
    __syncthreads();
  }

  // Epilogue: lane holds column li of each 32x32 block, rows 8*(v/4) + 4*lh + v%4.
  T* __restrict__ yp = (T*)a.y;
  const int li = lane & 31, lh = lane >> 5;
#pragma unroll
  for (int bn = 0; bn < 2; ++bn) {
    const int col = n0 + wn * 64 + bn * 32 + li;
    if (col >= a.Nn) continue;
    const float bv = a.bias ? a.bias[col] : 0.f;
#pragma unroll
    for (int bm = 0; bm < 2; ++bm) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = m0 + wm * 64 + bm * 32 + (v >> 2) * 8 + lh * 4 + (v & 3);
        if (row < a.M) {
          float val = acc[bm][bn][v] + bv;
          if (a.relu) val = fmaxf(val, 0.f);
          store_out<T>(yp + (size_t)row * a.Nn + col, val);
        }
      }
    }
  }
}

// ----------------------------------------------------------- filter gradient

struct WgradArgs {
  const void* x;
  const void* dy;
  float* partial;  // [splits][M][Nn]
  int M, Nn, T;    // M = K filters, Nn = R*S*C, T = N*P*Q
  int H, W, C, S, P, Q;
  int sh, sw, ph, pw;
  FastDiv dPQ, dQ, dC, dS;
  int tiles_n, kt_per_split, nkt;
};

// Rows of the thread's (TR x 4) block: TR = VEC taps of t, 4 columns.
// VA: dy columns loaded 4 at a time (M % 4 == 0); VB: x columns 4 at a time (C % 4 == 0).
template <typename T, bool VA, bool VB>
__global__ __launch_bounds__(NT) void conv_wgrad_kernel(WgradArgs a) {
  constexpr int TR = KT<T>::VEC;  // t-rows per block = elements per 16-byte LDS write
  constexpr int BK = KT<T>::BK;
  __shared__ __attribute__((aligned(16))) char smem[SMEM];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int tm = blockIdx.x / a.tiles_n, tn = blockIdx.x - tm * a.tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  const int split = blockIdx.y;
  const int kt_begin = split * a.kt_per_split;
  const int kt_end = min(a.nkt, kt_begin + a.kt_per_split);
  const T* __restrict__ xp = (const T*)a.x;
  const T* __restrict__ dyp = (const T*)a.dy;

  // thread -> (t-block tb, 4-column block cb); the same mapping serves A and B
  const int tb = tid & 7, cb = tid >> 3;
  const int i0 = m0 + cb * 4;  // first dy column (filter) of this thread
  const int j0 = n0 + cb * 4;  // first tap column of this thread
  // Taps of the four B columns (fixed for the whole reduction).
  int br[4], bs[4], bc[4];
  bool bok[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    int j = j0 + u;
    bok[u] = j < a.Nn;
    int jj = bok[u] ? j : 0;
    int rs = (int)fdiv((uint32_t)jj, a.dC);
    bc[u] = jj - rs * a.C;
    br[u] = (int)fdiv((uint32_t)rs, a.dS);
    bs[u] = rs - br[u] * a.S;
  }

  V16 ra[4], rb[4];
  auto load_tile = [&](int kt) {
    const int t0 = kt * BK + tb * TR;
    // decompose the first t of the block, then step along q
    int n = (int)fdiv((uint32_t)t0, a.dPQ);
    int pq = t0 - n * a.P * a.Q;
    int p = (int)fdiv((uint32_t)pq, a.dQ);
    int q = pq - p * a.Q;
    T av[TR][4], bv[TR][4];
#pragma unroll
    for (int e = 0; e < TR; ++e) {
      const int t = t0 + e;
      const bool tin = t < a.T;
      // A: dy[t][i0 .. i0+3]
      if constexpr (VA) {
        if (tin && i0 < a.M) {
          const T* src = dyp + (size_t)t * a.M + i0;
          if constexpr (sizeof(T) == 4) {
            float4 v = *(const float4*)src;
            av[e][0] = v.x; av[e][1] = v.y; av[e][2] = v.z; av[e][3] = v.w;
          } else {
            uint2 v = *(const uint2*)src;
            av[e][0] = (bf16_t)(v.x & 0xffffu); av[e][1] = (bf16_t)(v.x >> 16);
            av[e][2] = (bf16_t)(v.y & 0xffffu); av[e][3] = (bf16_t)(v.y >> 16);
          }
        } else {
#pragma unroll
          for (int u = 0; u < 4; ++u) av[e][u] = zero_elem<T>();
        }
      } else {
#pragma unroll
        for (int u = 0; u < 4; ++u)
          av[e][u] = (tin && i0 + u < a.M) ? dyp[(size_t)t * a.M + i0 + u] : zero_elem<T>();
      }
      // B: x[n, p*sh-ph+r, q*sw-pw+s, c] for the four tap columns
      const int hb = p * a.sh - a.ph, wb = q * a.sw - a.pw;
      const int xbase = n * a.H * a.W * a.C;
      if constexpr (VB) {
        const int h = hb + br[0], w = wb + bs[0];
        const bool ok = tin && bok[0] && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
        if (ok) {
          const T* src = xp + xbase + (h * a.W + w) * a.C + bc[0];
          if constexpr (sizeof(T) == 4) {
            float4 v = *(const float4*)src;
            bv[e][0] = v.x; bv[e][1] = v.y; bv[e][2] = v.z; bv[e][3] = v.w;
          } else {
            uint2 v = *(const uint2*)src;
            bv[e][0] = (bf16_t)(v.x & 0xffffu); bv[e][1] = (bf16_t)(v.x >> 16);
            bv[e][2] = (bf16_t)(v.y & 0xffffu); bv[e][3] = (bf16_t)(v.y >> 16);
          }
        } else {
#pragma unroll
          for (int u = 0; u < 4; ++u) bv[e][u] = zero_elem<T>();
        }
      } else {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int h = hb + br[u], w = wb + bs[u];
          const bool ok = tin && bok[u] && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
          bv[e][u] = ok ? xp[xbase + (h * a.W + w) * a.C + bc[u]] : zero_elem<T>();
        }
      }
      // step to the next output pixel
      if (++q == a.Q) {
        q = 0;
        if (++p == a.P) {
          p = 0;
          ++n;
        }
      }
    }
    // transpose: LDS row = column u, 16 bytes = the TR t-values
#pragma unroll
    for (int u = 0; u < 4; ++u) {
#pragma unroll
      for (int e = 0; e < TR; ++e) {
        set_elem<T>(ra[u], e, av[e][u]);
        set_elem<T>(rb[u], e, bv[e][u]);
      }
    }
  };
  auto store_tile = [&](int stage) {
    char* As = smem + stage * 2 * TILE;
    char* Bs = As + TILE;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      *(uint4*)(As + (cb * 4 + u) * PITCH + tb * 16) = ra[u].u;
      *(uint4*)(Bs + (cb * 4 + u) * PITCH + tb * 16) = rb[u].u;
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int wm = wave >> 1, wn = wave & 1;
  if (kt_begin < kt_end) {
    load_tile(kt_begin);
    store_tile(0);
    __syncthreads();
    for (int kt = kt_begin; kt < kt_end; ++kt) {
      const bool more = kt + 1 < kt_end;
      if (more) load_tile(kt + 1);
      const char* As = smem + ((kt - kt_begin) & 1) * 2 * TILE;
      mma_tile<T>(As, As + TILE, acc, wm, wn, lane);
      if (more) store_tile((kt + 1 - kt_begin) & 1);
      __syncthreads();
    }
  }

  float* __restrict__ out = a.partial + (size_t)split * a.M * a.Nn;
  const int li = lane & 31, lh = lane >> 5;
#pragma unroll
  for (int bn = 0; bn < 2; ++bn) {
    const int col = n0 + wn * 64 + bn * 32 + li;
    if (col >= a.Nn) continue;
#pragma unroll
    for (int bm = 0; bm < 2; ++bm) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = m0 + wm * 64 + bm * 32 + (v >> 2) * 8 + lh * 4 + (v & 3);
        if (row < a.M) out[(size_t)row * a.Nn + col] = acc[bm][bn][v];
      }
    }
  }
}

__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ partial, int splits,
                                                            size_t n, float* __restrict__ dw, int accumulate) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    float s = accumulate ? dw[i] : 0.f;
    float t = 0.f;
    for (int k = 0; k < splits; ++k) t += partial[(size_t)k * n + i];
    dw[i] = s + t;
  }
}

template <typename T> constexpr const char* tname();
template <> constexpr const char* tname<float>() { return "f32"; }
template <> constexpr const char* tname<bf16_t>() { return "bf16"; }

// "conv_fwd_kernel<dtype,vecA,vecB,bwd>" for each instance
template <typename T, bool VA, bool VB, bool BWD> const char* fwd_name() {
  static const char* names[2][2][2] = {
      {{"conv_fwd_kernel<%s,0,0,0>", "conv_fwd_kernel<%s,0,0,1>"},
       {"conv_fwd_kernel<%s,0,1,0>", "conv_fwd_kernel<%s,0,1,1>"}},
      {{"conv_fwd_kernel<%s,1,0,0>", "conv_fwd_kernel<%s,1,0,1>"},
       {"conv_fwd_kernel<%s,1,1,0>", "conv_fwd_kernel<%s,1,1,1>"}}};
  static char buf[2][2][2][48];
  static bool init = false;
  if (!init) {
    for (int i = 0; i < 2; ++i)
      for (int j = 0; j < 2; ++j)
        for (int k = 0; k < 2; ++k) snprintf(buf[i][j][k], sizeof buf[i][j][k], names[i][j][k], tname<T>());
    init = true;
  }
  return buf[VA][VB][BWD];
}

template <typename T, bool VA, bool VB, bool BWD>
void launch_fwd_instance(const FwdArgs& a, dim3 grid, double flops, hipStream_t st) {
  TraceScope ts(fwd_name<T, VA, VB, BWD>(), st, flops, WORK_FLOP);
  hipLaunchKernelGGL((conv_fwd_kernel<T, VA, VB, BWD>), grid, dim3(NT), 0, st, a);
}

template <typename T, bool BWD>
void launch_fwd_variant(bool va, bool vb, const FwdArgs& a, dim3 grid, double flops, hipStream_t st) {
  if (va && vb) launch_fwd_instance<T, true, true, BWD>(a, grid, flops, st);
  else if (vb) launch_fwd_instance<T, false, true, BWD>(a, grid, flops, st);
  else if (va) launch_fwd_instance<T, true, false, BWD>(a, grid, flops, st);
  else launch_fwd_instance<T, false, false, BWD>(a, grid, flops, st);
}

template <typename T>
hipError_t conv_fwd_dispatch(const ConvShape& s, const void* x, const void* w, const float* bias, void* y,
                             int relu, int bwd, double flops, hipStream_t st) {
  constexpr int VEC = KT<T>::VEC;
  FwdArgs a;
  a.x = x; a.w = w; a.bias = bias; a.y = y;
  a.M = s.N * s.P * s.Q;
  a.Nn = s.K;
  a.Kg = s.R * s.S * s.C;
  a.H = s.H; a.W = s.W; a.C = s.C; a.S = s.S; a.P = s.P; a.Q = s.Q;
  a.sh = s.sh; a.sw = s.sw; a.ph = s.ph; a.pw = s.pw;
  a.dPQ = make_fastdiv((uint32_t)(s.P * s.Q));
  a.dQ = make_fastdiv((uint32_t)s.Q);
  a.dC = make_fastdiv((uint32_t)s.C);
  a.dS = make_fastdiv((uint32_t)s.S);
  a.relu = relu;
  const int tiles_m = (a.M + BM - 1) / BM;
  a.tiles_n = (a.Nn + BN - 1) / BN;
  dim3 grid(tiles_m * a.tiles_n);
  const bool va = (s.C % VEC) == 0 && ((uintptr_t)x % 16) == 0;
  const bool vb = (a.Kg % VEC) == 0 && ((uintptr_t)w % 16) == 0;
  if (bwd)
    launch_fwd_variant<T, true>(va, vb, a, grid, flops, st);
  else
    launch_fwd_variant<T, false>(va, vb, a, grid, flops, st);
  return hipGetLastError();
}

template <typename T, bool VA, bool VB> const char* wgrad_name() {
  static char buf[48];
  static bool init = false;
  if (!init) {
    snprintf(buf, sizeof buf, "conv_wgrad_kernel<%s,%d,%d>", tname<T>(), (int)VA, (int)VB);
    init = true;
  }
  return buf;
}

template <typename T, bool VA, bool VB>
void launch_wgrad_instance(const WgradArgs& a, dim3 grid, double flops, hipStream_t st) {
  TraceScope ts(wgrad_name<T, VA, VB>(), st, flops, WORK_FLOP);
  hipLaunchKernelGGL((conv_wgrad_kernel<T, VA, VB>), grid, dim3(NT), 0, st, a);
}

template <typename T>
hipError_t conv_wgrad_dispatch(const ConvShape& s, const void* x, const void* dy, float* partial, hipStream_t st) {
  WgradArgs a;
  a.x = x; a.dy = dy; a.partial = partial;
  a.M = s.K;
  a.Nn = s.R * s.S * s.C;
  a.T = s.N * s.P * s.Q;
  a.H = s.H; a.W = s.W; a.C = s.C; a.S = s.S; a.P = s.P; a.Q = s.Q;
  a.sh = s.sh; a.sw = s.sw; a.ph = s.ph; a.pw = s.pw;
  a.dPQ = make_fastdiv((uint32_t)(s.P * s.Q));
  a.dQ = make_fastdiv((uint32_t)s.Q);
  a.dC = make_fastdiv((uint32_t)s.C);
  a.dS = make_fastdiv((uint32_t)s.S);
  const int tiles_m = (a.M + BM - 1) / BM;
  a.tiles_n = (a.Nn + BN - 1) / BN;
  constexpr int BK = KT<T>::BK;
  a.nkt = (a.T + BK - 1) / BK;
  const int splits = wgrad_splits(s);
  a.kt_per_split = (a.nkt + splits - 1) / splits;
  dim3 grid(tiles_m * a.tiles_n, splits);
  const bool va = (a.M % 4) == 0 && ((uintptr_t)dy % (4 * sizeof(T))) == 0;
  const bool vb = (s.C % 4) == 0 && ((uintptr_t)x % (4 * sizeof(T))) == 0;
  const double flops = 2.0 * a.M * (double)a.Nn * (double)a.T;
  if (va && vb)
    launch_wgrad_instance<T, true, true>(a, grid, flops, st);
  else if (va)
    launch_wgrad_instance<T, true, false>(a, grid, flops, st);
  else if (vb)
    launch_wgrad_instance<T, false, true>(a, grid, flops, st);
  else
    launch_wgrad_instance<T, false, false>(a, grid, flops, st);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_conv_fwd(int dt, const ConvShape& s, const void* x, const void* w, const float* bias, void* y,
                           int relu, int bwd, double flops, hipStream_t st) {
  if (dt == BF16) return conv_fwd_dispatch<bf16_t>(s, x, w, bias, y, relu, bwd, flops, st);
  return conv_fwd_dispatch<float>(s, x, w, bias, y, relu, bwd, flops, st);
}

int wgrad_splits(const ConvShape& s) {
  const long M = s.K, Nn = (long)s.R * s.S * s.C, T = (long)s.N * s.P * s.Q;
  const long tiles = ((M + BM - 1) / BM) * ((Nn + BN - 1) / BN);
  const long nkt = (T + 31) / 32;  // fp32 K-tiles (bf16 tiles are twice as long)
  // aim for about 4 workgroups per CU on 256 CUs, at least 8 K-tiles per split
  long splits = (1024 + tiles - 1) / tiles;
  long max_by_len = nkt / 8;
  if (splits > max_by_len) splits = max_by_len;
  if (splits < 1) splits = 1;
  if (splits > 256) splits = 256;
  return (int)splits;
}

size_t wgrad_partial_bytes(const ConvShape& s) {
  return (size_t)wgrad_splits(s) * s.K * s.R * s.S * s.C * sizeof(float);
}

hipError_t launch_conv_wgrad(int dt, const ConvShape& s, const void* x, const void* dy, float* partial,
                             hipStream_t st) {
  if (dt == BF16) return conv_wgrad_dispatch<bf16_t>(s, x, dy, partial, st);
  return conv_wgrad_dispatch<float>(s, x, dy, partial, st);
}

hipError_t launch_splitk_reduce(const float* partial, int splits, size_t n, float* dw, int accumulate,
                                hipStream_t st) {
  size_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  TraceScope ts("splitk_reduce_kernel", st, (double)n * 4.0 * (splits + 1 + (accumulate ? 1 : 0)), WORK_BYTE);
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, st, partial, splits, n, dw,
                     accumulate);
  return hipGetLastError();
}

}  // namespace singa
