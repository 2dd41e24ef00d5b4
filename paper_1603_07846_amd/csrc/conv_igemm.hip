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
#include <algorithm>
#include <cstdlib>

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
constexpr int BT_PITCH = 320;            // transposed-filter mode: 256-byte tap-major B row (128 columns) + 64
constexpr int BT_TILE = 64 * BT_PITCH;   // its B tile of one K-tile (64 bf16 taps)
constexpr int BT_SMEM = 2 * (TILE + BT_TILE);

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

template <typename T> __device__ __forceinline__ T one_elem();
template <> __device__ __forceinline__ float one_elem<float>() { return 1.f; }
template <> __device__ __forceinline__ bf16_t one_elem<bf16_t>() { return (bf16_t)0x3f80; }

template <typename T> __device__ __forceinline__ T zero_elem();
template <> __device__ __forceinline__ float zero_elem<float>() { return 0.f; }
template <> __device__ __forceinline__ bf16_t zero_elem<bf16_t>() { return (bf16_t)0; }

template <typename T> __device__ __forceinline__ void store_out(T* p, float v);
template <> __device__ __forceinline__ void store_out<float>(float* p, float v) { *p = v; }
template <> __device__ __forceinline__ void store_out<bf16_t>(bf16_t* p, float v) { *p = f32_to_bf16(v); }

__device__ __forceinline__ float elem_f(float v) { return v; }
__device__ __forceinline__ float elem_f(bf16_t v) { return bf16_to_f32(v); }

// ReLU backward folded into an epilogue: keep v where the ReLU's output is > 0.
template <typename T> __device__ __forceinline__ bool mask_pass(const void* m, size_t i);
template <> __device__ __forceinline__ bool mask_pass<float>(const void* m, size_t i) {
  return ((const float*)m)[i] > 0.f;
}
template <> __device__ __forceinline__ bool mask_pass<bf16_t>(const void* m, size_t i) {
  return bf16_to_f32(((const bf16_t*)m)[i]) > 0.f;
}

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

typedef short v4i16 __attribute__((ext_vector_type(4)));

// ds_read_b64_tr_b16: within each 16-lane group, lane i receives element
// i % 4 of the 8-byte chunks addressed by lanes 4k + i / 4 (k = 0..3).
__device__ __forceinline__ v4i16 lds_tr16(const char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4i16*)(__attribute__((address_space(3))) char*)p);
}

// The same K-tile product with the B operand in tap-major rows (BT_PITCH
// bytes, 128 columns each; the transposed-filter mode): A fragments as in
// mma_tile, B fragments (8 consecutive taps of one column) from pairs of
// transposing reads.  bf16 only.
__device__ __forceinline__ void mma_tile_bt(const char* As, const char* Bs, f32x16 (&acc)[2][2], int wm, int wn,
                                            int lane) {
  const int li = lane & 31, lh = lane >> 5;
  const char* ab = As + (wm * 64 + li) * PITCH + lh * 16;
  // lane l: column (l & 15) of a 16-column group, taps 8 (l >> 5) + 0..7 of the 16-tap step
  const int g = lane >> 4, sl = lane & 15;
  const int row = 8 * (g >> 1) + (sl >> 2);
  const int colb = 2 * (16 * (g & 1) + 4 * (sl & 3));
  const char* bb = Bs + row * BT_PITCH + 2 * (wn * 64) + colb;
#pragma unroll
  for (int kc = 0; kc < ROWB / 32; ++kc) {
    const bf16x8 a0 = *(const bf16x8*)(ab + kc * 32);
    const bf16x8 a1 = *(const bf16x8*)(ab + 32 * PITCH + kc * 32);
    bf16x8 bfr[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const v4i16 lo = lds_tr16(bb + kc * 16 * BT_PITCH + b * 64);
      const v4i16 hi = lds_tr16(bb + (kc * 16 + 4) * BT_PITCH + b * 64);
      bfr[b] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    }
    acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, bfr[0], acc[0][0], 0, 0, 0);
    acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, bfr[1], acc[0][1], 0, 0, 0);
    acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, bfr[0], acc[1][0], 0, 0, 0);
    acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, bfr[1], acc[1][1], 0, 0, 0);
  }
}

// ------------------------------------------------------------ global loads
//
// Operands are read with raw buffer loads: a tap outside the input (padding,
// ragged tails) gets the offset OOB, past the end of every tensor, and the
// hardware returns zeros for it.  No branch, no select on the loaded data.
constexpr uint32_t OOB = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ uint4 ld16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
}
__device__ __forceinline__ uint2 ld8(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0));
}
template <typename T> __device__ __forceinline__ T ld_elem(__amdgpu_buffer_rsrc_t r, uint32_t off);
template <> __device__ __forceinline__ float ld_elem<float>(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0));
}
template <> __device__ __forceinline__ bf16_t ld_elem<bf16_t>(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return (bf16_t)__builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, 0);
}

// Workgroups are dealt to the 8 XCDs round-robin; give each XCD a contiguous
// run of tiles so neighbouring tiles (shared input rows, shared filters) meet
// in the same L2.
__device__ __forceinline__ int xcd_remap(int b, int G) {
  const int q = G >> 3, r = G & 7, x = b & 7, l = b >> 3;
  return x * q + min(x, r) + l;
}

// All-ones in the bits of each element of a 32-bit word that is > 0 (not
// NaN), zero elsewhere, from the bit patterns alone: with x = bits - 1 taken
// as a signed integer, an element is > 0 exactly when 0 <= x < bits(+inf).
// Integer arithmetic only, so a mask of many elements needs no condition
// registers.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));

template <typename T> __device__ __forceinline__ uint32_t positive_bits(uint32_t w);
template <> __device__ __forceinline__ uint32_t positive_bits<bf16_t>(uint32_t w) {
  const int32_t xl = (int32_t)(w & 0xffffu) - 1, xh = (int32_t)(w >> 16) - 1;
  const uint32_t ml = (uint32_t)(((xl - 0x7f80) >> 31) & ~(xl >> 31)) & 0xffffu;
  const uint32_t mh = (uint32_t)(((xh - 0x7f80) >> 31) & ~(xh >> 31)) << 16;
  return ml | mh;
}
template <> __device__ __forceinline__ uint32_t positive_bits<float>(uint32_t w) {
  const uint32_t x = w - 1u;
  return (uint32_t)(((int32_t)(x - 0x7f800000u) >> 31) & ~((int32_t)x >> 31));
}

// ------------------------------------------------------------ epilogue
//
// y[row][col] = act(acc + bias[col]), optionally zeroed where mask <= 0, for
// row blocks B0 .. B0 + NB - 1 of one wave's (32 FM) x (32 FN) quadrant of
// the output tile (row0: the first row of block B0).  The accumulators hold
// one column per lane (rows 8 (v / 4) + 4 (lane / 32) + v % 4 of each 32 x 32
// block); they go through the wave's own LDS region as T so that the global
// stores (and the mask loads) are 16-byte vectors of consecutive columns.
// Needs (32 NB) * (32 FN * sizeof(T) + 16) bytes of LDS at `lds`; the caller
// has finished with the operand tiles there (barrier).  `vec`: y, mask and Nn
// allow 16-byte vectors; otherwise the staged values are stored one by one.
template <typename T, int FM, int FN, int B0 = 0, int NB = FM>
__device__ __forceinline__ void store_quadrant(const f32x16 (&acc)[FM][FN], char* lds, int lane, int row0, int col0,
                                               int M, int Nn, const float* bias, int relu, const void* mask,
                                               T* __restrict__ y, bool vec) {
  constexpr int ES = (int)sizeof(T);
  constexpr int COLS = FN * 32;
  constexpr int PIT = COLS * ES + 16;
  constexpr int VEC = 16 / ES;
  constexpr int CPR = COLS / VEC;    // 16-byte chunks per row
  constexpr int RPS = 64 / CPR;      // rows per pass of the wave (lanes past RPS * CPR idle)
  constexpr int PASSES = (NB * 32 + RPS - 1) / RPS;
  const int li = lane & 31, lh = lane >> 5;
  const int cc = lane % CPR, rr = lane / CPR;
  const int col = col0 + cc * VEC;
  const T* __restrict__ mk = (const T*)mask;
  // The mask vectors of every pass are requested before the values are
  // staged, so their latency overlaps the staging and each other (one load
  // waited for per pass would expose a memory latency per pass).
  uint4 mv[PASSES];
  if (vec && mk) {
#pragma unroll
    for (int pass = 0; pass < PASSES; ++pass) {
      const int r = pass * RPS + rr;
      const int row = row0 + r;
      // every lane loads (element 0 stands in for rows and columns past the
      // end), so no load sits in a branch that the next must wait for
      const bool ok = rr < RPS && r < NB * 32 && row < M && col < Nn;
      mv[pass] = *(const uint4*)(mk + (ok ? (size_t)row * Nn + col : 0));
    }
  }
#pragma unroll
  for (int bn = 0; bn < FN; ++bn) {
    const int c = bn * 32 + li;
    const float bv = (bias && col0 + c < Nn) ? bias[col0 + c] : 0.f;
#pragma unroll
    for (int bm = B0; bm < B0 + NB; ++bm)
#pragma unroll
      for (int v = 0; v < 16; v += 2) {
        // rows r and r + 1 of column c
        float v0 = acc[bm][bn][v] + bv, v1 = acc[bm][bn][v + 1] + bv;
        if (relu) {
          v0 = fmaxf(v0, 0.f);
          v1 = fmaxf(v1, 0.f);
        }
        const int r = (bm - B0) * 32 + (v >> 2) * 8 + lh * 4 + (v & 3);
        if constexpr (sizeof(T) == 2) {
          // one conversion instruction rounds both (the per-element
          // software rounding costs about six VALU operations per value)
          const uint32_t p = f32x2_to_bf16x2(v0, v1);
          *(uint16_t*)(lds + r * PIT + c * ES) = (uint16_t)p;
          *(uint16_t*)(lds + (r + 1) * PIT + c * ES) = (uint16_t)(p >> 16);
        } else {
          store_out<T>((T*)(lds + r * PIT + c * ES), v0);
          store_out<T>((T*)(lds + (r + 1) * PIT + c * ES), v1);
        }
      }
  }
  __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes are done
  __builtin_amdgcn_wave_barrier();
  if (rr >= RPS) return;
  if (vec) {
#pragma unroll
    for (int pass = 0; pass < PASSES; ++pass) {
      const int r = pass * RPS + rr;
      const int row = row0 + r;
      if (r >= NB * 32) break;
      uint4 val = *(const uint4*)(lds + r * PIT + cc * 16);
      if (row < M && col < Nn) {
        if (mk) {
          val.x &= positive_bits<T>(mv[pass].x);
          val.y &= positive_bits<T>(mv[pass].y);
          val.z &= positive_bits<T>(mv[pass].z);
          val.w &= positive_bits<T>(mv[pass].w);
        }
        // streamed past the caches' write allocation (measured 0.5-3 % faster
        // per layer, the consumers included)
        __builtin_nontemporal_store(__builtin_bit_cast(u32x4_t, val), (u32x4_t*)(y + (size_t)row * Nn + col));
      }
    }
  } else {
#pragma unroll
    for (int pass = 0; pass < PASSES; ++pass) {
      const int r = pass * RPS + rr;
      const int row = row0 + r;
      if (r >= NB * 32) break;
      union { uint4 u; T e[VEC]; } val;
      val.u = *(const uint4*)(lds + r * PIT + cc * 16);
      if (row < M) {
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
          const int cj = col + j;
          if (cj < Nn) {
            const size_t o = (size_t)row * Nn + cj;
            T e = val.e[j];
            if (mk && !(elem_f(mk[o]) > 0.f)) e = T(0);
            y[o] = e;
          }
        }
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
  uint32_t x_bytes, w_bytes;
  int M, Nn, Kg;
  int H, W, C, S, P, Q;
  int sh, sw, ph, pw;
  FastDiv dPQ, dQ, dC, dS;
  int relu;
  int tiles, tiles_n;
  float* partial;  // split-K: fp32 partial tiles [split][M][Nn] instead of y
  int kt_per_split;
  const void* mask;  // optional [M][Nn] tensor: an output is zeroed where mask <= 0
  // 256-row kernel: K-tile kt covers channels [cs BK, cs BK + BK) of tap
  // rs = kt mod RS, cs = kt div RS (taps fastest), instead of taps [kt BK,
  // kt BK + BK) in (r, s, c) order; needs C % BK == 0.
  int tap_major, RS;
  FastDiv dRS;
  // input patch (stride 1, tap-major): the padded input is Hp x Wp per image
  int patch, Hp, Wp;
  FastDiv dHp, dWp;
};

// Operand load modes.  VEC16: 16-byte vectors of VEC taps (C % VEC == 0 for
// the input, Kg % VEC == 0 for the filter rows).  VEC8 (bf16 only): two 8-byte
// halves of 4 taps each, for channel counts that are a multiple of 4 but not
// of 8 (the first layer's colour channels padded to 4).  ELEM: one element at
// a time.
// BT16 (bf16 filter only): the filter is given transposed, w[tap][col] with
// the Nn columns contiguous (Nn % 8 == 0); 16-byte vectors of 8 columns go
// into LDS as tap-major rows and the MFMA fragments come from transposing
// reads.  Serves the dense backward-data, whose B operand is the weight
// matrix as stored, without a transposed copy.
constexpr int ELEM = 0, VEC8 = 1, VEC16 = 2, BT16 = 3;


// AM / BMD: load mode of the input taps / filter rows.  BWD only names the
// instance that serves backward-data, so profiles tell them apart.
template <typename T, int AM, int BMD, bool BWD>
__global__ __launch_bounds__(NT) void conv_fwd_kernel(FwdArgs a) {
  constexpr int VEC = KT<T>::VEC;
  constexpr int BK = KT<T>::BK;
  constexpr uint32_t ES = sizeof(T);
  constexpr bool BT = BMD == BT16;
  static_assert(!BT || sizeof(T) == 2, "transposed filter: bf16 only");
  constexpr int BTILE = BT ? BT_TILE : TILE;  // bytes of the B tile
  __shared__ __attribute__((aligned(16))) char smem[BT ? BT_SMEM : SMEM];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  const int split = L / a.tiles, tile = L - split * a.tiles;
  const int tm = tile / a.tiles_n, tn = tile - tm * a.tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, a.x_bytes);
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(a.w, a.w_bytes);

  // Each thread fills one 16-byte column (cv) of 4 rows (rl + 32 i) of each operand.
  const int cv = tid & 7, rl = tid >> 3;
  int apix[4], ah0[4], aw0[4];  // element offset of input pixel (n, h0, w0); window origin
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + rl + 32 * i;
    if (m < a.M) {
      const int n = (int)fdiv((uint32_t)m, a.dPQ);
      const int pq = m - n * a.P * a.Q;
      const int p = (int)fdiv((uint32_t)pq, a.dQ);
      const int q = pq - p * a.Q;
      ah0[i] = p * a.sh - a.ph;
      aw0[i] = q * a.sw - a.pw;
      apix[i] = ((n * a.H + ah0[i]) * a.W + aw0[i]) * a.C;
    } else {
      ah0[i] = -(1 << 28);  // fails every bounds check
      aw0[i] = 0;
      apix[i] = 0;
    }
  }
  int brow[4];  // element offset of the filter row, or -1
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int n = n0 + rl + 32 * i;
    brow[i] = n < a.Nn ? n * a.Kg : -1;
  }

  auto load_tile = [&](int k0, V16 (&ra)[4], V16 (&rb)[4]) {
    const int kk = k0 + cv * VEC;
    if constexpr (AM == VEC16) {
      const bool kin = kk < a.Kg;
      const int rs = (int)fdiv((uint32_t)kk, a.dC);
      const int c = kk - rs * a.C;
      const int r = (int)fdiv((uint32_t)rs, a.dS);
      const int s = rs - r * a.S;
      const int tap = (r * a.W + s) * a.C + c;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int h = ah0[i] + r, w = aw0[i] + s;
        const bool ok = kin && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
        ra[i].u = ld16(xr, ok ? (uint32_t)(apix[i] + tap) * ES : OOB);
      }
    } else if constexpr (AM == VEC8) {
      // taps kk..kk+3 at (r0, s0, c0..c0+3), kk+4..kk+7 at (r1, s1, c1..c1+3)
      const int rs0 = (int)fdiv((uint32_t)kk, a.dC);
      const int c0 = kk - rs0 * a.C;
      const int r0 = (int)fdiv((uint32_t)rs0, a.dS);
      const int s0 = rs0 - r0 * a.S;
      const bool wrap = c0 + 4 >= a.C;
      const int c1 = wrap ? c0 + 4 - a.C : c0 + 4;
      const bool snext = wrap && s0 + 1 == a.S;
      const int s1 = wrap ? (snext ? 0 : s0 + 1) : s0;
      const int r1 = snext ? r0 + 1 : r0;
      const int tap0 = (r0 * a.W + s0) * a.C + c0, tap1 = (r1 * a.W + s1) * a.C + c1;
      const bool kin0 = kk < a.Kg, kin1 = kk + 4 < a.Kg;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int h0 = ah0[i] + r0, w0 = aw0[i] + s0, h1 = ah0[i] + r1, w1 = aw0[i] + s1;
        const bool ok0 = kin0 & ((unsigned)h0 < (unsigned)a.H) & ((unsigned)w0 < (unsigned)a.W);
        const bool ok1 = kin1 & ((unsigned)h1 < (unsigned)a.H) & ((unsigned)w1 < (unsigned)a.W);
        const uint2 lo = ld8(xr, ok0 ? (uint32_t)(apix[i] + tap0) * ES : OOB);
        const uint2 hi = ld8(xr, ok1 ? (uint32_t)(apix[i] + tap1) * ES : OOB);
        ra[i].u = make_uint4(lo.x, lo.y, hi.x, hi.y);
      }
    } else {
#pragma unroll
      for (int j = 0; j < VEC; ++j) {
        const int kj = kk + j;
        const bool kin = kj < a.Kg;
        const int rs = (int)fdiv((uint32_t)kj, a.dC);
        const int c = kj - rs * a.C;
        const int r = (int)fdiv((uint32_t)rs, a.dS);
        const int s = rs - r * a.S;
        const int tap = (r * a.W + s) * a.C + c;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int h = ah0[i] + r, w = aw0[i] + s;
          const bool ok = kin && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
          set_elem<T>(ra[i], j, ld_elem<T>(xr, ok ? (uint32_t)(apix[i] + tap) * ES : OOB));
        }
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if constexpr (BT) {
        // chunk tid + 256 i of the 64 x 128 tile: tap k0 + q / 16, columns n0 + 8 (q % 16) ..
        const int q = tid + 256 * i, kt = k0 + (q >> 4), col = n0 + 8 * (q & 15);
        const bool ok = kt < a.Kg && col < a.Nn;
        rb[i].u = ld16(wr, ok ? (uint32_t)(kt * a.Nn + col) * ES : OOB);
      } else if constexpr (BMD == VEC16) {
        const bool ok = brow[i] >= 0 && kk < a.Kg;
        rb[i].u = ld16(wr, ok ? (uint32_t)(brow[i] + kk) * ES : OOB);
      } else if constexpr (BMD == VEC8) {
        const bool ok0 = (brow[i] >= 0) & (kk < a.Kg), ok1 = (brow[i] >= 0) & (kk + 4 < a.Kg);
        const uint2 lo = ld8(wr, ok0 ? (uint32_t)(brow[i] + kk) * ES : OOB);
        const uint2 hi = ld8(wr, ok1 ? (uint32_t)(brow[i] + kk + 4) * ES : OOB);
        rb[i].u = make_uint4(lo.x, lo.y, hi.x, hi.y);
      } else {
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
          const bool ok = brow[i] >= 0 && kk + j < a.Kg;
          set_elem<T>(rb[i], j, ld_elem<T>(wr, ok ? (uint32_t)(brow[i] + kk + j) * ES : OOB));
        }
      }
    }
  };
  auto store_tile = [&](int stage, const V16 (&ra)[4], const V16 (&rb)[4]) {
    char* As = smem + stage * (TILE + BTILE);
    char* Bs = As + TILE;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *(uint4*)(As + (rl + 32 * i) * PITCH + cv * 16) = ra[i].u;
      if constexpr (BT) {
        const int q = tid + 256 * i;
        *(uint4*)(Bs + (q >> 4) * BT_PITCH + (q & 15) * 16) = rb[i].u;
      } else {
        *(uint4*)(Bs + (rl + 32 * i) * PITCH + cv * 16) = rb[i].u;
      }
    }
  };


  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  // Two LDS stages and two register sets: the global loads of tile k+2 are in
  // flight while tile k is multiplied and tile k+1 goes from registers to LDS.
  const int wm = wave >> 1, wn = wave & 1;
  auto mma = [&](const char* S) {
    if constexpr (BT) mma_tile_bt(S, S + TILE, acc, wm, wn, lane);
    else mma_tile<T>(S, S + TILE, acc, wm, wn, lane);
  };
  const int nkt_all = (a.Kg + BK - 1) / BK;
  const int kbase = split * a.kt_per_split * BK;                   // first tap of this split
  const int nkt = min(a.kt_per_split, nkt_all - split * a.kt_per_split);  // K-tiles of this split (>= 1)
  V16 a0[4], b0[4], a1[4], b1[4];
  load_tile(kbase, a0, b0);
  if (nkt > 1) load_tile(kbase + BK, a1, b1);
  store_tile(0, a0, b0);
  __syncthreads();
  int kt = 0;
  for (; kt + 1 < nkt; kt += 2) {  // tiles kt (stage 0) and kt + 1 (stage 1)
    if (kt + 2 < nkt) load_tile(kbase + (kt + 2) * BK, a0, b0);
    mma(smem);
    store_tile(1, a1, b1);
    __syncthreads();
    if (kt + 3 < nkt) load_tile(kbase + (kt + 3) * BK, a1, b1);
    mma(smem + TILE + BTILE);
    if (kt + 2 < nkt) store_tile(0, a0, b0);
    __syncthreads();
  }
  if (kt < nkt) mma(smem);  // odd count: last tile is in stage 0

  // Epilogue: lane holds column li of each 32x32 block, rows 8*(v/4) + 4*lh + v%4.
  const int li = lane & 31, lh = lane >> 5;
  if (a.partial) {
    float* __restrict__ out = a.partial + (size_t)split * a.M * a.Nn;
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
    return;
  }
  __syncthreads();  // every wave is done with the operand tiles
  const bool vec = a.Nn % VEC == 0 && (((uintptr_t)a.y | (uintptr_t)a.mask) % 16) == 0;
  store_quadrant<T, 2, 2>(acc, smem + wave * 64 * (64 * (int)sizeof(T) + 16), lane, m0 + wm * 64, n0 + wn * 64, a.M,
                       a.Nn, a.bias, a.relu, a.mask, (T*)a.y, vec);
}

// ------------------------------------------------- forward, large bf16 tiles
//
// The same implicit GEMM for bf16 operands whose taps and filter rows are
// whole 16-byte vectors (C % 8 == 0), with a 256 x 128 output tile: each of
// the 4 waves owns a 128 x 64 quadrant (4 x 2 blocks of 32 x 32), so one
// 16-byte fragment read feeds more MFMAs than in the 128 x 128 kernel.
// Global data goes straight from the buffer loads into LDS (each load
// instruction writes 64 consecutive 16-byte slots) with no register staging.
// Three LDS stages: the loads of K-tile k+2 are in flight while tile k is
// multiplied; one barrier per K-tile.  LBK taps per K-tile: 64 (144 KB of
// LDS, one workgroup per CU) or 32 (72 KB, two workgroups per CU; the
// 256 x 96 layout keeps two stages, 48 KB, three workgroups per CU).
//
// LDS rows (LBK * 2 bytes) are unpadded and XOR-swizzled: slot s of row r
// holds the 16-byte tap chunk s ^ ((r / RPW) % SL), with SL slots per row and
// RPW rows per 256-byte bank window, so a fragment read (16 lanes, 16
// consecutive rows, one chunk) touches 16 distinct 16-byte bank groups.
constexpr int L_BM = 256;
// input-patch entries (64 bytes: 32 channels of one padded input pixel) per
// buffer: with 3 filter stages of 8 KB and 2 x 28 KB of patch the 256 x 128
// layout keeps two workgroups per CU
constexpr int FWD_PATCH_ENTRIES = 448;
constexpr int L_STAGES = 3;
template <int LBK> struct LT {
  static constexpr int RB = LBK * 2;                  // row bytes
  static constexpr int SL = RB / 16;                  // 16-byte slots per row
  static constexpr int RPI = 64 / SL;                 // rows per load instruction
  static constexpr int RPW = 256 / RB;                // rows per 256-byte bank window
  static constexpr int ATILE = L_BM * RB, BTILE = BN * RB, STAGE = ATILE + BTILE;
  static constexpr int SMEM = L_STAGES * STAGE;
  static constexpr int AI = L_BM / RPI / 4, BI = BN / RPI / 4;  // load instructions per wave
  static constexpr int KS = LBK / 16;                 // MFMA k-steps per K-tile
};

typedef __attribute__((address_space(3))) void* lds_ptr;

// One 16-byte buffer load per lane into LDS slot (base + 16 * lane); base is
// wave-uniform.
__device__ __forceinline__ void ld_lds16(__amdgpu_buffer_rsrc_t r, uint32_t off, char* base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr)base, 16, off, 0, 0, 0);
}

// The same load issued from inline assembly.  The compiler then does not
// know that the instruction writes LDS, so it adds no vmcnt wait in front of
// later LDS reads (it does so for the transpose reads, which would serialize
// every prefetch); the kernel orders the two itself with wait_vmcnt and a
// barrier.  M0 carries the LDS address; no other code of these kernels uses
// M0.
__device__ __forceinline__ void ld_lds16_asm(__amdgpu_buffer_rsrc_t r, uint32_t off, char* base) {
  const uint32_t lds = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)base;
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" ::"s"(__builtin_amdgcn_readfirstlane(lds)),
               "v"(off), "s"(r)
               : "memory");
}

// s_waitcnt vmcnt(n) (n < 64), leaving the other counters alone.
template <int N> __device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__device__ __forceinline__ void block_barrier() { asm volatile("s_barrier" ::: "memory"); }

// WMW = 2: waves 2 (rows) x 2 (columns), each 128 x 64 of a 256 x 128 tile.
// WMW = 4: waves stacked along the rows, each 64 x 96 of a 256 x 96 tile, for
// layers with at most 96 output channels (the B tile still loads 128 rows,
// the last 32 out of range: no memory traffic).
// WMW = 8: 8 waves, 2 (rows) x 4 (columns), each 128 x 64 of a 256 x 256
// tile (512 threads, one workgroup per CU): half the operand bytes per flop
// of the 256 x 128 tile on the B side, for 256-column layers with enough
// row tiles.
// WMW = 6: the same 8 waves on a 192 x 256 tile, each 96 x 64: 4/3 as many
// tiles, for layers whose 256-row tiles leave much of the chip idle in their
// last round (AlexNet's 13 x 13 layers at batch 256: 169 tiles of 256 rows
// on 256 CUs, 226 of 192).  Loads and LDS are those of WMW = 8; the A rows
// 192 .. 255 of each stage are loaded as out-of-range zeros (no traffic)
// and never read.
template <bool BWD, int LBK, int WMW, bool PATCH>
__global__ __launch_bounds__(WMW >= 6 ? 2 * NT : NT, (LBK == 32 && WMW == 4) ? 3 : (LBK == 32 && WMW < 6) ? 2 : 1)
void conv_fwd_large_kernel(FwdArgs a) {
  typedef LT<LBK> G;
  static_assert(WMW == 2 || WMW == 4 || WMW == 6 || WMW == 8, "wave layouts");
  constexpr int NW = WMW >= 6 ? 8 : 4;       // waves
  constexpr int BNT = WMW >= 6 ? 256 : BN;   // tile columns
  constexpr int BMT = WMW == 6 ? 192 : L_BM;  // tile rows (the A stage keeps L_BM rows)
  constexpr int FM = WMW == 4 ? 2 : WMW == 6 ? 3 : 4, FN = WMW == 4 ? 3 : 2;
  constexpr int ABAND = L_BM / NW, BBAND = BNT / NW;  // operand rows each wave loads
  constexpr int AI = ABAND / G::RPI, BI = BBAND / G::RPI;  // its load instructions per K-tile
  // with the input patch the stages hold only the filter tile
  constexpr int ATILE = PATCH ? 0 : L_BM * G::RB, STAGE = ATILE + BNT * G::RB;
  constexpr int LOADS = (PATCH ? 0 : AI) + BI;  // 16-byte loads per thread per K-tile
  static_assert(AI * G::RPI == ABAND && BI * G::RPI == BBAND, "load bands");
  // LDS stages: K-tiles kt+1 .. kt+NS-1 are in flight while kt is multiplied.
  // The 256 x 96 layout keeps two (48 KB, three workgroups per CU): measured
  // 5 % faster on conv2's backward-data than three stages at two per CU.
  constexpr int NS = (WMW == 4 && LBK == 32) ? 2 : L_STAGES;
  // input patch: two buffers of PENT 64-byte entries (32 channels of one
  // padded input pixel), PL loads per thread per channel slice
  static_assert(!PATCH || (LBK == 32 && WMW == 2), "the patch serves 32-tap K-tiles of the 256 x 128 layout");
  constexpr int PENT = PATCH ? FWD_PATCH_ENTRIES : 0;
  constexpr int PBUF = PENT * 64, PL = PENT / (NW * 16);
  static_assert(!PATCH || PL * NW * 16 == PENT, "patch loads");
  __shared__ __attribute__((aligned(16))) char smem[NS * STAGE + 2 * PBUF];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  const int split = L / a.tiles, tile = L - split * a.tiles;
  const int tm = tile / a.tiles_n, tn = tile - tm * a.tiles_n;
  const int m0 = tm * BMT, n0 = tn * BNT;
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, a.x_bytes);
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(a.w, a.w_bytes);

  // Loader: instruction i of this wave fills rows RPI i .. RPI i + RPI - 1 of
  // the wave's A (64 rows) / B (32 rows) band; this lane owns row RPI i +
  // lane / SL, slot lane % SL, which holds chunk cpar[p] with p the parity of
  // i for 128-byte rows (always 0 for 64-byte rows).
  const int lrow = lane / G::SL;
  int cpar[2];
#pragma unroll
  for (int p = 0; p < 2; ++p) cpar[p] = (lane % G::SL) ^ ((4 * p * (G::SL == 8) + (lane >> 4)) % G::SL);
  constexpr int NPAR = G::SL == 8 ? 2 : 1;
  int apix[AI], ah0[AI], aw0[AI];
#pragma unroll
  for (int i = 0; i < AI; ++i) {
    const int m = m0 + ABAND * wave + G::RPI * i + lrow;
    if (m < a.M && ABAND * wave + G::RPI * i + lrow < BMT) {
      const int n = (int)fdiv((uint32_t)m, a.dPQ);
      const int pq = m - n * a.P * a.Q;
      const int p = (int)fdiv((uint32_t)pq, a.dQ);
      const int q = pq - p * a.Q;
      ah0[i] = p * a.sh - a.ph;
      aw0[i] = q * a.sw - a.pw;
      apix[i] = ((n * a.H + ah0[i]) * a.W + aw0[i]) * a.C;
    } else {
      ah0[i] = -(1 << 28);
      aw0[i] = 0;
      apix[i] = 0;
    }
  }
  int brow[BI];
#pragma unroll
  for (int i = 0; i < BI; ++i) {
    const int n = n0 + BBAND * wave + G::RPI * i + lrow;
    brow[i] = n < a.Nn ? n * a.Kg : -1;
  }

  // Tap decomposition of this lane's chunk(s) of the K-tile at k0; a K-tile
  // past the end gives OOB everywhere.
  struct Taps {
    int tap[2], r[2], s[2];
    bool kin[2];
    int kk[2];
  };
  auto taps = [&](int k0) {
    Taps t;
    if (a.tap_major && k0 < a.Kg) {
      // consecutive K-tiles read the same channels one tap apart: the input
      // rows they need overlap, so they meet in the caches
      const int kt = k0 / LBK;
      const int cs = (int)fdiv((uint32_t)kt, a.dRS);
      k0 = (kt - cs * a.RS) * a.C + cs * LBK;
    }
#pragma unroll
    for (int p = 0; p < NPAR; ++p) {
      const int kk = k0 + 8 * cpar[p];
      t.kk[p] = kk;
      t.kin[p] = kk < a.Kg;
      const int rs = (int)fdiv((uint32_t)kk, a.dC);
      const int c = kk - rs * a.C;
      t.r[p] = (int)fdiv((uint32_t)rs, a.dS);
      t.s[p] = rs - t.r[p] * a.S;
      t.tap[p] = (t.r[p] * a.W + t.s[p]) * a.C + c;
    }
    return t;
  };
  auto issue_a = [&](const Taps& t, char* As, int i) {
    const int p = NPAR == 2 ? (i & 1) : 0;
    const int h = ah0[i] + t.r[p], w = aw0[i] + t.s[p];
    const bool ok = t.kin[p] & ((unsigned)h < (unsigned)a.H) & ((unsigned)w < (unsigned)a.W);
    ld_lds16(xr, ok ? (uint32_t)(apix[i] + t.tap[p]) * 2u : OOB, As + (ABAND * wave + G::RPI * i) * G::RB);
  };
  auto issue_b = [&](const Taps& t, char* Bs, int i) {
    const int p = NPAR == 2 ? (i & 1) : 0;
    const bool ok = (brow[i] >= 0) & t.kin[p];
    ld_lds16(wr, ok ? (uint32_t)(brow[i] + t.kk[p]) * 2u : OOB, Bs + (BBAND * wave + G::RPI * i) * G::RB);
  };
  // the j-th of KS slices of the K-tile's loads (spread over its k-steps)
  auto issue_slice = [&](const Taps& t, char* St, int j) {
    constexpr int TOT = AI + BI;
#pragma unroll
    for (int q = 0; q < TOT; ++q) {
      if (q * G::KS / TOT != j) continue;
      if (q < AI) issue_a(t, St, q);
      else issue_b(t, St + ATILE, q - AI);
    }
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int wm = WMW == 2 ? wave >> 1 : WMW >= 6 ? wave >> 2 : wave;
  const int wn = WMW == 2 ? wave & 1 : WMW >= 6 ? wave & 3 : 0;
  const int li = lane & 31, lh = lane >> 5;
  // chunk 2 kc + lh of row r sits in slot (2 kc + lh) ^ ((r / RPW) % SL); r % 16 = li % 16
  const int tsw = (lh ^ ((li / G::RPW) % G::SL)) << 4;
  const int aoff = (wm * FM * 32 + li) * G::RB, boff = ATILE + (wn * FN * 32 + li) * G::RB;
  struct Frags {
    bf16x8 a[FM], b[FN];
  };
  auto frags = [&](const char* S, int kc) {
    Frags f;
    const int co = (32 * kc) ^ tsw;
#pragma unroll
    for (int b = 0; b < FM; ++b) f.a[b] = *(const bf16x8*)(S + aoff + b * 32 * G::RB + co);
#pragma unroll
    for (int b = 0; b < FN; ++b) f.b[b] = *(const bf16x8*)(S + boff + b * 32 * G::RB + co);
    return f;
  };
  auto mma = [&](const Frags& f) {
#pragma unroll
    for (int bm = 0; bm < FM; ++bm)
#pragma unroll
      for (int bn = 0; bn < FN; ++bn)
        acc[bm][bn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[bm], f.b[bn], acc[bm][bn], 0, 0, 0);
  };

  const int nkt_all = (a.Kg + LBK - 1) / LBK;
  const int kbase = split * a.kt_per_split * LBK;
  const int nkt = min(a.kt_per_split, nkt_all - split * a.kt_per_split);
  const int kend = kbase + nkt * LBK;  // K-tiles from here on are issued as all-OOB (zeros, no traffic)
  if constexpr (PATCH) {
    // Input patch (stride 1, tap-major K-tiles, one split).  Every tap (r, s)
    // of a channel slice reads the same input pixels shifted by r rows and s
    // columns, so the tile's input rows for all taps are loaded once per
    // slice: padded rows g = n Hp + h + ph from the first output line of the
    // tile to R - 1 past its last, each Wp padded columns wide (zeros outside
    // the input), 32 channels per entry, swizzled like the operand rows
    // (chunk c of entry e in slot c ^ ((e / 4) % 4)).  Output row (n, p, q)
    // reads tap (r, s) at entry ((n Hp + p - g0) Wp + q) + r Wp + s.  The host
    // checks that a tile's patch fits PENT entries.  The next slice's patch
    // loads go out at its predecessor's first tap, into the other buffer.
    char* const pbuf0 = smem + NS * STAGE;
    const int R = a.RS / a.S;
    const int mlast = min(m0 + L_BM, a.M) - 1;
    auto line = [&](int m, int& n, int& p, int& q) {
      n = (int)fdiv((uint32_t)m, a.dPQ);
      const int pq = m - n * a.P * a.Q;
      p = (int)fdiv((uint32_t)pq, a.dQ);
      q = pq - p * a.Q;
    };
    int nf, pf, qf, nl, pl, ql;
    line(m0, nf, pf, qf);
    line(mlast, nl, pl, ql);
    const int g0 = nf * a.Hp + pf;
    const int E = (nl * a.Hp + pl + R - g0) * a.Wp;  // entries in use (<= PENT)
    uint32_t goff[PL];
#pragma unroll
    for (int i = 0; i < PL; ++i) {
      const int e = (i * NW + wave) * 16 + (lane >> 2);
      const int c = (lane & 3) ^ ((e >> 2) & 3);
      goff[i] = OOB;
      if (e < E) {
        const int gr = (int)fdiv((uint32_t)e, a.dWp);
        const int col = e - gr * a.Wp;
        const int g = g0 + gr;
        const int n = (int)fdiv((uint32_t)g, a.dHp);
        const int ih = g - n * a.Hp - a.ph, iw = col - a.pw;
        if ((unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W)
          goff[i] = (uint32_t)(((n * a.H + ih) * a.W + iw) * a.C + 8 * c) * 2u;
      }
    }
    const int nslices = a.C / LBK;
    auto issue_patch = [&](int cs, char* buf) {
#pragma unroll
      for (int i = 0; i < PL; ++i)
        ld_lds16(xr, (goff[i] != OOB && cs < nslices) ? goff[i] + (uint32_t)(cs * LBK * 2) : OOB,
                 buf + (i * NW + wave) * 1024);
    };
    int bpos[FM];
#pragma unroll
    for (int b = 0; b < FM; ++b) {
      const int mr = m0 + wm * FM * 32 + b * 32 + (lane & 31);
      int n, p, q;
      line(mr <= mlast ? mr : m0, n, p, q);
      bpos[b] = (n * a.Hp + p - g0) * a.Wp + q;
    }
    // B slices of a K-tile: the filter rows only
    auto issue_b_slice = [&](const Taps& t, char* St, int j) {
#pragma unroll
      for (int q = 0; q < BI; ++q)
        if (q * G::KS / BI == j) issue_b(t, St, q);
    };
    issue_patch(0, pbuf0);
#pragma unroll
    for (int s = 0; s < NS - 1; ++s)
#pragma unroll
      for (int j = 0; j < G::KS; ++j) issue_b_slice(taps(nkt > s ? kbase + s * LBK : a.Kg), smem + s * STAGE, j);
    int stage = 0;
    for (int kt = 0; kt < nkt; ++kt) {
      const int cs = (int)fdiv((uint32_t)kt, a.dRS);
      const int rs = kt - cs * a.RS;
      // An iteration issues the next slice's patch (at a slice's first tap)
      // and then the B loads of tile kt + NS - 1.  B(kt) has landed for this
      // thread once only the loads issued after it may be in flight: the B
      // tiles kt + 1 .. kt + NS - 2 and, when iteration kt - 1 was a slice's
      // first tap, the patch loads it issued (before B(kt + 1), after B(kt)).
      // The patch of slice cs went out before B(kt), so it has landed too.
      static_assert(NS == 3, "the wait below counts the loads of three stages");
      const bool extra = kt >= 1 && (kt - 1) % a.RS == 0;
      if (extra) wait_vmcnt<(NS - 2) * LOADS + PL>();
      else wait_vmcnt<(NS - 2) * LOADS>();
      block_barrier();  // ... and for everyone; everyone is done with tile kt-1 and, at rs == 0, with slice cs-1
      const int nstage = stage == 0 ? NS - 1 : stage - 1;
      const int knext = kbase + (kt + NS - 1) * LBK;
      const Taps t = taps(knext < kend ? knext : a.Kg);
      if (rs == 0) issue_patch(cs + 1, pbuf0 + ((cs + 1) & 1) * PBUF);
      const char* S = smem + stage * STAGE;
      const char* Pb = pbuf0 + (cs & 1) * PBUF;
      const int r = (int)fdiv((uint32_t)rs, a.dS);
      const int toff = r * a.Wp + (rs - r * a.S);
#pragma unroll
      for (int kc = 0; kc < G::KS; ++kc) {
        bf16x8 fa[FM], fb[FN];
#pragma unroll
        for (int b = 0; b < FM; ++b) {
          const int pos = bpos[b] + toff;
          fa[b] = *(const bf16x8*)(Pb + pos * 64 + ((((2 * kc + lh) ^ ((pos >> 2) & 3))) << 4));
        }
#pragma unroll
        for (int b = 0; b < FN; ++b) fb[b] = *(const bf16x8*)(S + boff + b * 32 * G::RB + ((32 * kc) ^ tsw));
#pragma unroll
        for (int bm = 0; bm < FM; ++bm)
#pragma unroll
          for (int bn = 0; bn < FN; ++bn)
            acc[bm][bn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[bm], fb[bn], acc[bm][bn], 0, 0, 0);
        issue_b_slice(t, smem + nstage * STAGE, kc);
      }
      stage = stage == NS - 1 ? 0 : stage + 1;
    }
  } else {
#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
#pragma unroll
    for (int j = 0; j < G::KS; ++j) issue_slice(taps(nkt > s ? kbase + s * LBK : a.Kg), smem + s * STAGE, j);
  int stage = 0;
  for (int kt = 0; kt < nkt; ++kt) {
    wait_vmcnt<(NS - 2) * LOADS>();  // this thread's loads of tile kt have landed (later tiles' may be in flight)
    block_barrier();                 // ... and everyone's; everyone is also done with tile kt-1
    const int nstage = stage == 0 ? NS - 1 : stage - 1;
    char* Ns = smem + nstage * STAGE;
    const int knext = kbase + (kt + NS - 1) * LBK;
    const Taps t = taps(knext < kend ? knext : a.Kg);
    const char* S = smem + stage * STAGE;
    // fragments one k-step ahead; the loads of tile kt+2 spread over the k-steps
    Frags f = frags(S, 0);
#pragma unroll
    for (int kc = 0; kc < G::KS; ++kc) {
      Frags g;
      if (kc + 1 < G::KS) g = frags(S, kc + 1);
      mma(f);
      issue_slice(t, Ns, kc);
      if (kc + 1 < G::KS) f = g;
    }
    stage = stage == NS - 1 ? 0 : stage + 1;
  }
  }
  wait_vmcnt<0>();  // the trailing all-OOB loads still write LDS

  if (a.partial) {
    float* __restrict__ out = a.partial + (size_t)split * a.M * a.Nn;
#pragma unroll
    for (int bn = 0; bn < FN; ++bn) {
      const int col = n0 + wn * FN * 32 + bn * 32 + li;
      if (col >= a.Nn) continue;
#pragma unroll
      for (int bm = 0; bm < FM; ++bm)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int row = m0 + wm * FM * 32 + bm * 32 + (v >> 2) * 8 + lh * 4 + (v & 3);
          if (row < a.M) out[(size_t)row * a.Nn + col] = acc[bm][bn][v];
        }
    }
    return;
  }
  __syncthreads();  // every wave is done with the operand tiles
  const bool vec = a.Nn % 8 == 0 && (((uintptr_t)a.y | (uintptr_t)a.mask) % 16) == 0;
  if constexpr (WMW >= 6) {
    // the quadrant in passes of 64 rows (and 32 for the 96-row one): 8 waves
    // x 9 KB of staging
    char* q = smem + wave * 64 * (FN * 32 * 2 + 16);
    store_quadrant<bf16_t, FM, FN, 0, 2>(acc, q, lane, m0 + wm * FM * 32, n0 + wn * FN * 32, a.M, a.Nn, a.bias,
                                         a.relu, a.mask, (bf16_t*)a.y, vec);
    store_quadrant<bf16_t, FM, FN, 2, FM - 2>(acc, q, lane, m0 + wm * FM * 32 + 64, n0 + wn * FN * 32, a.M, a.Nn,
                                              a.bias, a.relu, a.mask, (bf16_t*)a.y, vec);
  } else if constexpr (NS == 2) {
    // two LDS stages hold less than the quadrant: two passes of 32 rows
    char* q = smem + wave * 32 * (FN * 32 * 2 + 16);
    store_quadrant<bf16_t, FM, FN, 0, 1>(acc, q, lane, m0 + wm * FM * 32, n0 + wn * FN * 32, a.M, a.Nn, a.bias,
                                         a.relu, a.mask, (bf16_t*)a.y, vec);
    store_quadrant<bf16_t, FM, FN, 1, 1>(acc, q, lane, m0 + wm * FM * 32 + 32, n0 + wn * FN * 32, a.M, a.Nn,
                                         a.bias, a.relu, a.mask, (bf16_t*)a.y, vec);
  } else {
    store_quadrant<bf16_t, FM, FN>(acc, smem + wave * FM * 32 * (FN * 32 * 2 + 16), lane, m0 + wm * FM * 32,
                                   n0 + wn * FN * 32, a.M, a.Nn, a.bias, a.relu, a.mask, (bf16_t*)a.y, vec);
  }
}

// ----------------------------------------------------------- filter gradient
//
// dW[i][j] = sum_t dy[t][i] * x^[t][j], i = filter, j = tap (r, s, c),
// t = output pixel of one image.  The order of the reduction is free.  NFAST
// runs t over (p, q) with the image n fastest, t = (p*Q + q)*N + n: when N is
// a multiple of the K-tile, all rows of a K-tile share one output pixel
// (p, q), so the bounds check of a tap is the same for every row and a row's
// address is n times the image stride.  Otherwise t is image-major,
// t = n*P*Q + p*Q + q, which keeps a workgroup's input reads inside one image
// (better L2 reuse when an image has many output pixels).  Both operand tiles sit in LDS exactly as loaded,
// t-major rows of 128 consecutive filters / taps.  For bf16 the MFMA fragment
// (8 consecutive t of one filter or tap) comes from ds_read_b64_tr_b16, which
// hands each lane of a 16-lane group one column of the 4 rows the group
// addresses; for fp32 (v_mfma_f32_32x32x2_f32) a lane needs a single value and
// reads it directly.


template <typename T> struct WG;
template <> struct WG<bf16_t> {
  static constexpr int BK = 64;     // t per K-tile
  static constexpr int PITCH = 320;  // 256 B row + 64 B: a tr-read group's 4 rows hit disjoint banks
};
template <> struct WG<float> {
  static constexpr int BK = 32;
  static constexpr int PITCH = 640;  // 512 B row + 128 B: the 2 rows of a fragment read hit disjoint banks
};
constexpr int WSMEM = 2 * 2 * 64 * 320;  // 2 stages x 2 operands (equal for both dtypes)

// With a bias, the GEMM gets one more column, Ng = Nn + 1, whose operand is
// 1 for every reduction index: its results are db[k] = sum_t dy[t][k].
struct WgradArgs {
  const void* x;
  const void* dy;
  float* out;  // partial tiles [splits][M][Ng], or dw itself when direct
  float* db;   // direct: the bias gradient (column Nn); NULL without bias
  uint32_t x_bytes, dy_bytes;
  int M, Nn, Ng, T;  // M = K filters, Nn = R*S*C taps, Ng = Nn (+1 with bias), T = N*P*Q
  int ldp;           // row stride of the partial tiles: Ng rounded up to 64 (256-byte rows)
  int N, H, W, C, S, P, Q;
  int sh, sw, ph, pw;
  FastDiv dN, dPQ, dQ, dC, dS;
  int tiles, tiles_n, kt_per_split, nkt;
  int direct, acc_dw, acc_db;
  int update;    // direct only: each element is applied to `u` (out / db: NULL, or where g is also stored)
  SgdTargets u;
};


// One K-tile of t-major operand rows: acc[bm][bn] += A(rows) * B(cols)^T.
template <typename T>
__device__ __forceinline__ void mma_tile_tmajor(const char* As, const char* Bs, f32x16 (&acc)[2][2], int wm, int wn,
                                                int lane) {
  constexpr int BK = WG<T>::BK, PIT = WG<T>::PITCH;
  if constexpr (sizeof(T) == 2) {
    // lane l: column (l & 15) of a 16-column group, t rows 8*(l >> 5) + 0..7 of the 16-t step
    const int g = lane >> 4, s = lane & 15;
    const int row = 8 * (g >> 1) + (s >> 2);
    const int colb = 2 * (16 * (g & 1) + 4 * (s & 3));  // byte offset within a 32-column block
    const char* ab = As + row * PIT + 2 * (wm * 64) + colb;
    const char* bb = Bs + row * PIT + 2 * (wn * 64) + colb;
#pragma unroll
    for (int kc = 0; kc < BK / 16; ++kc) {
      bf16x8 af[2], bfr[2];
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const v4i16 alo = lds_tr16(ab + kc * 16 * PIT + b * 64);
        const v4i16 ahi = lds_tr16(ab + (kc * 16 + 4) * PIT + b * 64);
        const v4i16 blo = lds_tr16(bb + kc * 16 * PIT + b * 64);
        const v4i16 bhi = lds_tr16(bb + (kc * 16 + 4) * PIT + b * 64);
        af[b] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(alo, ahi, 0, 1, 2, 3, 4, 5, 6, 7));
        bfr[b] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(blo, bhi, 0, 1, 2, 3, 4, 5, 6, 7));
      }
      acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[0], bfr[0], acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[0], bfr[1], acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[1], bfr[0], acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[1], bfr[1], acc[1][1], 0, 0, 0);
    }
  } else {
    // lane l: column (l & 31) of a 32-column block, t row (l >> 5) of the 2-t step
    const int li = lane & 31, lh = lane >> 5;
    const char* ab = As + lh * PIT + 4 * (wm * 64 + li);
    const char* bb = Bs + lh * PIT + 4 * (wn * 64 + li);
#pragma unroll
    for (int kc = 0; kc < BK / 2; ++kc) {
      const float a0 = *(const float*)(ab + 2 * kc * PIT);
      const float a1 = *(const float*)(ab + 2 * kc * PIT + 128);
      const float b0 = *(const float*)(bb + 2 * kc * PIT);
      const float b1 = *(const float*)(bb + 2 * kc * PIT + 128);
      acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b0, acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b1, acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b1, acc[1][1], 0, 0, 0);
    }
  }
}

// VA: the 16-byte filter chunks of dy are whole vectors (M % VEC == 0),
// otherwise element loads.  BMD: load mode of the tap chunks of x (VEC16 for
// C % VEC == 0, VEC8 for bf16 with C % 4 == 0, else ELEM).
// NFAST: N % BK == 0, so a K-tile's rows share one output pixel.
template <typename T, bool VA, int BMD, bool NFAST>
__global__ __launch_bounds__(NT) void conv_wgrad_kernel(WgradArgs a) {
  constexpr int VEC = 16 / (int)sizeof(T);
  constexpr int CH = 128 / VEC;  // 16-byte chunks per tile row
  constexpr int RPP = NT / CH;   // rows covered by one pass of the 256 threads
  constexpr int BK = WG<T>::BK;
  constexpr int PIT = WG<T>::PITCH;
  constexpr int OPB = BK * PIT;  // bytes of one operand tile
  constexpr uint32_t ES = sizeof(T);
  static_assert(BK == 4 * RPP, "four passes fill a K-tile");
  static_assert(2 * 2 * OPB == WSMEM, "LDS budget");
  __shared__ __attribute__((aligned(16))) char smem[WSMEM];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  const int split = L / a.tiles, tile = L - split * a.tiles;
  const int tm = tile / a.tiles_n, tn = tile - tm * a.tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  const int kt_begin = split * a.kt_per_split;
  const int nk = min(a.nkt, kt_begin + a.kt_per_split) - kt_begin;
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, a.x_bytes);
  const __amdgpu_buffer_rsrc_t dyr = make_rsrc(a.dy, a.dy_bytes);

  const int ch = tid % CH, r0 = tid / CH;  // this thread's chunk column and first row
  const int i0 = m0 + ch * VEC;            // first filter of its dy chunk
  const int j0 = n0 + ch * VEC;            // first tap of its x chunk
  const int PQ = a.P * a.Q;
  const int ystride = PQ * a.M;            // dy elements per image
  const int xstride = a.H * a.W * a.C;     // x elements per image
  // position of the bias column Nn in this thread's chunk, or -1, and the
  // chunk with a 1 there (static indexing: no register array in scratch)
  const int ones = (a.Ng > a.Nn && j0 <= a.Nn && a.Nn < j0 + VEC) ? a.Nn - j0 : -1;
  V16 onesv;
#pragma unroll
  for (int e = 0; e < VEC; ++e) set_elem<T>(onesv, e, e == ones ? one_elem<T>() : zero_elem<T>());
  // taps of the x chunk, fixed for the whole reduction: NG groups of GS
  // consecutive channels of one tap (r, s) each
  constexpr int NG = BMD == VEC16 ? 1 : BMD == VEC8 ? 2 : VEC;
  constexpr int GS = VEC / NG;
  int br[NG], bs[NG], btap[NG];
  bool bok[NG];
#pragma unroll
  for (int e = 0; e < NG; ++e) {
    const int j = j0 + e * GS;
    bok[e] = j < a.Nn;
    const int jj = bok[e] ? j : 0;
    const int rs = (int)fdiv((uint32_t)jj, a.dC);
    const int c = jj - rs * a.C;
    br[e] = (int)fdiv((uint32_t)rs, a.dS);
    bs[e] = rs - br[e] * a.S;
    btap[e] = (br[e] * a.W + bs[e]) * a.C + c;
  }

  // Row d of the K-tile starting at t0: dy offset and x pixel (n, hb, wb).
  auto load_tile = [&](int kt, V16 (&ra)[4], V16 (&rb)[4]) {
    const int t0 = kt * BK;
    int pq = 0, nb = 0, hb = 0, wb = 0;
    if constexpr (NFAST) {
      pq = (int)fdiv((uint32_t)t0, a.dN);
      nb = t0 - pq * a.N;
      const int p = (int)fdiv((uint32_t)pq, a.dQ);
      hb = p * a.sh - a.ph;
      wb = (pq - p * a.Q) * a.sw - a.pw;
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int d = r0 + RPP * v;
      int n, rpq, h0, w0;
      bool tin;
      if constexpr (NFAST) {
        n = nb + d;
        rpq = pq;
        h0 = hb;
        w0 = wb;
        tin = true;  // T is a multiple of BK
      } else {  // image-major order: t = n P Q + p Q + q
        const int t = t0 + d;
        tin = t < a.T;
        n = (int)fdiv((uint32_t)t, a.dPQ);
        rpq = t - n * PQ;
        const int p = (int)fdiv((uint32_t)rpq, a.dQ);
        h0 = p * a.sh - a.ph;
        w0 = (rpq - p * a.Q) * a.sw - a.pw;
      }
      // A: dy[n][p][q][i0 .. i0 + VEC)
      const int aoff = n * ystride + rpq * a.M + i0;
      if constexpr (VA) {
        ra[v].u = ld16(dyr, (tin && i0 < a.M) ? (uint32_t)aoff * ES : OOB);
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e)
          set_elem<T>(ra[v], e, ld_elem<T>(dyr, (tin && i0 + e < a.M) ? (uint32_t)(aoff + e) * ES : OOB));
      }
      // B: x[n][h0 + r][w0 + s][c .. c + VEC)
      const int xpix = n * xstride + (h0 * a.W + w0) * a.C;
      if constexpr (BMD == VEC16) {
        const int h = h0 + br[0], w = w0 + bs[0];
        const bool ok = tin && bok[0] && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
        rb[v].u = ld16(xr, ok ? (uint32_t)(xpix + btap[0]) * ES : OOB);
      } else if constexpr (BMD == VEC8) {
        uint2 half[2];
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const int h = h0 + br[e], w = w0 + bs[e];
          const bool ok = tin & bok[e] & ((unsigned)h < (unsigned)a.H) & ((unsigned)w < (unsigned)a.W);
          half[e] = ld8(xr, ok ? (uint32_t)(xpix + btap[e]) * ES : OOB);
        }
        rb[v].u = make_uint4(half[0].x, half[0].y, half[1].x, half[1].y);
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const int h = h0 + br[e], w = w0 + bs[e];
          const bool ok = tin && bok[e] && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
          set_elem<T>(rb[v], e, ld_elem<T>(xr, ok ? (uint32_t)(xpix + btap[e]) * ES : OOB));
        }
      }
    }
  };
  // The bias column is OR-ed in as the tile goes to LDS (its element was
  // loaded as an out-of-range zero), not at load time, so the loads stay in
  // flight across the MFMAs.  Rows past the end hold dy = 0, so the column
  // can be 1 there too.
  auto store_tile = [&](int stage, const V16 (&ra)[4], const V16 (&rb)[4]) {
    char* As = smem + stage * 2 * OPB;
    char* Bs = As + OPB;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      *(uint4*)(As + (r0 + RPP * v) * PIT + ch * 16) = ra[v].u;
      uint4 b = rb[v].u;
      b.x |= onesv.u.x;
      b.y |= onesv.u.y;
      b.z |= onesv.u.z;
      b.w |= onesv.u.w;
      *(uint4*)(Bs + (r0 + RPP * v) * PIT + ch * 16) = b;
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
  if (nk > 0) {
    V16 a0[4], b0[4], a1[4], b1[4];
    load_tile(kt_begin, a0, b0);
    if (nk > 1) load_tile(kt_begin + 1, a1, b1);
    store_tile(0, a0, b0);
    __syncthreads();
    int k = 0;
    for (; k + 1 < nk; k += 2) {  // tiles k (stage 0) and k + 1 (stage 1)
      if (k + 2 < nk) load_tile(kt_begin + k + 2, a0, b0);
      mma_tile_tmajor<T>(smem, smem + OPB, acc, wm, wn, lane);
      store_tile(1, a1, b1);
      __syncthreads();
      if (k + 3 < nk) load_tile(kt_begin + k + 3, a1, b1);
      mma_tile_tmajor<T>(smem + 2 * OPB, smem + 3 * OPB, acc, wm, wn, lane);
      if (k + 2 < nk) store_tile(0, a0, b0);
      __syncthreads();
    }
    if (k < nk) mma_tile_tmajor<T>(smem, smem + OPB, acc, wm, wn, lane);  // odd count: last tile in stage 0
  }

  const int li = lane & 31, lh = lane >> 5;
  if (!a.direct) {
    float* __restrict__ out = a.out + (size_t)split * a.M * a.ldp;
#pragma unroll
    for (int bn = 0; bn < 2; ++bn) {
      const int col = n0 + wn * 64 + bn * 32 + li;
      if (col >= a.Ng) continue;
#pragma unroll
      for (int bm = 0; bm < 2; ++bm)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int row = m0 + wm * 64 + bm * 32 + (v >> 2) * 8 + lh * 4 + (v & 3);
          if (row < a.M) out[(size_t)row * a.ldp + col] = acc[bm][bn][v];
        }
    }
    return;
  }
#pragma unroll
  for (int bn = 0; bn < 2; ++bn) {
    const int col = n0 + wn * 64 + bn * 32 + li;
    if (col >= a.Ng) continue;
    const bool is_db = col == a.Nn;
    float* __restrict__ base = is_db ? a.db : a.out + col;
    const size_t stride = is_db ? 1 : (size_t)a.Nn;
    const int accum = is_db ? a.acc_db : a.acc_dw;
#pragma unroll
    for (int bm = 0; bm < 2; ++bm)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = m0 + wm * 64 + bm * 32 + (v >> 2) * 8 + lh * 4 + (v & 3);
        if (row < a.M) {
          float* o = base + (size_t)row * stride;
          *o = accum ? *o + acc[bm][bn][v] : acc[bm][bn][v];
        }
      }
  }
}

// ----------------------------------------------- filter gradient, large tiles
//
// The same product for bf16 operands with whole 16-byte filter and tap chunks
// (K % 8 == 0, C % 8 == 0), on a 128 (filters) x 256 (taps) tile: each of 8
// waves owns 64 x 64 (2 x 2 blocks of 32 x 32), or, with the update fused,
// each of 4 waves 64 x 128 (2 x 4 blocks).  Operands go from buffer loads
// straight into LDS as t-major rows (256 bytes of filters, 512 bytes of taps
// per reduction index); one load instruction fills 1 KB, i.e. 4 (A) or 2 (B)
// rows.  Rows are unpadded and XOR-swizzled: the 16-byte chunk c of row r sits
// in slot c ^ (4 (r & 3)), so the 4 rows x 2 column groups that 32 lanes of a
// transpose read touch fall in 8 distinct 32-byte bank groups.  Three LDS stages; loads of K-tile k+2 are issued while k
// is multiplied; one barrier per K-tile.  The bias column (tap index Nn) is
// loaded as an out-of-range zero and set to 1 in the B fragments.
// With NFAST, K-tile kt holds images 32 g .. 32 g + 31 at output pixel pq,
// kt = g P Q + pq: consecutive K-tiles step to the neighbouring pixel of the
// same images, whose 3x3 / 5x5 input windows overlap, so the tap rows of a
// split meet again in the L2 (2-3 % faster than running the image groups of
// one pixel back to back).
constexpr int WL_BM = 128, WL_BN = 256, WL_BK = 32;  // BK: reduction rows per K-tile
constexpr int WL_ARB = WL_BM * 2, WL_BRB = WL_BN * 2;  // row bytes
constexpr int WL_AT = WL_BK * WL_ARB, WL_BT = WL_BK * WL_BRB;
constexpr int WL_STAGE = WL_AT + WL_BT;
constexpr int WL_SMEM = 3 * WL_STAGE;  // 72 KB: two workgroups per CU

template <bool NFAST, bool UPD, bool W8>
__device__ __forceinline__ void wgrad_large_body(const WgradArgs& a) {
  constexpr uint32_t ES = 2;
  // waves: 4 of 64 x 128 (2 x 4 blocks of 32 x 32), or with W8 8 of 64 x 64
  constexpr int NWV = W8 ? 8 : 4;
  constexpr int FM = 2, FN = W8 ? 2 : 4;
  constexpr int RPW = WL_BK / NWV;  // K-tile rows loaded by each wave (of A and of B)
  constexpr int AI = RPW / 4;       // A load instructions per wave (4 rows each)
  constexpr int BI = RPW / 2;       // B load instructions per wave (2 rows each)
  static_assert(AI >= 1 && BI >= 2 && BI % 2 == 0, "load split");
  __shared__ __attribute__((aligned(16))) char smem[WL_SMEM];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  const int split = L / a.tiles, tile = L - split * a.tiles;
  const int tm = tile / a.tiles_n, tn = tile - tm * a.tiles_n;
  const int m0 = tm * WL_BM, n0 = tn * WL_BN;
  const int kt_begin = split * a.kt_per_split;
  const int nk = min(a.nkt, kt_begin + a.kt_per_split) - kt_begin;
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, a.x_bytes);
  const __amdgpu_buffer_rsrc_t dyr = make_rsrc(a.dy, a.dy_bytes);
  const int PQ = a.P * a.Q;
  const int ystride = PQ * a.M, xstride = a.H * a.W * a.C;

  // A loads: instruction i fills rows 16 wave + 4 i + lane / 16; this lane's chunk
  const int arow = lane >> 4;
  const int i0 = m0 + 8 * ((lane & 15) ^ (4 * arow));
  const bool aok = i0 < a.M;
  // B loads: instruction i fills rows 16 wave + 2 i + lane / 32; chunk per parity of i
  const int brow = lane >> 5;
  int btap[2], br[2], bs[2];
  bool bok[2];
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const int j0 = n0 + 8 * ((lane & 31) ^ (4 * (2 * p + brow)));
    bok[p] = j0 < a.Nn;
    const int jj = bok[p] ? j0 : 0;
    const int rs = (int)fdiv((uint32_t)jj, a.dC);
    const int c = jj - rs * a.C;
    br[p] = (int)fdiv((uint32_t)rs, a.dS);
    bs[p] = rs - br[p] * a.S;
    btap[p] = (br[p] * a.W + bs[p]) * a.C + c;
  }

  // row d of the K-tile starting at t0 -> (n, output pixel) and validity
  auto row_pix = [&](int t0, int d, int& n, int& pq, bool& tin) {
    if constexpr (NFAST) {
      const int kt = t0 / WL_BK;
      const int g = (int)fdiv((uint32_t)kt, a.dPQ);
      pq = kt - g * PQ;
      n = g * WL_BK + d;
      tin = true;
    } else {
      const int t = t0 + d;
      tin = t < a.T;
      n = (int)fdiv((uint32_t)t, a.dPQ);
      pq = t - n * PQ;
    }
  };
  auto issue = [&](int kt, int stage, int part) {  // part 0: A rows, 1 / 2: first / second half of the B rows
    char* As = smem + stage * WL_STAGE;
    char* Bs = As + WL_AT;
    const int t0 = kt * WL_BK;
    const bool live = kt < kt_begin + nk;
    if (part == 0) {
#pragma unroll
      for (int i = 0; i < AI; ++i) {
        const int d = RPW * wave + 4 * i + arow;
        int n, pq;
        bool tin;
        row_pix(t0, d, n, pq, tin);
        const bool ok = live & tin & aok;
        ld_lds16_asm(dyr, ok ? (uint32_t)(n * ystride + pq * a.M + i0) * ES : OOB, As + (RPW * wave + 4 * i) * WL_ARB);
      }
    } else {
#pragma unroll
      for (int ii = 0; ii < BI / 2; ++ii) {
        const int i = (part - 1) * (BI / 2) + ii;
        const int p = i & 1;
        const int d = RPW * wave + 2 * i + brow;
        int n, pq;
        bool tin;
        row_pix(t0, d, n, pq, tin);
        const int pr = (int)fdiv((uint32_t)pq, a.dQ);
        const int h = pr * a.sh - a.ph + br[p], w = (pq - pr * a.Q) * a.sw - a.pw + bs[p];
        const bool ok = live & tin & bok[p] & ((unsigned)h < (unsigned)a.H) & ((unsigned)w < (unsigned)a.W);
        const int xoff = n * xstride + ((pr * a.sh - a.ph) * a.W + (pq - pr * a.Q) * a.sw - a.pw) * a.C + btap[p];
        ld_lds16_asm(xr, ok ? (uint32_t)xoff * ES : OOB, Bs + (RPW * wave + 2 * i) * WL_BRB);
      }
    }
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  // transpose-read addresses: lane -> column (lane & 31) of a 32-column block,
  // reduction rows 8 (lane / 32) + 0..7 of a 16-row step
  const int wrow = W8 ? (wave >> 2) * 64 : (wave >> 1) * 64, wcol = W8 ? (wave & 3) * 64 : (wave & 1) * 128;
  const int trow = 8 * (lane >> 5) + ((lane & 15) >> 2);
  const int low = 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1);  // chunk bits 0-1 within a 32-column block
  const int rr = (lane & 15) >> 2;                                // row & 3 (same for every step)
  const int off = 8 * (lane & 1);
  int aaddr[FM], baddr[FN];
#pragma unroll
  for (int b = 0; b < FM; ++b) {
    const int x32 = (wrow + b * 32) / 32;  // chunk = 4 x32 + low, stored in slot chunk ^ (4 rr)
    aaddr[b] = trow * WL_ARB + ((4 * (x32 ^ rr) + low) << 4) + off;
  }
#pragma unroll
  for (int b = 0; b < FN; ++b) {
    const int x32 = (wcol + b * 32) / 32;
    baddr[b] = WL_AT + trow * WL_BRB + ((4 * (x32 ^ rr) + low) << 4) + off;
  }
  // the bias column as ones in the B fragments of the wave that holds it
  uint32_t onesm[FN];
  bool bias_wave = false;
#pragma unroll
  for (int b = 0; b < FN; ++b) {
    const int cb = n0 + wcol + b * 32;
    onesm[b] = (a.Ng > a.Nn && cb + (lane & 31) == a.Nn) ? 0x3f803f80u : 0u;
    bias_wave |= a.Ng > a.Nn && cb <= a.Nn && a.Nn < cb + 32;
  }

  auto compute = [&](const char* S) {
#pragma unroll
    for (int kc = 0; kc < WL_BK / 16; ++kc) {
      bf16x8 af[FM], bfr[FN];
#pragma unroll
      for (int b = 0; b < FM; ++b) {
        const v4i16 lo = lds_tr16(S + aaddr[b] + kc * 16 * WL_ARB);
        const v4i16 hi = lds_tr16(S + aaddr[b] + (kc * 16 + 4) * WL_ARB);
        af[b] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      }
#pragma unroll
      for (int b = 0; b < FN; ++b) {
        const v4i16 lo = lds_tr16(S + baddr[b] + kc * 16 * WL_BRB);
        const v4i16 hi = lds_tr16(S + baddr[b] + (kc * 16 + 4) * WL_BRB);
        bfr[b] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      }
      if (bias_wave) {
#pragma unroll
        for (int b = 0; b < FN; ++b) {
          uint4 u = __builtin_bit_cast(uint4, bfr[b]);
          u.x |= onesm[b];
          u.y |= onesm[b];
          u.z |= onesm[b];
          u.w |= onesm[b];
          bfr[b] = __builtin_bit_cast(bf16x8, u);
        }
      }
#pragma unroll
      for (int bm = 0; bm < FM; ++bm)
#pragma unroll
        for (int bn = 0; bn < FN; ++bn)
          acc[bm][bn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[bm], bfr[bn], acc[bm][bn], 0, 0, 0);
    }
  };

  if (nk > 0) {
    constexpr int LOADS = AI + BI;  // per thread per K-tile
#pragma unroll
    for (int part = 0; part < 3; ++part) issue(kt_begin, 0, part);
#pragma unroll
    for (int part = 0; part < 3; ++part) issue(kt_begin + 1, 1, part);
    int stage = 0;
    for (int k = 0; k < nk; ++k) {
      wait_vmcnt<LOADS>();  // tile k has landed for this thread (tile k+1 may be in flight)
      block_barrier();      // ... and for everyone; everyone is done with tile k-1
      // While it issues the A loads and multiplies, the wave takes the SIMD
      // before the other workgroup's wave that computes B addresses or waits
      // (measured 2-5 % faster per layer than equal priorities).
      __builtin_amdgcn_s_setprio(1);
      const int nstage = stage == 0 ? 2 : stage - 1;
      const char* S = smem + stage * WL_STAGE;
      issue(kt_begin + k + 2, nstage, 0);  // past the split's end: all-OOB, no traffic
      compute(S);
      __builtin_amdgcn_s_setprio(0);
      issue(kt_begin + k + 2, nstage, 1);
      issue(kt_begin + k + 2, nstage, 2);
      stage = stage == 2 ? 0 : stage + 1;
    }
    wait_vmcnt<0>();
  }

  const int li = lane & 31, lh = lane >> 5;
  if (!a.direct) {
    float* __restrict__ out = a.out + (size_t)split * a.M * a.ldp;
#pragma unroll
    for (int bn = 0; bn < FN; ++bn) {
      const int col = n0 + wcol + bn * 32 + li;
      if (col >= a.Ng) continue;
#pragma unroll
      for (int bm = 0; bm < FM; ++bm)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int row = m0 + wrow + bm * 32 + (v >> 2) * 8 + lh * 4 + (v & 3);
          if (row < a.M) out[(size_t)row * a.ldp + col] = acc[bm][bn][v];
        }
    }
    return;
  }
  if constexpr (UPD) {
    static_assert(!W8 && FM == 2 && FN == 4, "the update epilogue assumes waves of 64 x 128");
    // Update fused, vector form (taps a multiple of 4, w / v / g 16-byte and
    // the bf16 copy 8-byte aligned): a wave's 64 x 128 block goes through
    // its own LDS region in four passes of 16 rows, so that a lane updates 4
    // consecutive taps of a row with 16-byte non-temporal loads and stores
    // (a wave instruction covers 512 contiguous bytes of each of two rows,
    // against 128 bytes of each with one column per lane); a pass's 16 loads
    // are issued before its staging.  The bias column (tap index Nn, the
    // first of its 4-tap group) is updated on its own.
    const bool v4 = a.Nn % 4 == 0 && (((uintptr_t)a.u.w | (uintptr_t)a.u.v | (uintptr_t)a.out) % 16) == 0 &&
                    ((uintptr_t)a.u.wb % 8) == 0;
    if (v4) {
      constexpr int UP = 128 * 4 + 32;  // row pitch: rows r and r + 4 of a lane pair 32 banks apart
      constexpr int PR = 16;            // rows per pass
      static_assert(4 * PR * UP <= WL_SMEM, "staging fits the operand stages");
      __syncthreads();  // every wave is done with the operand tiles
      char* const q = smem + wave * PR * UP;
      const int g4 = lane & 31, rh = lane >> 5;  // taps 4 g4 .. 4 g4 + 3 of the wave's 128, rows rh, rh + 2, ...
      const int col = n0 + wcol + 4 * g4;
      const bool in_w = col < a.Nn, is_db = col == a.Nn && a.Ng > a.Nn;
#pragma unroll
      for (int pass = 0; pass < 4; ++pass) {
        // block bm = pass / 2, accumulator elements v = 8 (pass % 2) .. + 7
        const int bm = pass >> 1, vb0 = 8 * (pass & 1);
        const int row0 = m0 + wrow + 16 * pass;
        f32x4 wv[PR / 2], vv[PR / 2];
#pragma unroll
        for (int i = 0; i < PR / 2; ++i) {
          // every lane loads (element 0 stands in for rows and taps past the
          // end), so no load sits in a branch that the next must wait for
          const int row = row0 + 2 * i + rh;
          const size_t o = (in_w && row < a.M) ? (size_t)row * a.Nn + col : 0;
          wv[i] = __builtin_nontemporal_load((const f32x4*)(a.u.w + o));
          vv[i] = __builtin_nontemporal_load((const f32x4*)(a.u.v + o));
        }
        // element v of column bn 32 + li is row 8 (v / 4) + 4 lh + v % 4 of the block
#pragma unroll
        for (int bn = 0; bn < FN; ++bn)
#pragma unroll
          for (int v = vb0; v < vb0 + 8; ++v)
            *(float*)(q + (((v >> 2) & 1) * 8 + lh * 4 + (v & 3)) * UP + (bn * 32 + li) * 4) = acc[bm][bn][v];
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes are done
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int i = 0; i < PR / 2; ++i) {
          const int r = 2 * i + rh, row = row0 + r;
          if (row >= a.M) continue;
          const f32x4 gr = *(const f32x4*)(q + r * UP + g4 * 16);
          if (in_w) {
            const size_t o = (size_t)row * a.Nn + col;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              float we = wv[i][e], ve = vv[i][e];
              sgd_step(we, ve, gr[e], a.u.lr, a.u.mom, a.u.wd);
              wv[i][e] = we;
              vv[i][e] = ve;
            }
            __builtin_nontemporal_store(vv[i], (f32x4*)(a.u.v + o));
            __builtin_nontemporal_store(wv[i], (f32x4*)(a.u.w + o));
            if (a.u.wb) {
              const u32x2_t pb = {f32x2_to_bf16x2(wv[i][0], wv[i][1]), f32x2_to_bf16x2(wv[i][2], wv[i][3])};
              __builtin_nontemporal_store(pb, (u32x2_t*)(a.u.wb + o));
            }
            if (a.out) __builtin_nontemporal_store(gr, (f32x4*)(a.out + o));
          }
        }
        if (is_db) {
          // the two lanes that hold the bias column (rows rh, rh + 2, ...)
          float bw[PR / 2], bv[PR / 2];
#pragma unroll
          for (int i = 0; i < PR / 2; ++i) {
            const int row = row0 + 2 * i + rh;
            bw[i] = a.u.b[row < a.M ? row : 0];
            bv[i] = a.u.vb[row < a.M ? row : 0];
          }
#pragma unroll
          for (int i = 0; i < PR / 2; ++i) {
            const int r = 2 * i + rh, row = row0 + r;
            if (row >= a.M) continue;
            const float gb = *(const float*)(q + r * UP + g4 * 16);
            sgd_step(bw[i], bv[i], gb, a.u.lr, a.u.mom, a.u.wd);
            a.u.b[row] = bw[i];
            a.u.vb[row] = bv[i];
            if (a.u.bb) a.u.bb[row] = f32_to_bf16(bw[i]);
            if (a.db) a.db[row] = gb;
          }
        }
      }
      return;
    }
    // Element form: each lane owns one column (filter tap, or the bias) of
    // 32 rows per block; the rows' w and v are loaded before any is used.
#pragma unroll
    for (int bn = 0; bn < FN; ++bn) {
      const int col = n0 + wcol + bn * 32 + li;
      if (col >= a.Ng) continue;
      const bool is_db = col == a.Nn;
      float* __restrict__ W = is_db ? a.u.b : a.u.w + col;
      float* __restrict__ V = is_db ? a.u.vb : a.u.v + col;
      uint16_t* __restrict__ WB = is_db ? a.u.bb : (a.u.wb ? a.u.wb + col : nullptr);
      float* __restrict__ G = is_db ? a.db : (a.out ? a.out + col : nullptr);
      const size_t stride = is_db ? 1 : (size_t)a.Nn;
      float wv[2][16], vv[2][16];
#pragma unroll
      for (int bm = 0; bm < FM; ++bm)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int row = m0 + wrow + bm * 32 + (v >> 2) * 8 + lh * 4 + (v & 3);
          const size_t o = (size_t)(row < a.M ? row : 0) * stride;
          wv[bm][v] = W[o];
          vv[bm][v] = V[o];
        }
#pragma unroll
      for (int bm = 0; bm < FM; ++bm)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int row = m0 + wrow + bm * 32 + (v >> 2) * 8 + lh * 4 + (v & 3);
          if (row >= a.M) continue;
          const size_t o = (size_t)row * stride;
          const float g = acc[bm][bn][v];
          sgd_step(wv[bm][v], vv[bm][v], g, a.u.lr, a.u.mom, a.u.wd);
          W[o] = wv[bm][v];
          V[o] = vv[bm][v];
          if (WB) WB[o] = f32_to_bf16(wv[bm][v]);
          if (G) G[o] = g;
        }
    }
    return;
  }
#pragma unroll
  for (int bn = 0; bn < FN; ++bn) {
    const int col = n0 + wcol + bn * 32 + li;
    if (col >= a.Ng) continue;
    const bool is_db = col == a.Nn;
    float* __restrict__ base = is_db ? a.db : a.out + col;
    const size_t stride = is_db ? 1 : (size_t)a.Nn;
    const int accum = is_db ? a.acc_db : a.acc_dw;
#pragma unroll
    for (int bm = 0; bm < FM; ++bm)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = m0 + wrow + bm * 32 + (v >> 2) * 8 + lh * 4 + (v & 3);
        if (row < a.M) {
          float* o = base + (size_t)row * stride;
          *o = accum ? *o + acc[bm][bn][v] : acc[bm][bn][v];
        }
      }
  }
}

// Eight waves of 64 x 64 for the gradient alone: four waves per SIMD (109
// VGPRs) cover more of the operand stream's latency than two of 64 x 128,
// for a third more fragment reads per MFMA (conv2 0.2512 -> 0.2293 ms,
// conv4 0.1305 -> 0.1201, the others 1-3 %; bitwise the same results).  The
// fused update keeps four waves.
template <bool NFAST, bool UPD>
__global__ __launch_bounds__(UPD ? NT : 2 * NT, 2) void conv_wgrad_large_kernel(WgradArgs a) {
  wgrad_large_body<NFAST, UPD, !UPD>(a);
}

// Filter-gradient split-K reduction over partial[split][M][Ng] (rows of ldp
// floats, ldp % 4 == 0): element (row, col) goes to dw[row][col] for col < Nn
// and to db[row] for col == Nn (the bias column), each added to or
// overwriting its target.  A block of 256 threads is G groups of 256 / G
// lanes; a lane owns 4 consecutive elements of one row, group g sums splits
// g, g + G, g + 2G, ... in that order (four 16-byte loads in flight), then
// group 0 adds the G partial sums in group order, so the result does not
// depend on timing.  Many splits (the first layer's long reduction over few
// filter elements) take G = 16, so the grid still fills the chip.
template <int G, bool UPD>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ partial, int splits, int M,
                                                            int ldp, int Ng, int Nn, float* __restrict__ dw,
                                                            float* __restrict__ db, int acc_dw, int acc_db,
                                                            SgdTargets u) {
  constexpr int LG = 256 / G;
  __shared__ float4 part[G][LG];
  const size_t n = (size_t)M * ldp;
  const int g = threadIdx.x / LG, l = threadIdx.x % LG;
  const size_t i = ((size_t)blockIdx.x * LG + l) * 4;  // 4 consecutive elements of one row (ldp % 4 == 0)
  const int row = (int)(i / (size_t)ldp);
  const int col = (int)(i - (size_t)row * ldp);
  float4 t = make_float4(0.f, 0.f, 0.f, 0.f);
  if (i < n && col < Ng) {
    const float4* __restrict__ p = (const float4*)(partial + i);
    const size_t n4 = n / 4;
    int k = g;
    for (; k + 3 * G < splits; k += 4 * G) {
      float4 q[4];
#pragma unroll
      for (int uu = 0; uu < 4; ++uu) q[uu] = p[(size_t)(k + uu * G) * n4];
#pragma unroll
      for (int uu = 0; uu < 4; ++uu) {
        t.x += q[uu].x; t.y += q[uu].y; t.z += q[uu].z; t.w += q[uu].w;
      }
    }
    for (; k < splits; k += G) {
      const float4 q = p[(size_t)k * n4];
      t.x += q.x; t.y += q.y; t.z += q.z; t.w += q.w;
    }
  }
  part[g][l] = t;
  __syncthreads();
  if (g == 0 && i < n) {
    float4 s = part[0][l];
#pragma unroll
    for (int h = 1; h < G; ++h) {
      const float4 q = part[h][l];
      s.x += q.x; s.y += q.y; s.z += q.z; s.w += q.w;
    }
    const float s4[4] = {s.x, s.y, s.z, s.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int ce = col + e;
      if (ce >= Ng) break;
      const bool is_w = ce < Nn;
      const size_t o = is_w ? (size_t)row * Nn + ce : (size_t)row;
      if constexpr (UPD) {
        // the Updater's step on the complete gradient element; dw / db (may
        // be NULL) also receive the gradient
        float* W = is_w ? u.w : u.b;
        float* V = is_w ? u.v : u.vb;
        uint16_t* WB = is_w ? u.wb : u.bb;
        float* Gd = is_w ? dw : db;
        float wv = W[o], vv = V[o];
        sgd_step(wv, vv, s4[e], u.lr, u.mom, u.wd);
        W[o] = wv;
        V[o] = vv;
        if (WB) WB[o] = f32_to_bf16(wv);
        if (Gd) Gd[o] = s4[e];
      } else {
        float* out = is_w ? dw + o : db + o;
        *out = (is_w ? acc_dw : acc_db) ? *out + s4[e] : s4[e];
      }
    }
  }
}

// Split-K forward: y[i] = act(sum over splits of partial[split][i] + bias[col]),
// splits added in order.
template <typename T>
__global__ __launch_bounds__(256) void splitk_epilogue_kernel(const float* __restrict__ partial, int splits, int M,
                                                              int Nn, const float* __restrict__ bias, int relu,
                                                              const void* mask, T* __restrict__ y) {
  const size_t n = (size_t)M * Nn;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    float t = 0.f;
    for (int k = 0; k < splits; ++k) t += partial[(size_t)k * n + i];
    if (bias) t += bias[i % Nn];
    if (relu) t = fmaxf(t, 0.f);
    if (mask && !mask_pass<T>(mask, i)) t = 0.f;
    store_out<T>(y + i, t);
  }
}

// The same, four consecutive columns per thread (Nn % 4 == 0; y and mask
// aligned to four elements): 16-byte partial loads, four splits' loads in
// flight before they are added, still in split order.
template <typename T>
__global__ __launch_bounds__(256) void splitk_epilogue_vec_kernel(const float* __restrict__ partial, int splits,
                                                                  int M, int Nn, const float* __restrict__ bias,
                                                                  int relu, const void* mask, T* __restrict__ y) {
  struct alignas(4 * sizeof(T)) V4 { T e[4]; };
  const size_t n = (size_t)M * Nn, n4 = n / 4;
  const float4* __restrict__ p4 = (const float4*)partial;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (size_t)gridDim.x * blockDim.x) {
    float4 t = make_float4(0.f, 0.f, 0.f, 0.f);
    int k = 0;
    for (; k + 4 <= splits; k += 4) {
      float4 q[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) q[u] = p4[(size_t)(k + u) * n4 + i];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        t.x += q[u].x; t.y += q[u].y; t.z += q[u].z; t.w += q[u].w;
      }
    }
    for (; k < splits; ++k) {
      const float4 q = p4[(size_t)k * n4 + i];
      t.x += q.x; t.y += q.y; t.z += q.z; t.w += q.w;
    }
    float v[4] = {t.x, t.y, t.z, t.w};
    if (bias) {
      const float4 b = *(const float4*)(bias + (4 * i) % (size_t)Nn);
      v[0] += b.x; v[1] += b.y; v[2] += b.z; v[3] += b.w;
    }
    V4 m;
    if (mask) m = ((const V4*)mask)[i];
    V4 o;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float e = relu ? fmaxf(v[j], 0.f) : v[j];
      if (mask && !(elem_f(m.e[j]) > 0.f)) e = 0.f;
      store_out<T>(&o.e[j], e);
    }
    ((V4*)y)[i] = o;
  }
}

// Layout and split overrides for A/B measurements (SINGA_CONV_TILE,
// SINGA_FWD_BK, SINGA_FWD_WIDE, SINGA_FWD_SHORT, SINGA_FWD_PATCH, SINGA_WGRAD_ORDER, SINGA_WGRAD_TARGET): read
// from the environment only in a library built with -DSINGA_TUNING.  The
// default build ignores the environment; its dispatch rules are the tested
// ones.
#ifdef SINGA_TUNING
inline const char* tuning_env(const char* name) { return getenv(name); }
#else
constexpr const char* tuning_env(const char*) { return nullptr; }
#endif

// "conv_fwd_kernel<dtype,modeA,modeB,bwd>" for each instance, as string
// literals (the launch path writes no state)
#define FWD_NAME(T, A, B, W) "conv_fwd_kernel<" T "," #A "," #B "," #W ">"
#define FWD_NAME_W(T, A, B) {FWD_NAME(T, A, B, 0), FWD_NAME(T, A, B, 1)}
#define FWD_NAME_B(T, A) {FWD_NAME_W(T, A, 0), FWD_NAME_W(T, A, 1), FWD_NAME_W(T, A, 2), FWD_NAME_W(T, A, 3)}
#define FWD_NAME_A(T) {FWD_NAME_B(T, 0), FWD_NAME_B(T, 1), FWD_NAME_B(T, 2)}
constexpr const char* kFwdNames[2][3][4][2] = {FWD_NAME_A("f32"), FWD_NAME_A("bf16")};
#undef FWD_NAME_A
#undef FWD_NAME_B
#undef FWD_NAME_W
#undef FWD_NAME
static_assert(ELEM == 0 && VEC8 == 1 && VEC16 == 2 && BT16 == 3, "name table order");

template <typename T, int AM, int BMD, bool BWD> constexpr const char* fwd_name() {
  return kFwdNames[sizeof(T) == 2][AM][BMD][BWD];
}

template <typename T, int AM, int BMD, bool BWD>
void launch_fwd_instance(const FwdArgs& a, dim3 grid, double flops, hipStream_t st) {
  TraceScope ts(fwd_name<T, AM, BMD, BWD>(), st, flops, WORK_FLOP);
  hipLaunchKernelGGL((conv_fwd_kernel<T, AM, BMD, BWD>), grid, dim3(NT), 0, st, a);
}

// "conv_fwd_large_kernel<bwd,taps per K-tile,wave layout>" (",1" appended:
// the input-patch variant)
const char* fwd_large_name(bool bwd, bool deep, bool narrow, bool wide, bool patch) {
  if (patch) return bwd ? "conv_fwd_large_kernel<1,32,2,1>" : "conv_fwd_large_kernel<0,32,2,1>";
  static const char* names[2][2][2] = {
      {{"conv_fwd_large_kernel<0,32,2>", "conv_fwd_large_kernel<0,32,4>"},
       {"conv_fwd_large_kernel<0,64,2>", "conv_fwd_large_kernel<0,64,4>"}},
      {{"conv_fwd_large_kernel<1,32,2>", "conv_fwd_large_kernel<1,32,4>"},
       {"conv_fwd_large_kernel<1,64,2>", "conv_fwd_large_kernel<1,64,4>"}}};
  if (wide) return bwd ? "conv_fwd_large_kernel<1,32,8>" : "conv_fwd_large_kernel<0,32,8>";
  return names[bwd][deep][narrow];
}

// The 192 x 256 layout instead of 256 x 256 when it takes at most 90 % of
// the 256-row layout's time, counted as rounds of 256 workgroups (one per
// CU) times the rows of a tile.
bool use_short_wide_fwd(long M, long Nn) {
  static const int forced = [] {
    const char* e = tuning_env("SINGA_FWD_SHORT");
    return e ? atoi(e) : -1;
  }();
  if (forced == 0 || forced == 1) return forced == 1;
  const long cols = (Nn + 255) / 256;
  const long t256 = (M + 255) / 256 * cols, t192 = (M + 191) / 192 * cols;
  return 10 * ((t192 + 255) / 256) * 192 <= 9 * ((t256 + 255) / 256) * 256;
}

// Workgroups of the 256 x 128 kernel per full round of the chip (one per CU)
// against those of the 128 x 128 kernel (two per CU): the large tile is used
// when it does not leave a much emptier last round.
// SINGA_CONV_TILE=128 or =256 forces the tile choice in a tuning build
// (read once; anything else, or unset, keeps the automatic rule).
int forced_tile() {
  static const int v = [] {
    const char* e = tuning_env("SINGA_CONV_TILE");
    return e ? atoi(e) : 0;
  }();
  return v;
}

// K-tile depth of the 256 x 128 forward kernel: 32 taps (two workgroups per
// CU, more latency hiding) unless the reduction is very long, where 64 (one
// workgroup per CU, half the barriers) measured faster.  SINGA_FWD_BK=32|64
// forces one.
int fwd_large_bk(long Kg) {
  static const int forced = [] {
    const char* e = tuning_env("SINGA_FWD_BK");
    return e ? atoi(e) : 0;
  }();
  if (forced == 32 || forced == 64) return forced;
  return Kg >= 4096 ? 64 : 32;
}

// The input-patch variant of the 256 x 128 kernel: stride 1, 32-channel
// slices (tap-major K-tiles), at least 4 taps to share a slice's loads, and
// every tile's patch within the buffer.  (On the 256 x 256 layout, one
// workgroup per CU, it measured 5-16 % slower and is not built.)
// SINGA_FWD_PATCH=0 turns it off in a tuning build.
bool use_patch_fwd(const ConvShape& s, long M, bool wide, bool narrow, bool deep) {
  static const int forced = [] {
    const char* e = tuning_env("SINGA_FWD_PATCH");
    return e ? atoi(e) : -1;
  }();
  if (wide || narrow || deep || s.sh != 1 || s.sw != 1 || s.C % 32 != 0 || s.R * s.S < 4 || forced == 0)
    return false;
  const long Hp = s.H + 2L * s.ph, Wp = s.W + 2L * s.pw, PQ = (long)s.P * s.Q;
  const long cap = FWD_PATCH_ENTRIES;
  for (long m0 = 0; m0 < M; m0 += L_BM) {
    const long m1 = std::min(m0 + L_BM, M) - 1;
    const long n0 = m0 / PQ, p0 = (m0 % PQ) / s.Q, n1 = m1 / PQ, p1 = (m1 % PQ) / s.Q;
    if ((n1 * Hp + p1 + s.R - (n0 * Hp + p0)) * Wp > cap) return false;
  }
  return true;
}

bool use_large_fwd(long M, long Nn, long Kg) {
  if (forced_tile() == 128) return false;
  if (forced_tile() == 256) return ((M + L_BM - 1) / L_BM) * ((Nn + BN - 1) / BN) > 0;
  // a very short reduction leaves the prologue and epilogue exposed
  if ((Kg + 63) / 64 < 4) return false;
  const long big = ((M + L_BM - 1) / L_BM) * ((Nn + BN - 1) / BN);
  const long small = ((M + BM - 1) / BM) * ((Nn + BN - 1) / BN);
  if (big < 256) return false;
  const double eff_big = (double)big / (double)(((big + 255) / 256) * 256);
  const double eff_small = (double)small / (double)(((small + 511) / 512) * 512);
  return eff_big >= 0.85 * eff_small;
}

// The 256 x 256 layout (one workgroup of 8 waves per CU) instead of 256 x 128
// (two of 4 waves): when its columns are at least 3/4 used, pad no more than
// the 128-column tiles do, and its rounds of 256 workgroups are about as full
// as the other's rounds of 512.  SINGA_FWD_WIDE=0|1 forces the choice.
bool use_wide_fwd(long M, long Nn) {
  static const int forced = [] {
    const char* e = tuning_env("SINGA_FWD_WIDE");
    return e ? atoi(e) : -1;
  }();
  if (Nn <= 96) return false;
  if (forced == 0 || forced == 1) return forced == 1;
  const long cw = (Nn + 255) / 256 * 256, cn = (Nn + BN - 1) / BN * BN;
  if (cw > cn || 4 * Nn < 3 * cw) return false;
  const long rows = (M + L_BM - 1) / L_BM, tw = rows * (cw / 256), tn = rows * (cn / BN);
  const double eff_w = (double)tw / (double)(((tw + 255) / 256) * 256);
  const double eff_n = (double)tn / (double)(((tn + 511) / 512) * 512);
  return eff_w >= 0.95 * eff_n;
}

int fwd_splits_for(long M, long Nn, long Kg, long bk) {
  const long tiles = ((M + BM - 1) / BM) * ((Nn + BN - 1) / BN);
  const long nkt = (Kg + bk - 1) / bk;
  if (tiles >= 256 || nkt < 8) return 1;
  long splits = (512 + tiles - 1) / tiles;
  if (splits > nkt / 4) splits = nkt / 4;
  if (splits > 16) splits = 16;
  if (splits < 2) return 1;
  const long per = (nkt + splits - 1) / splits;
  return (int)((nkt + per - 1) / per);  // every split gets at least one K-tile
}

template <typename T, int AM, bool BWD>
void launch_fwd_bmode(int bm, const FwdArgs& a, dim3 grid, double flops, hipStream_t st) {
  if (sizeof(T) == 2 && bm == BT16) launch_fwd_instance<T, AM, sizeof(T) == 2 ? BT16 : ELEM, BWD>(a, grid, flops, st);
  else if (bm == VEC16) launch_fwd_instance<T, AM, VEC16, BWD>(a, grid, flops, st);
  else if (sizeof(T) == 2 && bm == VEC8) launch_fwd_instance<T, AM, sizeof(T) == 2 ? VEC8 : ELEM, BWD>(a, grid, flops, st);
  else launch_fwd_instance<T, AM, ELEM, BWD>(a, grid, flops, st);
}

template <typename T, bool BWD>
void launch_fwd_variant(int am, int bm, const FwdArgs& a, dim3 grid, double flops, hipStream_t st) {
  if (am == VEC16) launch_fwd_bmode<T, VEC16, BWD>(bm, a, grid, flops, st);
  else if (sizeof(T) == 2 && am == VEC8) launch_fwd_bmode<T, sizeof(T) == 2 ? VEC8 : ELEM, BWD>(bm, a, grid, flops, st);
  else launch_fwd_bmode<T, ELEM, BWD>(bm, a, grid, flops, st);
}

// Load mode for rows of `len` contiguous elements starting at multiples of
// `len` from base pointer p.
template <typename T> int load_mode(long len, const void* p) {
  constexpr int VEC = 16 / (int)sizeof(T);
  if (len % VEC == 0 && ((uintptr_t)p % 16) == 0) return VEC16;
  if (sizeof(T) == 2 && len % 4 == 0 && ((uintptr_t)p % 8) == 0) return VEC8;
  return ELEM;
}

template <typename T>
hipError_t conv_fwd_dispatch(const ConvShape& s, const void* x, const void* w, const float* bias, void* y,
                             int relu, int bwd, double flops, float* partial, const void* mask, hipStream_t st,
                             bool wt = false) {
  FwdArgs a;
  a.x = x; a.w = w; a.bias = bias; a.y = y; a.mask = mask;
  a.tap_major = 0;
  a.patch = 0; a.Hp = a.Wp = 1;
  a.dHp = a.dWp = make_fastdiv(1u);
  a.RS = s.R * s.S;
  a.dRS = make_fastdiv((uint32_t)a.RS);
  a.x_bytes = (uint32_t)((size_t)s.N * s.H * s.W * s.C * sizeof(T));
  a.w_bytes = (uint32_t)((size_t)s.K * s.R * s.S * s.C * sizeof(T));
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
  a.tiles = tiles_m * a.tiles_n;
  constexpr int BK = KT<T>::BK;
  const int nkt = (a.Kg + BK - 1) / BK;
  const int splits = partial ? fwd_splits_for(a.M, a.Nn, a.Kg, BK) : 1;
  a.partial = splits > 1 ? partial : nullptr;
  a.kt_per_split = (nkt + splits - 1) / splits;
  dim3 grid(a.tiles * splits);
  const int am = load_mode<T>(s.C, x);
  const int bm = wt ? BT16 : load_mode<T>(a.Kg, w);
  if (!wt && sizeof(T) == 2 && am == VEC16 && bm == VEC16 && splits == 1 && use_large_fwd(a.M, a.Nn, a.Kg)) {
    const bool narrow = a.Nn <= 96;  // one 96-column tile
    const bool wide = use_wide_fwd(a.M, a.Nn);
    const bool short_wide = wide && use_short_wide_fwd(a.M, a.Nn);
    const int tile_rows = short_wide ? 192 : L_BM;
    a.tiles_n = (a.Nn + (wide ? 255 : BN - 1)) / (wide ? 256 : BN);
    a.tiles = ((a.M + tile_rows - 1) / tile_rows) * a.tiles_n;
    a.partial = nullptr;
    // 64-tap K-tiles only for the 256 x 128 layout (the 256 x 96 one measured
    // faster at 32 taps, two workgroups per CU, on a 6400-tap reduction; the
    // 256 x 256 one has LDS for three 32-tap stages only and is never deep,
    // whatever SINGA_FWD_BK says)
    const bool deep = !wide && fwd_large_bk(narrow ? 0 : a.Kg) == 64;
    a.kt_per_split = (a.Kg + (deep ? 64 : 32) - 1) / (deep ? 64 : 32);  // one split: every K-tile of this depth
    a.tap_major = a.RS > 1 && s.C % (deep ? 64 : 32) == 0;
    const bool patch = use_patch_fwd(s, a.M, wide, narrow, deep);
    a.patch = patch;
    a.Hp = s.H + 2 * s.ph;
    a.Wp = s.W + 2 * s.pw;
    a.dHp = make_fastdiv((uint32_t)a.Hp);
    a.dWp = make_fastdiv((uint32_t)a.Wp);
    TraceScope ts(short_wide ? (bwd ? "conv_fwd_large_kernel<1,32,6>" : "conv_fwd_large_kernel<0,32,6>")
                             : fwd_large_name(bwd, deep, narrow, wide, patch),
                  st, flops, WORK_FLOP);
#define LAUNCH_LARGE(B, K, W) \
  hipLaunchKernelGGL((conv_fwd_large_kernel<B, K, W, false>), dim3(a.tiles), dim3(W >= 6 ? 2 * NT : NT), 0, st, a)
#define LAUNCH_PATCH(B, W) \
  hipLaunchKernelGGL((conv_fwd_large_kernel<B, 32, W, true>), dim3(a.tiles), dim3(W == 8 ? 2 * NT : NT), 0, st, a)
    if (patch) {
      if (bwd) LAUNCH_PATCH(true, 2); else LAUNCH_PATCH(false, 2);
    } else if (short_wide) {
      if (bwd) LAUNCH_LARGE(true, 32, 6); else LAUNCH_LARGE(false, 32, 6);
    } else if (wide) {
      if (bwd) LAUNCH_LARGE(true, 32, 8); else LAUNCH_LARGE(false, 32, 8);
    } else if (bwd) {
      if (narrow) { if (deep) LAUNCH_LARGE(true, 64, 4); else LAUNCH_LARGE(true, 32, 4); }
      else { if (deep) LAUNCH_LARGE(true, 64, 2); else LAUNCH_LARGE(true, 32, 2); }
    } else {
      if (narrow) { if (deep) LAUNCH_LARGE(false, 64, 4); else LAUNCH_LARGE(false, 32, 4); }
      else { if (deep) LAUNCH_LARGE(false, 64, 2); else LAUNCH_LARGE(false, 32, 2); }
    }
#undef LAUNCH_LARGE
#undef LAUNCH_PATCH
    return hipGetLastError();
  }
  if (bwd)
    launch_fwd_variant<T, true>(am, bm, a, grid, flops, st);
  else
    launch_fwd_variant<T, false>(am, bm, a, grid, flops, st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  const size_t n = (size_t)a.M * a.Nn;
  size_t blocks = (n + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  TraceScope ts("splitk_epilogue_kernel", st, (double)n * (4.0 * splits + sizeof(T)), WORK_BYTE);
  const uintptr_t al = 4 * sizeof(T);
  if (a.Nn % 4 == 0 && (uintptr_t)y % al == 0 && (uintptr_t)mask % al == 0 && (uintptr_t)bias % 16 == 0) {
    size_t vb = (n / 4 + 255) / 256;
    if (vb > 8192) vb = 8192;
    hipLaunchKernelGGL(splitk_epilogue_vec_kernel<T>, dim3((unsigned)vb), dim3(256), 0, st, partial, splits, a.M,
                       a.Nn, bias, relu, mask, (T*)y);
  } else {
    hipLaunchKernelGGL(splitk_epilogue_kernel<T>, dim3((unsigned)blocks), dim3(256), 0, st, partial, splits, a.M,
                       a.Nn, bias, relu, mask, (T*)y);
  }
  return hipGetLastError();
}

// "conv_wgrad_kernel<dtype,vector A,modeB,image fastest>", as literals
#define WG_NAME(T, V, B, F) "conv_wgrad_kernel<" T "," #V "," #B "," #F ">"
#define WG_NAME_F(T, V, B) {WG_NAME(T, V, B, 0), WG_NAME(T, V, B, 1)}
#define WG_NAME_B(T, V) {WG_NAME_F(T, V, 0), WG_NAME_F(T, V, 1), WG_NAME_F(T, V, 2)}
#define WG_NAME_V(T) {WG_NAME_B(T, 0), WG_NAME_B(T, 1)}
constexpr const char* kWgradNames[2][2][3][2] = {WG_NAME_V("f32"), WG_NAME_V("bf16")};
#undef WG_NAME_V
#undef WG_NAME_B
#undef WG_NAME_F
#undef WG_NAME

template <typename T, bool VA, int BMD, bool NF> constexpr const char* wgrad_name() {
  return kWgradNames[sizeof(T) == 2][VA][BMD][NF];
}

template <typename T, bool VA, int BMD, bool NF>
void launch_wgrad_instance(const WgradArgs& a, dim3 grid, double flops, hipStream_t st) {
  TraceScope ts(wgrad_name<T, VA, BMD, NF>(), st, flops, WORK_FLOP);
  hipLaunchKernelGGL((conv_wgrad_kernel<T, VA, BMD, NF>), grid, dim3(NT), 0, st, a);
}

template <typename T, bool VA, bool NF>
void launch_wgrad_bmode(int bm, const WgradArgs& a, dim3 grid, double flops, hipStream_t st) {
  if (bm == VEC16) launch_wgrad_instance<T, VA, VEC16, NF>(a, grid, flops, st);
  else if (sizeof(T) == 2 && bm == VEC8)
    launch_wgrad_instance<T, VA, sizeof(T) == 2 ? VEC8 : ELEM, NF>(a, grid, flops, st);
  else launch_wgrad_instance<T, VA, ELEM, NF>(a, grid, flops, st);
}

template <typename T, bool NF>
void launch_wgrad_variant(bool va, int bm, const WgradArgs& a, dim3 grid, double flops, hipStream_t st) {
  if (va) launch_wgrad_bmode<T, true, NF>(bm, a, grid, flops, st);
  else launch_wgrad_bmode<T, false, NF>(bm, a, grid, flops, st);
}

// Reduction order of the filter gradient: K-tiles of BK images at one output
// pixel (needs N % BK == 0) or image-major.  The large kernel, which steps
// such K-tiles along neighbouring pixels, takes the former whenever it can
// (measured faster on every AlexNet layer, the first one included); the
// 128 x 128 kernel only when an image has few output pixels (otherwise
// image-major keeps a workgroup's input reads local).
// SINGA_WGRAD_ORDER=image|pixel forces one.
bool use_image_fastest(const ConvShape& s, int bk, bool large) {
  static const int forced = [] {
    const char* e = tuning_env("SINGA_WGRAD_ORDER");
    if (!e) return 0;
    return e[0] == 'p' ? 1 : e[0] == 'i' ? 2 : 0;  // pixel-major (image fastest) / image-major
  }();
  if (s.N % bk != 0) return false;
  if (forced) return forced == 1;
  return large || s.P * s.Q < 1024;
}

// Split-K count of the filter gradient on `tiles` output tiles and `nkt`
// K-tiles: about `target` workgroups, at least 8 K-tiles each, every split
// non-empty.
int wgrad_split_count(long tiles, long nkt, long target) {
  long splits = (target + tiles - 1) / tiles;
  const long max_by_len = nkt / 8;
  if (splits > max_by_len) splits = max_by_len;
  if (splits < 1) splits = 1;
  if (splits > 256) splits = 256;
  const long per = (nkt + splits - 1) / splits;
  return (int)((nkt + per - 1) / per);
}

// The 128 x 256 kernel: bf16 with whole 16-byte filter and tap chunks
// (SINGA_CONV_TILE=128 keeps the 128 x 128 kernel).
bool wgrad_large_shape(const ConvShape& s, int dt) {
  return dt == BF16 && s.K % 8 == 0 && s.C % 8 == 0 && forced_tile() != 128;
}

// Splits used by the kernel that runs shape s (large: the 128 x 256 kernel).
int wgrad_splits_for(const ConvShape& s, int dt, bool bias, bool large) {
  const long M = s.K, Ng = (long)s.R * s.S * s.C + (bias ? 1 : 0), T = (long)s.N * s.P * s.Q;
  if (large) {
    const long tiles = ((M + WL_BM - 1) / WL_BM) * ((Ng + WL_BN - 1) / WL_BN);
    // about 448 workgroups: one round a little under the 512 slots of two
    // workgroups per CU, so that the backward-data passes that run beside
    // the filter gradient on another stream keep some CUs.  Measured on the
    // AlexNet training step (two streams): 432 - 480 give the best step,
    // 2.5 % faster than 640 (1280 for conv2) and 512, which fill the chip
    // or spill into a second round.  A layer of at most 4 output tiles takes
    // 640 (AlexNet's conv1, whose long reduction runs last, with nothing
    // beside it: 8 us per step faster).  SINGA_WGRAD_TARGET overrides both.
    static const long forced = [] {
      const char* e = tuning_env("SINGA_WGRAD_TARGET");
      const long v = e ? atol(e) : 0;
      return v > 0 ? v : 0L;
    }();
    const long nkt = (T + WL_BK - 1) / WL_BK;
    const long target = forced ? forced : tiles <= 4 ? 640 : 448;
    return wgrad_split_count(tiles, nkt, target);
  }
  const long tiles = ((M + BM - 1) / BM) * ((Ng + BN - 1) / BN);
  const long bk = dt == BF16 ? WG<bf16_t>::BK : WG<float>::BK;
  return wgrad_split_count(tiles, (T + bk - 1) / bk, 1024);  // about 4 workgroups per CU
}

template <typename T>
hipError_t conv_wgrad_dispatch(const ConvShape& s, const void* x, const void* dy, float* partial, float* dw,
                               float* db, int acc_dw, int acc_db, const SgdTargets* upd, double flops,
                               hipStream_t st) {
  constexpr int VEC = 16 / (int)sizeof(T);
  constexpr int DT = sizeof(T) == 2 ? BF16 : F32;
  WgradArgs a;
  a.x = x; a.dy = dy;
  a.x_bytes = (uint32_t)((size_t)s.N * s.H * s.W * s.C * sizeof(T));
  a.dy_bytes = (uint32_t)((size_t)s.N * s.P * s.Q * s.K * sizeof(T));
  a.M = s.K;
  a.Nn = s.R * s.S * s.C;
  a.T = s.N * s.P * s.Q;
  a.N = s.N; a.H = s.H; a.W = s.W; a.C = s.C; a.S = s.S; a.P = s.P; a.Q = s.Q;
  a.sh = s.sh; a.sw = s.sw; a.ph = s.ph; a.pw = s.pw;
  a.dN = make_fastdiv((uint32_t)s.N);
  a.dPQ = make_fastdiv((uint32_t)(s.P * s.Q));
  a.dQ = make_fastdiv((uint32_t)s.Q);
  a.dC = make_fastdiv((uint32_t)s.C);
  a.dS = make_fastdiv((uint32_t)s.S);
  const bool va = (a.M % VEC) == 0 && ((uintptr_t)dy % 16) == 0;
  const int vb = load_mode<T>(s.C, x);
  const bool large = wgrad_large_shape(s, DT) && va && vb == VEC16;
  const int bm = large ? WL_BM : BM, bn = large ? WL_BN : BN, bk = large ? WL_BK : WG<T>::BK;
  a.nkt = (a.T + bk - 1) / bk;
  const bool bias = upd ? upd->b != nullptr : db != nullptr;
  a.Ng = a.Nn + (bias ? 1 : 0);
  a.ldp = (a.Ng + 63) / 64 * 64;
  a.tiles_n = (a.Ng + bn - 1) / bn;
  a.tiles = ((a.M + bm - 1) / bm) * a.tiles_n;
  const int splits = wgrad_splits_for(s, DT, bias, large);
  // the update goes into the large kernel when it writes each element once,
  // otherwise into the split-K reduction; a single split of the 128 x 128
  // kernel has no place for it
  if (upd && splits == 1 && !(large && wgrad_update_fusable(s, DT, bias))) return hipErrorNotSupported;
  if (upd && splits > 1 && !partial) return hipErrorNotSupported;
  a.kt_per_split = (a.nkt + splits - 1) / splits;
  a.direct = splits == 1;
  a.acc_dw = upd ? 0 : acc_dw;
  a.acc_db = upd ? 0 : acc_db;
  a.out = a.direct ? dw : partial;
  a.db = db;
  a.update = upd != nullptr && a.direct;  // split: the reduction applies it
  if (upd) a.u = *upd;
  dim3 grid(a.tiles * splits);
  const bool nf = use_image_fastest(s, bk, large);
  if (large) {
    // "conv_wgrad_large_kernel<image fastest,update fused>"
    static const char* names[2][2] = {{"conv_wgrad_large_kernel<0,0>", "conv_wgrad_large_kernel<0,1>"},
                                      {"conv_wgrad_large_kernel<1,0>", "conv_wgrad_large_kernel<1,1>"}};
    TraceScope ts(names[nf][a.update], st, flops, WORK_FLOP);
    if (a.update) {
      if (nf) hipLaunchKernelGGL((conv_wgrad_large_kernel<true, true>), grid, dim3(NT), 0, st, a);
      else hipLaunchKernelGGL((conv_wgrad_large_kernel<false, true>), grid, dim3(NT), 0, st, a);
    } else {
      if (nf) hipLaunchKernelGGL((conv_wgrad_large_kernel<true, false>), grid, dim3(2 * NT), 0, st, a);
      else hipLaunchKernelGGL((conv_wgrad_large_kernel<false, false>), grid, dim3(2 * NT), 0, st, a);
    }
  } else if (nf) {
    launch_wgrad_variant<T, true>(va, vb, a, grid, flops, st);
  } else {
    launch_wgrad_variant<T, false>(va, vb, a, grid, flops, st);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  // fixed-order sum of the partial tiles into dw (and db), or, with the
  // update, the Updater's step on each summed element
  const size_t n = (size_t)a.M * a.ldp;
  const SgdTargets none{};
  if (upd) {
    const double bytes = (double)a.M * a.Ng * (4.0 * splits + 18.0 + (dw ? 4.0 : 0.0));
    TraceScope ts("splitk_reduce_sgd_kernel", st, bytes, WORK_BYTE);
    if (splits >= 64)
      hipLaunchKernelGGL((splitk_reduce_kernel<16, true>), dim3((unsigned)((n + 63) / 64)), dim3(256), 0, st, partial,
                         splits, a.M, a.ldp, a.Ng, a.Nn, dw, db, 0, 0, *upd);
    else
      hipLaunchKernelGGL((splitk_reduce_kernel<4, true>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, partial,
                         splits, a.M, a.ldp, a.Ng, a.Nn, dw, db, 0, 0, *upd);
    return hipGetLastError();
  }
  TraceScope ts("splitk_reduce_kernel", st, (double)a.M * a.Ng * 4.0 * (splits + 1 + (acc_dw ? 1 : 0)), WORK_BYTE);
  if (splits >= 64)
    hipLaunchKernelGGL((splitk_reduce_kernel<16, false>), dim3((unsigned)((n + 63) / 64)), dim3(256), 0, st, partial,
                       splits, a.M, a.ldp, a.Ng, a.Nn, dw, db, acc_dw, acc_db, none);
  else
    hipLaunchKernelGGL((splitk_reduce_kernel<4, false>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, partial,
                       splits, a.M, a.ldp, a.Ng, a.Nn, dw, db, acc_dw, acc_db, none);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_conv_fwd(int dt, const ConvShape& s, const void* x, const void* w, const float* bias, void* y,
                           int relu, int bwd, double flops, float* partial, const void* mask, hipStream_t st) {
  if (dt == BF16) return conv_fwd_dispatch<bf16_t>(s, x, w, bias, y, relu, bwd, flops, partial, mask, st);
  return conv_fwd_dispatch<float>(s, x, w, bias, y, relu, bwd, flops, partial, mask, st);
}

hipError_t launch_conv_fwd_wt(int dt, const ConvShape& s, const void* x, const void* wt, void* y, int bwd,
                              double flops, float* partial, const void* mask, hipStream_t st) {
  if (dt != BF16 || s.R != 1 || s.S != 1 || s.K % 8 != 0 || (uintptr_t)wt % 16 != 0 ||
      (size_t)s.C * s.K * 2 > 0x7fffffffu)
    return hipErrorNotSupported;
  return conv_fwd_dispatch<bf16_t>(s, x, wt, nullptr, y, 0, bwd, flops, partial, mask, st, true);
}

size_t fwd_partial_bytes(const ConvShape& s, int dt) {
  const long M = (long)s.N * s.P * s.Q, Nn = s.K, Kg = (long)s.R * s.S * s.C;
  const int splits = fwd_splits_for(M, Nn, Kg, dt == BF16 ? KT<bf16_t>::BK : KT<float>::BK);
  return splits > 1 ? (size_t)splits * M * Nn * sizeof(float) : 0;
}

size_t wgrad_partial_bytes(const ConvShape& s, int dt, bool bias) {
  const size_t Ng = (size_t)s.R * s.S * s.C + (bias ? 1 : 0);
  const size_t ldp = (Ng + 63) / 64 * 64;
  // either kernel may run (the large one also needs aligned pointers)
  int splits = wgrad_splits_for(s, dt, bias, false);
  if (wgrad_large_shape(s, dt)) splits = std::max(splits, wgrad_splits_for(s, dt, bias, true));
  return splits > 1 ? (size_t)splits * s.K * ldp * sizeof(float) : 0;
}

hipError_t launch_conv_wgrad(int dt, const ConvShape& s, const void* x, const void* dy, float* partial, float* dw,
                             float* db, int acc_dw, int acc_db, double flops, hipStream_t st) {
  if (dt == BF16) return conv_wgrad_dispatch<bf16_t>(s, x, dy, partial, dw, db, acc_dw, acc_db, nullptr, flops, st);
  return conv_wgrad_dispatch<float>(s, x, dy, partial, dw, db, acc_dw, acc_db, nullptr, flops, st);
}

bool wgrad_update_fusable(const ConvShape& s, int dt, bool bias) {
  return wgrad_large_shape(s, dt) && wgrad_splits_for(s, dt, bias, true) == 1;
}

hipError_t launch_conv_wgrad_reduce_sgd(int dt, const ConvShape& s, const void* x, const void* dy, float* partial,
                                        float* dw, float* db, const SgdTargets& u, double flops, hipStream_t st) {
  if (!partial) return hipErrorNotSupported;
  if (dt == BF16) return conv_wgrad_dispatch<bf16_t>(s, x, dy, partial, dw, u.b ? db : nullptr, 0, 0, &u, flops, st);
  return conv_wgrad_dispatch<float>(s, x, dy, partial, dw, u.b ? db : nullptr, 0, 0, &u, flops, st);
}

hipError_t launch_conv_wgrad_sgd(int dt, const ConvShape& s, const void* x, const void* dy, float* dw, float* db,
                                 const SgdTargets& u, hipStream_t st) {
  if (dt != BF16 || !wgrad_update_fusable(s, dt, u.b != nullptr) || (uintptr_t)x % 16 || (uintptr_t)dy % 16)
    return hipErrorNotSupported;
  // never a rewritten geometry: the GEMM's work is the layer's
  const double flops = 2.0 * s.N * (double)s.P * s.Q * s.K * (double)s.R * s.S * s.C;
  return conv_wgrad_dispatch<bf16_t>(s, x, dy, nullptr, dw, u.b ? db : nullptr, 0, 0, &u, flops, st);
}

}  // namespace singa
