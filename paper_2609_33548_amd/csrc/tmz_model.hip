// BitNet decoder forward around the ternary BitLinear projections, and the
// next-token cross-entropy that TerMeZO evaluates at w +/- eps z (Sec. 3,
// eq. objective_est).  The full-precision parameters are the token embedding
// (tied to the LM head) and the RMSNorm weights (one unless the caller gives a
// weight table); when they are registered as theta the forward reads their
// current, possibly perturbed, values.  Activations are stored in fp32 or bf16
// between kernels.  The RMSNorm output feeding a projection goes to the int8
// activation quantiser in fp32 without being stored; the SwiGLU product
// silu(g) * u is stored in the activation dtype (by the fused gate|up GEMM
// epilogue for bf16, by a row kernel otherwise) and then quantised.
#include <algorithm>
#include <cmath>
#include <new>
#include <string>
#include <type_traits>
#include <vector>

#include <hip/hip_ext.h>

#include "tmz_device.h"
#include "tmz_internal.h"

namespace tmz {

typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float round_to(const float*, float v) { return v; }
__device__ __forceinline__ float round_to(const uint16_t*, float v) { return (float)(__bf16)v; }
__device__ __forceinline__ float ld_act(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ld_act(const uint16_t* p, int64_t i) { return bf16_to_f32(p[i]); }
__device__ __forceinline__ void st_act(float* p, int64_t i, float v) { p[i] = v; }
__device__ __forceinline__ void st_act(uint16_t* p, int64_t i, float v) { p[i] = f32_to_bf16_rne(v); }

__device__ __forceinline__ float wsum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}
__device__ __forceinline__ int wsum_i(int v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}
__device__ __forceinline__ float wmax(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

// Block (256 threads) reductions through a 4-entry LDS scratch.
__device__ __forceinline__ float bsum(float v, float* red) {
  v = wsum(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}
__device__ __forceinline__ float bmax(float v, float* red) {
  v = wmax(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

__device__ __forceinline__ int8_t q8(float x, float s) {
  return (int8_t)fminf(fmaxf(__builtin_rintf(x * s), -128.0f), 127.0f);
}


// ---------------------------------------------------------------------------
// h[m] = E[tok[m]].  An id outside [0, V) reads row 0 instead and sets bit 8 of
// the deferred error word, so the embedding is never read out of bounds.
// ---------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) k_embed(const int32_t* tok, const T* E, int64_t d,
                                               int64_t V, T* h, int32_t* err) {
  const int64_t m = blockIdx.x;
  int64_t t = tok[m];
  if (t < 0 || t >= V) {
    if (threadIdx.x == 0) atomicOr(err, 8);
    t = 0;
  }
  const T* src = E + t * d;
  T* dst = h + m * d;
  constexpr int EPC = 16 / (int)sizeof(T);    // elements per 16-byte chunk
  const bool vec = d % EPC == 0 && reinterpret_cast<uintptr_t>(E) % 16 == 0 &&
                   reinterpret_cast<uintptr_t>(h) % 16 == 0;
  if (vec) {
    for (int64_t c = threadIdx.x; c < d / EPC; c += 256)
      reinterpret_cast<uint4*>(dst)[c] = reinterpret_cast<const uint4*>(src)[c];
  } else {
    for (int64_t i = threadIdx.x; i < d; i += 256) dst[i] = src[i];
  }
}

// ---------------------------------------------------------------------------
// Row kernels, one wave per token row, 8 elements (one 16-byte bf16 load, or
// two 16-byte fp32 loads) per lane per chunk, the row kept in registers:
//   kRowNormQuant  x = (h / sqrt(mean(h^2) + eps)) * weight (RMSNorm; the weight
//                  row is the u argument, one when null), then
//                  the 8-bit quantiser: s = 127 / max(max|x|, 1e-5),
//                  x_q = clamp(rne(x s), -128, 127)
//   kRowNormStore  the RMSNorm output stored in the activation dtype
//   kRowSwiGLU     a = silu(g) * u rounded to the activation dtype, then the quantiser
//   kRowQuant      the quantiser alone
// Rows up to 64 * 8 * kRowChunks elements.
// ---------------------------------------------------------------------------
constexpr int kRowNormQuant = 0, kRowNormStore = 1, kRowSwiGLU = 2, kRowQuant = 3;
constexpr int kRowChunks = 16;

__device__ __forceinline__ void load8(const uint16_t* p, float v[8]) {
  const uint4 r = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    v[2 * j] = __uint_as_float(w[j] << 16);
    v[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
  }
}
__device__ __forceinline__ void load8(const float* p, float v[8]) {
  const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ void store8(uint16_t* p, const float v[8]) {
  uint32_t w[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const __bf16 a = (__bf16)v[2 * j], b = (__bf16)v[2 * j + 1];
    w[j] = (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
  }
  *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
}
__device__ __forceinline__ void store8(float* p, const float v[8]) {
  reinterpret_cast<float4*>(p)[0] = make_float4(v[0], v[1], v[2], v[3]);
  reinterpret_cast<float4*>(p)[1] = make_float4(v[4], v[5], v[6], v[7]);
}

// Eight bf16 values of a 16-byte chunk to fp32, and back (exact: the values are
// bf16 numbers).
__device__ __forceinline__ void unpack8(const uint4 r, float v[8]) {
  const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    v[2 * j] = __uint_as_float(w[j] << 16);
    v[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
  }
}
__device__ __forceinline__ uint4 pack8(const float v[8]) {
  uint32_t w[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
    w[j] = (__float_as_uint(v[2 * j]) >> 16) | (__float_as_uint(v[2 * j + 1]) & 0xFFFF0000u);
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// Long bf16 rows: the row stays in registers as packed bf16 (4 registers per chunk:
// the input, or for the SwiGLU the rounded product, both bf16 numbers); the RMSNorm
// output is recomputed from it where it is needed, with the same operations.  (For
// rows of up to 8 chunks per lane the fp32 copy below leaves enough waves per SIMD
// and measured faster.)
template <int MODE, bool WEIGHTED, int CH>
__device__ __forceinline__ void row_bf16(const uint16_t* __restrict__ x,
                                         const uint16_t* __restrict__ u, int64_t m, int64_t K,
                                         float eps, int8_t* xq, float* xs, int32_t* xrs,
                                         uint16_t* xf) {
  const int lane = threadIdx.x & 63;
  const int nch = (int)(K / 8);
  uint4 raw[CH];
  float acc = 0.0f;
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int idx = c * 64 + lane;
    raw[c] = make_uint4(0u, 0u, 0u, 0u);
    if (idx < nch) {
      raw[c] = *reinterpret_cast<const uint4*>(x + m * K + idx * 8);
      float v[8];
      unpack8(raw[c], v);
      if (MODE == kRowSwiGLU) {
        float uu[8];
        load8(u + m * K + idx * 8, uu);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          v[j] = round_to(x, silu_mul(v[j], uu[j]));   // the product is an activation
          acc = fmaxf(acc, fabsf(v[j]));
        }
        raw[c] = pack8(v);
      } else if (MODE == kRowQuant) {
#pragma unroll
        for (int j = 0; j < 8; ++j) acc = fmaxf(acc, fabsf(v[j]));
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) acc = fmaf(v[j], v[j], acc);
      }
    }
  }
  float r = 1.0f;
  // the values the quantiser sees, for chunk c (the RMSNorm output, or the row itself)
  auto values = [&](int c, float v[8]) __attribute__((always_inline)) {
    unpack8(raw[c], v);
    if (MODE == kRowNormQuant || MODE == kRowNormStore) {
      if constexpr (WEIGHTED) {            // RMSNorm weight row (the u argument)
        float wt[8] = {1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f};
        const int idx = c * 64 + lane;
        if (idx < nch) load8(u + idx * 8, wt);
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = v[j] * r * wt[j];
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = v[j] * r;
      }
    }
  };
  float amax;
  if (MODE == kRowSwiGLU || MODE == kRowQuant) {
    amax = wmax(acc);
  } else {
    const float ss = wsum(acc);
    r = __fdiv_rn(1.0f, sqrt_rn(ss / (float)K + eps));
    float a = 0.0f;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const int idx = c * 64 + lane;
      if (idx < nch) {
        float v[8];
        values(c, v);
        if (MODE == kRowNormStore) {
          store8(xf + m * K + idx * 8, v);
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j) a = fmaxf(a, fabsf(v[j]));
        }
      }
    }
    if (MODE == kRowNormStore) return;
    amax = wmax(a);
  }
  const float sc = __fdiv_rn(127.0f, fmaxf(amax, 1e-5f));
  if (lane == 0) xs[m] = sc;
  int qs = 0;                                 // sum of the row's quantised values
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int idx = c * 64 + lane;
    if (idx < nch) {
      float v[8];
      values(c, v);
      uint32_t w0 = 0, w1 = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int8_t q0 = q8(v[j], sc), q1 = q8(v[4 + j], sc);
        qs += q0 + q1;
        w0 |= ((uint32_t)(uint8_t)q0) << (8 * j);
        w1 |= ((uint32_t)(uint8_t)q1) << (8 * j);
      }
      *reinterpret_cast<uint2*>(xq + m * K + idx * 8) = make_uint2(w0, w1);
    }
  }
  qs = wsum_i(qs);
  if (lane == 0) xrs[m] = qs;
}

// The same row work on a bf16 row already in registers (packed, 8 values per chunk):
// modes other than kRowSwiGLU.
template <int MODE, bool WEIGHTED, int CH>
__device__ __forceinline__ void row_bf16_held(const uint4 (&raw)[CH], const uint16_t* __restrict__ u,
                                              int64_t m, int64_t K, float eps, int8_t* xq,
                                              float* xs, int32_t* xrs, uint16_t* xf) {
  static_assert(MODE != kRowSwiGLU, "mode");
  const int lane = threadIdx.x & 63;
  const int nch = (int)(K / 8);
  float acc = 0.0f;
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    float v[8];
    unpack8(raw[c], v);                       // zero beyond the row: no effect below
    if (MODE == kRowQuant) {
#pragma unroll
      for (int j = 0; j < 8; ++j) acc = fmaxf(acc, fabsf(v[j]));
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) acc = fmaf(v[j], v[j], acc);
    }
  }
  float r = 1.0f;
  auto values = [&](int c, float v[8]) __attribute__((always_inline)) {
    unpack8(raw[c], v);
    if (MODE == kRowNormQuant || MODE == kRowNormStore) {
      if constexpr (WEIGHTED) {
        float wt[8] = {1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f};
        const int idx = c * 64 + lane;
        if (idx < nch) load8(u + idx * 8, wt);
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = v[j] * r * wt[j];
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = v[j] * r;
      }
    }
  };
  float amax;
  if (MODE == kRowQuant) {
    amax = wmax(acc);
  } else {
    const float ss = wsum(acc);
    r = __fdiv_rn(1.0f, sqrt_rn(ss / (float)K + eps));
    float a = 0.0f;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const int idx = c * 64 + lane;
      if (idx < nch) {
        float v[8];
        values(c, v);
        if (MODE == kRowNormStore) {
          store8(xf + m * K + idx * 8, v);
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j) a = fmaxf(a, fabsf(v[j]));
        }
      }
    }
    if (MODE == kRowNormStore) return;
    amax = wmax(a);
  }
  const float sc = __fdiv_rn(127.0f, fmaxf(amax, 1e-5f));
  if (lane == 0) xs[m] = sc;
  int qs = 0;
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int idx = c * 64 + lane;
    if (idx < nch) {
      float v[8];
      values(c, v);
      uint32_t w0 = 0, w1 = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int8_t q0 = q8(v[j], sc), q1 = q8(v[4 + j], sc);
        qs += q0 + q1;
        w0 |= ((uint32_t)(uint8_t)q0) << (8 * j);
        w1 |= ((uint32_t)(uint8_t)q1) << (8 * j);
      }
      *reinterpret_cast<uint2*>(xq + m * K + idx * 8) = make_uint2(w0, w1);
    }
  }
  qs = wsum_i(qs);
  if (lane == 0) xrs[m] = qs;
}

// bf16 rows, modes other than kRowSwiGLU: a grid of at most the resident blocks, each
// wave walking rows m, m + 4 grid, ...; the next row's loads are issued before the
// current row is worked on, so a wave with two rows has both in flight.  (With one row
// per wave the 8192 rows of a step took about 1.3 rounds of resident waves, the last
// one mostly idle.)
template <int MODE, bool WEIGHTED, int CH>
__global__ void __launch_bounds__(256) k_row_pf(const uint16_t* __restrict__ x,
                                                const uint16_t* __restrict__ u, int64_t M,
                                                int64_t K, float eps, int8_t* xq, float* xs,
                                                int32_t* xrs, uint16_t* xf) {
  const int lane = threadIdx.x & 63;
  const int64_t stride = (int64_t)gridDim.x * 4;
  int64_t m = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (m >= M) return;                         // whole wave
  const int nch = (int)(K / 8);
  auto load = [&](int64_t r, uint4 (&dst)[CH]) __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const int idx = c * 64 + lane;
      dst[c] = make_uint4(0u, 0u, 0u, 0u);
      if (idx < nch) dst[c] = *reinterpret_cast<const uint4*>(x + r * K + idx * 8);
    }
  };
  uint4 nxt[CH];
  load(m, nxt);
  for (; m < M; m += stride) {
    uint4 cur[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) cur[c] = nxt[c];
    if (m + stride < M) load(m + stride, nxt);
    row_bf16_held<MODE, WEIGHTED, CH>(cur, u, m, K, eps, xq, xs, xrs, xf);
  }
}

// CH: chunks per lane the row needs at most (the kernel is instantiated for a few
// row lengths so that the registers holding the row match it).
template <int MODE, typename T, bool WEIGHTED = false, int CH = kRowChunks>
__global__ void __launch_bounds__(256) k_row(const T* __restrict__ x, const T* __restrict__ u,
                                             int64_t M, int64_t K, float eps, int8_t* xq,
                                             float* xs, int32_t* xrs, T* xf) {
  const int lane = threadIdx.x & 63;
  const int64_t m = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (m >= M) return;                       // whole wave
  if constexpr (sizeof(T) == 2 && CH > 8) {   // long rows: half the registers
    row_bf16<MODE, WEIGHTED, CH>(x, u, m, K, eps, xq, xs, xrs, xf);
    return;
  }
  const int nch = (int)(K / 8);
  float v[CH][8];
  float acc = 0.0f;
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int idx = c * 64 + lane;
    if (idx < nch) {
      load8(x + m * K + idx * 8, v[c]);
      if (MODE == kRowSwiGLU) {
        float uu[8];
        load8(u + m * K + idx * 8, uu);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          v[c][j] = round_to(x, silu_mul(v[c][j], uu[j]));   // the product is an activation
          acc = fmaxf(acc, fabsf(v[c][j]));
        }
      } else if (MODE == kRowQuant) {
#pragma unroll
        for (int j = 0; j < 8; ++j) acc = fmaxf(acc, fabsf(v[c][j]));
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) acc = fmaf(v[c][j], v[c][j], acc);
      }
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) v[c][j] = 0.0f;
    }
  }
  float amax;
  if (MODE == kRowSwiGLU || MODE == kRowQuant) {
    amax = wmax(acc);
  } else {
    const float ss = wsum(acc);
    const float r = __fdiv_rn(1.0f, sqrt_rn(ss / (float)K + eps));
    float a = 0.0f;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      if constexpr (WEIGHTED) {            // RMSNorm weight row (the u argument)
        float wt[8] = {1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f};
        const int idx = c * 64 + lane;
        if (idx < nch) load8(u + idx * 8, wt);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          v[c][j] = v[c][j] * r * wt[j];
          a = fmaxf(a, fabsf(v[c][j]));
        }
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          v[c][j] = v[c][j] * r;
          a = fmaxf(a, fabsf(v[c][j]));
        }
      }
    }
    if (MODE == kRowNormStore) {
#pragma unroll
      for (int c = 0; c < CH; ++c) {
        const int idx = c * 64 + lane;
        if (idx < nch) store8(xf + m * K + idx * 8, v[c]);
      }
      return;
    }
    amax = wmax(a);
  }
  const float sc = __fdiv_rn(127.0f, fmaxf(amax, 1e-5f));
  if (lane == 0) xs[m] = sc;
  int qs = 0;                                 // sum of the row's quantised values
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int idx = c * 64 + lane;
    if (idx < nch) {
      uint32_t w0 = 0, w1 = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int8_t q0 = q8(v[c][j], sc), q1 = q8(v[c][4 + j], sc);
        qs += q0 + q1;
        w0 |= ((uint32_t)(uint8_t)q0) << (8 * j);
        w1 |= ((uint32_t)(uint8_t)q1) << (8 * j);
      }
      *reinterpret_cast<uint2*>(xq + m * K + idx * 8) = make_uint2(w0, w1);
    }
  }
  qs = wsum_i(qs);
  if (lane == 0) xrs[m] = qs;
}

// One row kernel launch (4 rows per block), instantiated for the chunks per lane
// the row length needs: 3 (up to 1536 elements), 5 (2560), 8 (4096), 14 (7168),
// else kRowChunks.
template <int MODE, bool W, int CH>
static unsigned row_pf_grid(int64_t M, int n_cu) {
  static int per_cu = -1;                       // resident blocks per compute unit
  if (per_cu < 0) {
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, k_row_pf<MODE, W, CH>, 256, 0) !=
            hipSuccess || nb < 1)
      nb = 1;
    per_cu = nb;
  }
  const int64_t need = (M + 3) / 4;
  const int64_t cap = (int64_t)per_cu * (n_cu > 0 ? n_cu : 1);
  return (unsigned)(need < cap ? need : cap);
}

template <int MODE, typename T, bool W = false>
static void row_launch(unsigned grid, hipStream_t s, const T* x, const T* u, int64_t M, int64_t K,
                       float eps, int8_t* xq, float* xs, int32_t* xrs, T* xf, int n_cu = 0) {
  const int64_t need = (K / 8 + 63) / 64;
  // the prefetching walk measured faster for the quantiser alone (12.7 against 13.1 us at
  // 8192 x 2560, 32.3 against 35.3 us at 8192 x 6912) and for rows of more than 8 chunks per
  // lane, slower for RMSNorm + quantiser at 2560 (14.3 against 13.7 us: more registers)
  if constexpr (sizeof(T) == 2 && MODE != kRowSwiGLU) {
    if (n_cu > 0 && need <= 14 && (MODE == kRowQuant || need > 8)) {
#define TMZ_ROWPF(CHN)                                                                        \
  hipLaunchKernelGGL((k_row_pf<MODE, W, CHN>), dim3(row_pf_grid<MODE, W, CHN>(M, n_cu)),      \
                     dim3(256), 0, s, x, u, M, K, eps, xq, xs, xrs, xf)
      if (need <= 3)
        TMZ_ROWPF(3);
      else if (need <= 5)
        TMZ_ROWPF(5);
      else if (need <= 8)
        TMZ_ROWPF(8);
      else
        TMZ_ROWPF(14);
#undef TMZ_ROWPF
      return;
    }
  }
#define TMZ_ROW(CHN) \
  hipLaunchKernelGGL((k_row<MODE, T, W, CHN>), dim3(grid), dim3(256), 0, s, x, u, M, K, eps, xq, xs, xrs, xf)
  if (need <= 3)
    TMZ_ROW(3);
  else if (need <= 5)
    TMZ_ROW(5);
  else if (need <= 8)
    TMZ_ROW(8);
  else if (need <= 14)
    TMZ_ROW(14);
  else
    TMZ_ROW(kRowChunks);
#undef TMZ_ROW
}

// ---------------------------------------------------------------------------
// Rotary embedding in place on x [M][H * hd]; pairs (i, i + hd/2) rotated by
// the angle pos * base^(-2i/hd), cos/sin from a table [S][hd/2].
// ---------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) k_rope(T* x, int64_t M, int H, int hd, int S,
                                              const float* cs, const float* sn) {
  const int half = hd / 2;
  const int64_t total = M * H * half;
  for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * 256) {
    const int i = (int)(t % half);
    const int64_t mh = t / half;
    const int64_t m = mh / H;
    const int h = (int)(mh % H);
    const int p = (int)(m % S);
    const float c = cs[p * half + i], s = sn[p * half + i];
    const int64_t base = m * (int64_t)H * hd + (int64_t)h * hd;
    const float a = ld_act(x, base + i), b = ld_act(x, base + i + half);
    st_act(x, base + i, a * c - b * s);
    st_act(x, base + i + half, a * s + b * c);
  }
}

// ---------------------------------------------------------------------------
// Causal GQA attention, fp32 activations (small shapes): one block per
// (query row, head); scores staged in LDS.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) k_attn_f32(const float* q, const float* k, const float* v,
                                                  float* o, int S, int Hq, int Hkv, int hd,
                                                  float scale) {
  extern __shared__ float sc[];  // S scores
  __shared__ float red[4];
  const int64_t m = blockIdx.x;  // b * S + p
  const int h = blockIdx.y;
  const int p = (int)(m % S);
  const int64_t b0 = m - p;
  const int kh = h / (Hq / Hkv);
  const float* qr = q + m * (int64_t)Hq * hd + (int64_t)h * hd;
  float mx = -INFINITY;
  for (int j = threadIdx.x; j <= p; j += 256) {
    const float* kr = k + (b0 + j) * (int64_t)Hkv * hd + (int64_t)kh * hd;
    float acc = 0.0f;
    for (int e = 0; e < hd; ++e) acc = fmaf(qr[e], kr[e], acc);
    sc[j] = acc * scale;
    mx = fmaxf(mx, sc[j]);
  }
  mx = bmax(mx, red);
  float sum = 0.0f;
  for (int j = threadIdx.x; j <= p; j += 256) {
    const float e = expf(sc[j] - mx);
    sc[j] = e;
    sum += e;
  }
  sum = bsum(sum, red);
  __syncthreads();
  for (int e = threadIdx.x; e < hd; e += 256) {
    float acc = 0.0f;
    for (int j = 0; j <= p; ++j) acc = fmaf(sc[j], v[(b0 + j) * (int64_t)Hkv * hd + (int64_t)kh * hd + e], acc);
    o[m * (int64_t)Hq * hd + (int64_t)h * hd + e] = acc / sum;
  }
}

// ---------------------------------------------------------------------------
// Per-layer preparation of K and V for attention (one block per 64 tokens of
// one KV head): K is rotated in place (RoPE, as in k_rope), V is transposed to
// vt [B*Hkv][hd][S] through an LDS tile (16-byte reads and writes).
// ---------------------------------------------------------------------------
// Rotary embedding of one 8-dim chunk at dims d0..d0+7 given its partner
// chunk (d0 -/+ hd/2), as in k_rope: low half a c - b s, high half a s + b c
// (a = low-half value, b = high-half value), rounded to bf16.
__device__ __forceinline__ uint4 rope_chunk(uint4 own, uint4 par, bool low, const float* cs,
                                            const float* sn) {
  float o8[8], p8[8];
  load8(reinterpret_cast<const uint16_t*>(&own), o8);
  load8(reinterpret_cast<const uint16_t*>(&par), p8);
  float r[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float c = cs[j], sv = sn[j];
    r[j] = low ? o8[j] * c - p8[j] * sv : p8[j] * sv + o8[j] * c;
  }
  return make_uint4(pack_bf16x2(r[0], r[1]), pack_bf16x2(r[2], r[3]), pack_bf16x2(r[4], r[5]),
                    pack_bf16x2(r[6], r[7]));
}

template <int HD>
__global__ void __launch_bounds__(256) k_kv_prep(uint16_t* __restrict__ k,
                                                 const uint16_t* __restrict__ v,
                                                 uint16_t* __restrict__ vt, int S, int Hkv,
                                                 const float* __restrict__ rope_c,
                                                 const float* __restrict__ rope_s) {
  constexpr int HALF = HD / 2;
  __shared__ __attribute__((aligned(16))) uint16_t t[64][HD + 8];
  const int s0 = blockIdx.x * 64, bh = blockIdx.y;
  const int b = bh / Hkv, h = bh % Hkv;
  const int64_t rowkv = (int64_t)Hkv * HD;
  // V rows first (64 tokens in 16-byte chunks, into registers): their latency overlaps the
  // rotation of K below
  constexpr int VPT = 64 * HD / 8 / 256;     // chunks per thread
  uint4 vreg[VPT];
#pragma unroll
  for (int q = 0; q < VPT; ++q) {
    const int i = q * 256 + threadIdx.x;
    const int r = i / (HD / 8), c8 = (i % (HD / 8)) * 8;
    vreg[q] = make_uint4(0, 0, 0, 0);
    if (s0 + r < S) vreg[q] = *reinterpret_cast<const uint4*>(v + ((int64_t)b * S + s0 + r) * rowkv + (int64_t)h * HD + c8);
  }
  // K: rotary chunk pairs, in place
  for (int e = threadIdx.x; e < 64 * HALF / 8; e += 256) {
    const int r = e / (HALF / 8), dc = (e % (HALF / 8)) * 8;
    if (s0 + r >= S) continue;
    uint16_t* kp = k + ((int64_t)b * S + s0 + r) * rowkv + (int64_t)h * HD;
    const uint4 lo = *reinterpret_cast<const uint4*>(kp + dc);
    const uint4 hi = *reinterpret_cast<const uint4*>(kp + dc + HALF);
    const int ti = (s0 + r) * HALF + dc;
    *reinterpret_cast<uint4*>(kp + dc) = rope_chunk(lo, hi, true, rope_c + ti, rope_s + ti);
    *reinterpret_cast<uint4*>(kp + dc + HALF) = rope_chunk(hi, lo, false, rope_c + ti, rope_s + ti);
  }
  // V^T: the token rows into LDS, then 8 tokens of one dim per 16-byte store
#pragma unroll
  for (int q = 0; q < VPT; ++q) {
    const int i = q * 256 + threadIdx.x;
    const int r = i / (HD / 8), c8 = (i % (HD / 8)) * 8;
    *reinterpret_cast<uint4*>(&t[r][c8]) = vreg[q];
  }
  __syncthreads();
  for (int i = threadIdx.x; i < HD * 8; i += 256) {
    const int r = i / 8, c8 = (i % 8) * 8;   // r: dim, c8: first of 8 tokens
    uint32_t w[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) w[j] = (uint32_t)t[c8 + 2 * j][r] | ((uint32_t)t[c8 + 2 * j + 1][r] << 16);
    uint16_t* dst = vt + ((int64_t)bh * HD + r) * S + s0 + c8;
    if ((S & 7) == 0 && s0 + c8 + 8 <= S) {
      *reinterpret_cast<uint4*>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (s0 + c8 + j < S) dst[j] = t[c8 + j][r];
    }
  }
}

// ---------------------------------------------------------------------------
// Causal GQA flash attention on bf16 matrix cores (v_mfma_f32_16x16x32_bf16).
// Block = 128 queries of one (batch, head), 8 waves of 16 queries.  For each
// 64-key tile: S^T = K Q^T (K from LDS as the A operand, rope(Q)^T from
// registers as B), online softmax per query column (the query is the lane's
// column, so row statistics stay in the lane), then O^T += V^T P^T with P^T
// taken straight from the S^T accumulators (K index of the 32-key step: group
// g, element j -> key 16 (j / 4) + 4 g + j % 4) and V^T rows from vt.  K/V
// tiles are double-buffered in LDS with the next tile's global loads in
// flight during the current tile's MFMAs; a wave skips tiles entirely in its
// causal future, and only the diagonal tile is masked.
// ---------------------------------------------------------------------------
template <int HD>
__global__ void __launch_bounds__(512) k_attn_bf16(const uint16_t* __restrict__ q,
                                                   const uint16_t* __restrict__ k,
                                                   const uint16_t* __restrict__ vt,
                                                   uint16_t* __restrict__ o, int S, int Hq,
                                                   int Hkv, float scale_log2,
                                                   const float* __restrict__ rope_c,
                                                   const float* __restrict__ rope_s) {
  constexpr int HALF = HD / 2;
  constexpr int QB = 128;              // queries per block
  constexpr int KT = 64;               // keys per tile
  constexpr int KS = HD + 8;           // K tile row stride (bf16)
  constexpr int VS = KT + 8;           // V^T tile row stride (bf16)
  constexpr int KCH = KT * HD / 8;     // 16-byte chunks per K tile (= per V^T tile)
  constexpr int CPT = (KCH + 511) / 512;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2][KT * KS];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[2][HD * VS];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int c = lane & 15, g = lane >> 4;
  const int qt = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int kh = h / (Hq / Hkv);
  const int64_t rowq = (int64_t)Hq * HD, rowkv = (int64_t)Hkv * HD;
  const int64_t base = (int64_t)b * S;
  const uint16_t* kb = k + base * rowkv + (int64_t)kh * HD;
  const uint16_t* vtb = vt + ((int64_t)b * Hkv + kh) * HD * S;
  const int qw0 = qt * QB + w * 16;             // first query of this wave
  const int qpos = qw0 + c;                     // this lane's query
  const bool vec_v = (S & 7) == 0;

  // rope(Q)^T fragments: lane holds rope(Q)[qpos][32 s + 8 g .. +7]
  v8bf qf[HD / 32];
#pragma unroll
  for (int s = 0; s < HD / 32; ++s) {
    uint4 raw = make_uint4(0, 0, 0, 0);
    if (qpos < S) {
      const int d0 = 32 * s + 8 * g;
      const bool low = d0 < HALF;
      const uint16_t* qr = q + (base + qpos) * rowq + (int64_t)h * HD;
      const uint4 own = *reinterpret_cast<const uint4*>(qr + d0);
      const uint4 par = *reinterpret_cast<const uint4*>(qr + (low ? d0 + HALF : d0 - HALF));
      const int ti = qpos * HALF + (low ? d0 : d0 - HALF);
      raw = rope_chunk(own, par, low, rope_c + ti, rope_s + ti);
    }
    qf[s] = __builtin_bit_cast(v8bf, raw);
  }

  uint4 rk[CPT], rv[CPT];
  auto gload = [&](int kt) __attribute__((always_inline)) {
    const int k0 = kt * KT;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int e = tid + 512 * i;
      rk[i] = make_uint4(0, 0, 0, 0);
      rv[i] = make_uint4(0, 0, 0, 0);
      if (e < KCH) {
        const int kr = e / (HD / 8), dc = (e % (HD / 8)) * 8;
        if (k0 + kr < S) rk[i] = *reinterpret_cast<const uint4*>(kb + (int64_t)(k0 + kr) * rowkv + dc);
        const int dr = e / (KT / 8), kc = (e % (KT / 8)) * 8;
        const uint16_t* vp = vtb + (int64_t)dr * S + k0 + kc;
        if (vec_v && k0 + kc + 8 <= S) {
          rv[i] = *reinterpret_cast<const uint4*>(vp);
        } else {
          uint32_t t4[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const uint32_t lo16 = (k0 + kc + 2 * j < S) ? vp[2 * j] : 0u;
            const uint32_t hi16 = (k0 + kc + 2 * j + 1 < S) ? vp[2 * j + 1] : 0u;
            t4[j] = lo16 | (hi16 << 16);
          }
          rv[i] = make_uint4(t4[0], t4[1], t4[2], t4[3]);
        }
      }
    }
  };
  auto lstore = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int e = tid + 512 * i;
      if (e < KCH) {
        const int kr = e / (HD / 8), dc = (e % (HD / 8)) * 8;
        *reinterpret_cast<uint4*>(&Ks[buf][kr * KS + dc]) = rk[i];
        const int dr = e / (KT / 8), kc = (e % (KT / 8)) * 8;
        *reinterpret_cast<uint4*>(&Vs[buf][dr * VS + kc]) = rv[i];
      }
    }
  };

  v4f ot[HD / 16];
#pragma unroll
  for (int t = 0; t < HD / 16; ++t) ot[t] = v4f{0.f, 0.f, 0.f, 0.f};
  float mrun = -INFINITY, lrun = 0.0f;

  const int q_last = min(qt * QB + QB, S) - 1;             // block's last query
  const int ntile = q_last / KT + 1;
  gload(0);
  lstore(0);
  if (ntile > 1) gload(1);
  __syncthreads();
  for (int kt = 0; kt < ntile; ++kt) {
    const int k0 = kt * KT;
    const uint16_t* Kb = Ks[kt & 1];
    const uint16_t* Vb = Vs[kt & 1];
    if (k0 <= qw0 + 15 && qw0 < S) {            // wave-uniform: tile not entirely in the future
      v4f st[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        st[t] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < HD / 32; ++s) {
          const uint4 raw = *reinterpret_cast<const uint4*>(Kb + (16 * t + c) * KS + 32 * s + 8 * g);
          st[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, raw), qf[s],
                                                          st[t], 0, 0, 0);
        }
      }
      // st[t][i] = score(query qpos, key k0 + 16 t + 4 g + i)
      const bool diag = k0 + KT - 1 > qw0;      // some key may exceed some query of the wave
      float mx = mrun;
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float sv = st[t][i] * scale_log2;
          if (diag) {
            const int key = k0 + 16 * t + 4 * g + i;
            if (key > qpos || key >= S) sv = -INFINITY;
          }
          st[t][i] = sv;
          mx = fmaxf(mx, sv);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mnew = mx;
      const float alpha = (mrun == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(mrun - mnew);
      mrun = mnew;
      float psum = 0.0f;
      v8bf pf[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        uint32_t pk[4];
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const int j0 = 2 * jj, j1 = 2 * jj + 1;
          const float p0 = __builtin_amdgcn_exp2f(st[2 * hh + j0 / 4][j0 % 4] - mnew);
          const float p1 = __builtin_amdgcn_exp2f(st[2 * hh + j1 / 4][j1 % 4] - mnew);
          psum += p0 + p1;
          const __bf16 b0 = (__bf16)p0, b1 = (__bf16)p1;
          pk[jj] = (uint32_t)__builtin_bit_cast(uint16_t, b0) |
                   ((uint32_t)__builtin_bit_cast(uint16_t, b1) << 16);
        }
        pf[hh] = __builtin_bit_cast(v8bf, make_uint4(pk[0], pk[1], pk[2], pk[3]));
      }
      lrun = lrun * alpha + psum;
#pragma unroll
      for (int t = 0; t < HD / 16; ++t) {
        ot[t] *= alpha;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const uint16_t* vr = Vb + (16 * t + c) * VS + 32 * hh + 4 * g;
          const uint2 lo = *reinterpret_cast<const uint2*>(vr);
          const uint2 hi = *reinterpret_cast<const uint2*>(vr + 16);
          const v8bf af = __builtin_bit_cast(v8bf, make_uint4(lo.x, lo.y, hi.x, hi.y));
          ot[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, pf[hh], ot[t], 0, 0, 0);
        }
      }
    }
    if (kt + 1 < ntile) {
      lstore((kt + 1) & 1);
      if (kt + 2 < ntile) gload(kt + 2);
    }
    __syncthreads();
  }
  lrun += __shfl_xor(lrun, 16, 64);
  lrun += __shfl_xor(lrun, 32, 64);
  if (qpos < S) {
    const float inv = 1.0f / lrun;
    uint16_t* orow = o + (base + qpos) * rowq + (int64_t)h * HD;
#pragma unroll
    for (int t = 0; t < HD / 16; ++t) {
      const __bf16 e0 = (__bf16)(ot[t][0] * inv), e1 = (__bf16)(ot[t][1] * inv);
      const __bf16 e2 = (__bf16)(ot[t][2] * inv), e3 = (__bf16)(ot[t][3] * inv);
      const uint32_t w0 = (uint32_t)__builtin_bit_cast(uint16_t, e0) |
                          ((uint32_t)__builtin_bit_cast(uint16_t, e1) << 16);
      const uint32_t w1 = (uint32_t)__builtin_bit_cast(uint16_t, e2) |
                          ((uint32_t)__builtin_bit_cast(uint16_t, e3) << 16);
      *reinterpret_cast<uint2*>(orow + 16 * t + 4 * g) = make_uint2(w0, w1);
    }
  }
}

// ---------------------------------------------------------------------------
// Causal GQA flash attention for a whole query group (v_mfma_f32_32x32x16_bf16).
// Block = QT = 256 / G queries of one (sequence, KV head) for all G query
// heads that share the KV head, 8 waves of 32 (query, head) rows, so every K
// and V^T tile brought into LDS feeds all G heads.
//  * Q: the block's rows are read coalesced (item = one query and one pair of
//    rotary-partner 16-byte chunks, for all G heads, so the cos/sin entries
//    are read once per query), rotated, and staged in LDS; each wave then
//    takes its rope(Q)^T fragments into registers.  The normalised output
//    goes back through the same staging rows and leaves as whole rows.
//  * Per 64-key tile a wave computes S^T = K rope(Q)^T (K rows from LDS as
//    the first operand), an online softmax per query (the query is the lane's
//    accumulator column, so its statistics stay in the lane pair l, l ^ 32)
//    and O^T += V^T P^T with P^T taken straight from the S^T accumulators.
//    For that the K rows of a 32-key block are read in the order pi (bits 2
//    and 3 of the row swapped): accumulator element j of lane half h then
//    holds key 16 (j / 8) + 8 h + j % 8, i.e. in every 16-key step a lane owns
//    8 consecutive keys, the B-operand layout, and the matching V^T fragment
//    is one 16-byte chunk of a V^T row.  The row sum is taken from the bf16
//    probabilities that enter the product (v_dot2 with ones).
//  * K and V^T tiles stream through 2 LDS stages with direct global -> LDS
//    loads; 16-byte chunk c of a K row r sits at c ^ (r & 15) (128-dim rows),
//    c ^ ((r >> 1) & 7) (64-dim rows) or c ^ ((r >> 2) & 3) (96-dim rows of 12
//    chunks: the swap stays inside aligned groups of 4 chunks), of a V^T row at
//    c ^ ((r >> 1) & 7), so the fragment reads of 16 lanes hit distinct banks;
//    staging rows put chunk c at c ^ (r & (CPR - 1)) (96-dim rows: c ^ (r & 3)).
//  * 32-key blocks entirely in a wave's causal future are skipped and only
//    the diagonal block is masked.  The running maximum is raised only when a
//    tile's maximum exceeds it by more than 2^8 (in exp2 units); the
//    normalised result does not depend on that choice.  Query tiles are
//    dispatched heaviest first.
// Requires S % 64 == 0 and S % QT == 0.
// ---------------------------------------------------------------------------
template <int HD, int G>
__global__ void __launch_bounds__(512) k_attn_gqa(const uint16_t* __restrict__ q,
                                                  const uint16_t* __restrict__ k,
                                                  const uint16_t* __restrict__ vt,
                                                  uint16_t* __restrict__ o, int S, int Hkv,
                                                  int nbh, int nqt, float scale_log2,
                                                  const float* __restrict__ rope_c,
                                                  const float* __restrict__ rope_s) {
  constexpr int HALF = HD / 2;
  constexpr int QT = 256 / G;                 // queries per block
  constexpr int KT = 64;                      // keys per stage
  constexpr int KROWB = 2 * HD, CPR = HD / 8; // bytes and 16-byte chunks per K / Q row
  constexpr int TB = KT * KROWB;              // bytes per K tile (= per V^T tile)
  constexpr int QB = 256 * KROWB;             // Q / O staging: 256 (query, head) rows
  constexpr int NLD = TB / 1024;              // 1 KB loads per operand per stage
  constexpr int LPW = (NLD + 7) / 8;          // per wave (load L = 8 j + wave, L < NLD)
  constexpr int NS = HD / 16;                 // 16-dim K steps of S^T
  constexpr int ND = HD / 32;                 // 32-dim blocks of O^T
  static_assert(HD == 64 || HD == 96 || HD == 128, "head dim");
  static_assert(TB % 1024 == 0, "tile");
  static_assert(G == 1 || G == 2 || G == 4 || G == 8, "group");
  __shared__ __attribute__((aligned(1024))) uint8_t lds[4 * TB + QB];
  uint8_t* stg = lds + 4 * TB;                // Q / O staging rows (query r, head g) -> r G + g
  auto swk = [](int r) __attribute__((always_inline)) {
    return CPR == 16 ? (r & 15) : CPR == 12 ? ((r >> 2) & 3) : ((r >> 1) & 7);
  };
  auto sws = [](int r) __attribute__((always_inline)) {   // staging rows
    return CPR == 12 ? (r & 3) : (r & (CPR - 1));
  };
  auto swv = [](int r) __attribute__((always_inline)) { return (r >> 1) & 7; };

  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 31, h = lane >> 5;
  const int lb = blockIdx.x;
  const int qt = nqt - 1 - lb / nbh, bh = lb % nbh;
  const int b = bh / Hkv, kvh = bh % Hkv;
  const int Hq = Hkv * G;
  const int64_t rowq = (int64_t)Hq * HD, rowkv = (int64_t)Hkv * HD;
  const int64_t base = (int64_t)b * S;
  const int q0 = qt * QT;
  const int hq0 = kvh * G;                    // first query head of the group
  const int rq = 32 * (wid / G) + n;          // this lane's query within the block
  const int qw0 = q0 + 32 * (wid / G);        // first query of this wave
  const int qpos = q0 + rq;                   // this lane's query
  const int srow = rq * G + wid % G;          // this lane's staging row

  // direct-load sources: load L = 8 j + w (wave w, L < NLD) fills LDS chunks 64 L + lane
  const uint8_t* ksrc[LPW];
  const uint8_t* vsrc[LPW];
#pragma unroll
  for (int j = 0; j < LPW; ++j) {
    const int L = 8 * j + wid;
    const int c = (L < NLD ? L : 0) * 64 + lane;
    const int kr = c / CPR, kc = (c % CPR) ^ swk(kr);
    ksrc[j] = reinterpret_cast<const uint8_t*>(k + (base + kr) * rowkv + (int64_t)kvh * HD) + 16 * kc;
    const int vr = c / 8, vc = (c % 8) ^ swv(vr);
    vsrc[j] = reinterpret_cast<const uint8_t*>(vt + (((int64_t)b * Hkv + kvh) * HD + vr) * S) + 16 * vc;
  }
  auto issue = [&](int kt, int st) __attribute__((always_inline)) {
    const uint32_t kb = lds_offset(lds + st * 2 * TB), vb = kb + TB;
#pragma unroll
    for (int j = 0; j < LPW; ++j) {
      const int L = 8 * j + wid;                   // wave-uniform
      if (NLD % 8 == 0 || L < NLD) {
        dma16(ksrc[j] + (int64_t)kt * KT * rowkv * 2, kb + 1024u * L);
        dma16(vsrc[j] + (int64_t)kt * KT * 2, vb + 1024u * L);
      }
    }
  };

  const int ntile = (q0 + QT - 1) / KT + 1;
  issue(0, 0);

  // rope(Q) into the staging rows
  for (int it = tid; it < QT * (CPR / 2); it += 512) {
    const int r = it / (CPR / 2), cg = it % (CPR / 2);
    const int pos = q0 + r;
    const uint16_t* qr = q + (base + pos) * rowq + (int64_t)hq0 * HD + 8 * cg;
    uint4 lo[G], hi[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      lo[g] = *reinterpret_cast<const uint4*>(qr + g * HD);
      hi[g] = *reinterpret_cast<const uint4*>(qr + g * HD + HALF);
    }
    const int ti = pos * HALF + 8 * cg;
    const int sw = sws(r);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      uint8_t* row = stg + (r * G + g) * KROWB;
      *reinterpret_cast<uint4*>(row + 16 * (cg ^ sw)) = rope_chunk(lo[g], hi[g], true, rope_c + ti, rope_s + ti);
      *reinterpret_cast<uint4*>(row + 16 * ((cg + CPR / 2) ^ sw)) =
          rope_chunk(hi[g], lo[g], false, rope_c + ti, rope_s + ti);
    }
  }
  __syncthreads();
  // rope(Q)^T fragments: for K step s the lane holds dims 16 s + 8 h .. + 7 of its query
  v8bf qf[NS];
  {
    const uint8_t* row = stg + srow * KROWB;
#pragma unroll
    for (int s = 0; s < NS; ++s)
      qf[s] = __builtin_bit_cast(v8bf, *reinterpret_cast<const uint4*>(row + 16 * ((2 * s + h) ^ sws(rq))));
  }

  v16f ot[ND];
#pragma unroll
  for (int d = 0; d < ND; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) ot[d][r] = 0.0f;
  float mrun = -INFINITY, lrun = 0.0f;

  typedef uint32_t v4u __attribute__((ext_vector_type(4)));
  // K row read by lane n of a 32-key block: pi(n) swaps bits 2 and 3
  const int krow = (n & ~12) | ((n & 4) << 1) | ((n & 8) >> 1);
  // lane parts of the fragment addresses (stage, key block and dim block parts are constants)
  uint32_t kad[NS], vad[4];
#pragma unroll
  for (int s = 0; s < NS; ++s) kad[s] = krow * KROWB + 16 * ((2 * s + h) ^ swk(krow));
#pragma unroll
  for (int s = 0; s < 4; ++s) vad[s] = n * 128 + 16 * ((2 * s + h) ^ swv(n));
  const v2bf ones2 = {(__bf16)1.0f, (__bf16)1.0f};

  // one 64-key tile of keys k0.. in stage ST with NKB 32-key blocks; diag: mask the last one
  auto tile = [&](auto st_c, int k0, auto nkb_c, bool diag) __attribute__((always_inline)) {
    constexpr int NKB = decltype(nkb_c)::value;
    constexpr int ST = decltype(st_c)::value;
    const uint8_t* Ks = lds + ST * 2 * TB;
    const uint8_t* Vs = Ks + TB;
    v16f sc[NKB];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sc[kb][r] = 0.0f;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const v8bf kf = __builtin_bit_cast(v8bf, *reinterpret_cast<const v4u*>(Ks + kad[s] + 32 * kb * KROWB));
        sc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s], sc[kb], 0, 0, 0);
      }
    }
    if (diag) {   // key offset within the last block vs this lane's query offset
      const int lim = qpos - (k0 + 32 * (NKB - 1));
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (16 * (r >> 3) + 8 * h + (r & 7) > lim) sc[NKB - 1][r] = -INFINITY;
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[kb][r]);
    {   // combine the two lane halves (same query, other keys)
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
      mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
    }
    const float ms = mx * scale_log2;
    const bool raise = ms > mrun + 8.0f;
    if (__builtin_amdgcn_ballot_w64(raise)) {
      const float mnew = raise ? ms : mrun;
      const float alpha = __builtin_amdgcn_exp2f(mrun - mnew);
      lrun *= alpha;
#pragma unroll
      for (int d = 0; d < ND; ++d) ot[d] *= alpha;
      mrun = mnew;
    }
    v8bf pf[2 * NKB];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        uint32_t pk[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float p0 = __builtin_amdgcn_exp2f(fmaf(sc[kb][8 * t + 2 * i], scale_log2, -mrun));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(sc[kb][8 * t + 2 * i + 1], scale_log2, -mrun));
          pk[i] = pack_bf16x2(p0, p1);
          lrun = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(v2bf, pk[i]), ones2, lrun, false);
        }
        pf[2 * kb + t] = __builtin_bit_cast(v8bf, make_uint4(pk[0], pk[1], pk[2], pk[3]));
      }
#pragma unroll
    for (int s = 0; s < 2 * NKB; ++s)
#pragma unroll
      for (int d = 0; d < ND; ++d) {
        const v8bf vf = __builtin_bit_cast(v8bf, *reinterpret_cast<const v4u*>(Vs + vad[s] + 32 * d * 128));
        ot[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[s], ot[d], 0, 0, 0);
      }
  };

  // tile kt in stage kt & 1; the next tile's loads are in flight during the current one
  auto body = [&](int kt, auto st_c) __attribute__((always_inline)) {
    constexpr int ST = decltype(st_c)::value;
    if (kt + 1 < ntile) issue(kt + 1, ST ^ 1);
    const int k0 = kt * KT;
    if (k0 + 32 < qw0) {
      tile(st_c, k0, std::integral_constant<int, 2>{}, false);
    } else if (k0 + 32 == qw0) {
      tile(st_c, k0, std::integral_constant<int, 2>{}, true);
    } else if (k0 == qw0) {
      tile(st_c, k0, std::integral_constant<int, 1>{}, true);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  };
  for (int kt = 0; kt < ntile; kt += 2) {
    body(kt, std::integral_constant<int, 0>{});
    if (kt + 1 < ntile) body(kt + 1, std::integral_constant<int, 1>{});
  }

  {
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(lrun), __float_as_uint(lrun), false, false);
    lrun = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
  }
  const float inv = 1.0f / lrun;
  {
    uint8_t* row = stg + srow * KROWB;
#pragma unroll
    for (int d = 0; d < ND; ++d)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const uint32_t w0 = pack_bf16x2(ot[d][4 * g] * inv, ot[d][4 * g + 1] * inv);
        const uint32_t w1 = pack_bf16x2(ot[d][4 * g + 2] * inv, ot[d][4 * g + 3] * inv);
        *reinterpret_cast<uint2*>(row + 16 * ((4 * d + g) ^ sws(rq)) + 8 * h) = make_uint2(w0, w1);
      }
  }
  __syncthreads();
  for (int it = tid; it < QT * (CPR / 2); it += 512) {
    const int r = it / (CPR / 2), cg = it % (CPR / 2);
    const int sw = sws(r);
    uint16_t* orow = o + (base + q0 + r) * rowq + (int64_t)hq0 * HD + 8 * cg;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const uint8_t* row = stg + (r * G + g) * KROWB;
      *reinterpret_cast<uint4*>(orow + g * HD) = *reinterpret_cast<const uint4*>(row + 16 * (cg ^ sw));
      *reinterpret_cast<uint4*>(orow + g * HD + HALF) =
          *reinterpret_cast<const uint4*>(row + 16 * ((cg + CPR / 2) ^ sw));
    }
  }
}

// ---------------------------------------------------------------------------
// Tied LM head with cross-entropy partials.  For a tile of rows and 128 vocab
// columns: the row maximum of the logits and the sum of exp(logit - max) over
// the tile, plus the label logit when the label falls in the tile.
// ---------------------------------------------------------------------------
constexpr int kVT = 128;   // vocab columns per tile

// fp32 activations: one thread per (row, column).
__global__ void __launch_bounds__(256) k_lmhead_f32(const float* x, const float* E, int64_t M,
                                                    int64_t d, int64_t V, const int32_t* labels,
                                                    float* pmax, float* psum, float* lab,
                                                    int64_t nvt) {
  __shared__ float red[2][4];
  const int64_t m = (int64_t)blockIdx.y * 2 + (threadIdx.x >> 7);
  const int64_t n = (int64_t)blockIdx.x * kVT + (threadIdx.x & 127);
  float logit = -INFINITY;
  if (m < M && n < V) {
    float acc = 0.0f;
    for (int64_t e = 0; e < d; ++e) acc = fmaf(x[m * d + e], E[n * d + e], acc);
    logit = acc;
    if (labels[m] == n) lab[m] = acc;
  }
  // per half-block (one row) reductions: 2 waves per row
  const int half = threadIdx.x >> 7, wv = (threadIdx.x >> 6) & 1;
  float mx = wmax(logit);
  if ((threadIdx.x & 63) == 0) red[half][wv] = mx;
  __syncthreads();
  mx = fmaxf(red[half][0], red[half][1]);
  __syncthreads();
  float e = (logit == -INFINITY) ? 0.0f : expf(logit - mx);
  e = wsum(e);
  if ((threadIdx.x & 63) == 0) red[half][2 + wv] = e;
  __syncthreads();
  if ((threadIdx.x & 127) == 0 && m < M) {
    pmax[m * nvt + blockIdx.x] = mx;
    psum[m * nvt + blockIdx.x] = red[half][2] + red[half][3];
  }
}

// bf16 activations and embedding: 256 x 256 tiles of 8 waves (128 x 64 per
// wave) of v_mfma_f32_32x32x16_bf16, K step 64 (128 bytes per row, 144-byte
// LDS rows), double-buffered LDS, XCD-grouped tile order.  Epilogue: per row,
// max and sum of exp over the tile's columns by lane shuffles (each row's 64
// columns of a wave live in 32 lanes x 2 registers), then the 4 waves along N
// are combined through LDS.
constexpr int kLmBK = 64;                  // bf16 elements per K step
constexpr int kLmStride = 2 * kLmBK + 16;  // bytes per LDS row
constexpr int kLmTile = 256;               // rows and vocab columns per block
// direct-load LM head: ring stages, stage width, waves along N (8 waves of 128 x 64; four
// waves of 128 x 128 measured 17% slower at the 2B shape)
constexpr int kLmDmaStages = 2, kLmDmaBK = 64, kLmDmaNWN = 4;

template <bool FULL>
__global__ void __launch_bounds__(512) k_lmhead_bf16(const uint16_t* __restrict__ x,
                                                     const uint16_t* __restrict__ E, int64_t M,
                                                     int64_t d, int64_t V,
                                                     const int32_t* __restrict__ labels,
                                                     float* pmax, float* psum, float* lab,
                                                     int64_t nvt) {
  constexpr int BM = kLmTile, BN = kLmTile, WM = 128, WN = 64, NT = 512;
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int CPR = 2 * kLmBK / 16;      // 16-byte chunks per row (8)
  constexpr int CH = BM * CPR / NT;        // chunks per thread per operand (4)
  constexpr int STAGE = (BM + BN) * kLmStride;
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * STAGE];
  __shared__ int32_t lbl[BM];

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm = wid / (BN / WN), wn = wid % (BN / WN);
  int64_t tm, tn;
  tile_of_block((M + BM - 1) / BM, nvt, tm, tn);
  const int64_t m0 = tm * BM, n0 = tn * BN;
  const int nk = (int)((d + kLmBK - 1) / kLmBK);
  for (int i = tid; i < BM; i += NT) lbl[i] = m0 + i < M ? labels[m0 + i] : -1;

  typedef uint32_t v4u __attribute__((ext_vector_type(4)));
  v4u ra[CH], rb[CH];
  const uint8_t* xa = reinterpret_cast<const uint8_t*>(x) + m0 * d * 2;
  const uint8_t* eb = reinterpret_cast<const uint8_t*>(E) + n0 * d * 2;
  auto gload = [&](int kt) __attribute__((always_inline)) {
    const int64_t kb0 = (int64_t)kt * kLmBK * 2;   // byte offset in a row
#pragma unroll
    for (int it = 0; it < CH; ++it) {
      const int c = tid + NT * it;
      const int row = c / CPR, col = c % CPR;
      const int64_t kb = kb0 + 16 * col;
      const bool kin = FULL || kb < d * 2;
      ra[it] = (kin && (FULL || m0 + row < M))
                   ? *reinterpret_cast<const v4u*>(xa + row * d * 2 + kb)
                   : v4u{0u, 0u, 0u, 0u};
      rb[it] = (kin && (FULL || n0 + row < V))
                   ? *reinterpret_cast<const v4u*>(eb + row * d * 2 + kb)
                   : v4u{0u, 0u, 0u, 0u};
    }
  };
  auto lstore = [&](int buf) __attribute__((always_inline)) {
    uint8_t* As = smem + buf * STAGE;
    uint8_t* Bs = As + BM * kLmStride;
#pragma unroll
    for (int it = 0; it < CH; ++it) {
      const int c = tid + NT * it;
      const int off = (c / CPR) * kLmStride + 16 * (c % CPR);
      *reinterpret_cast<v4u*>(As + off) = ra[it];
      *reinterpret_cast<v4u*>(Bs + off) = rb[it];
    }
  };

  v16f acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;

  gload(0);
  lstore(0);
  if (nk > 1) gload(1);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const uint8_t* As = smem + (kt & 1) * STAGE;
    const uint8_t* Bs = As + BM * kLmStride;
#pragma unroll
    for (int ks = 0; ks < 2 * kLmBK / 32; ++ks) {
      const int kb = 32 * ks + 16 * (lane >> 5);
      v8bf af[TM], bf[TN];
#pragma unroll
      for (int a = 0; a < TM; ++a)
        af[a] = __builtin_bit_cast(
            v8bf, *reinterpret_cast<const v4u*>(As + (wm * WM + a * 32 + (lane & 31)) * kLmStride + kb));
#pragma unroll
      for (int b = 0; b < TN; ++b)
        bf[b] = __builtin_bit_cast(
            v8bf, *reinterpret_cast<const v4u*>(Bs + (wn * WN + b * 32 + (lane & 31)) * kLmStride + kb));
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[a], bf[b], acc[a][b], 0, 0, 0);
    }
    if (kt + 1 < nk) {
      lstore((kt + 1) & 1);
      if (kt + 2 < nk) gload(kt + 2);
    }
    __syncthreads();
  }

  // ---- epilogue: row statistics of this tile ----
  float* red = reinterpret_cast<float*>(smem);     // [4 waves along N][BM][2]
  const float L2E = 1.4426950408889634f;
  bool colok[TN];
  int64_t col[TN];
#pragma unroll
  for (int b = 0; b < TN; ++b) {
    col[b] = n0 + wn * WN + b * 32 + (lane & 31);
    colok[b] = FULL || col[b] < V;
  }
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int li = wm * WM + a * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      float mx = -INFINITY;
#pragma unroll
      for (int b = 0; b < TN; ++b)
        if (colok[b]) mx = fmaxf(mx, acc[a][b][r]);
#pragma unroll
      for (int off = 1; off < 32; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
      float se = 0.0f;
      const int lb = lbl[li];
#pragma unroll
      for (int b = 0; b < TN; ++b)
        if (colok[b]) {
          se += __builtin_amdgcn_exp2f((acc[a][b][r] - mx) * L2E);
          if (col[b] == lb) lab[m0 + li] = acc[a][b][r];
        }
#pragma unroll
      for (int off = 1; off < 32; off <<= 1) se += __shfl_xor(se, off, 64);
      if ((lane & 31) == 0) {
        red[(wn * BM + li) * 2 + 0] = mx;
        red[(wn * BM + li) * 2 + 1] = se;
      }
    }
  __syncthreads();
  if (tid < BM && (FULL || m0 + tid < M)) {
    float mx = -INFINITY;
#pragma unroll
    for (int w = 0; w < BN / WN; ++w) mx = fmaxf(mx, red[(w * BM + tid) * 2]);
    float se = 0.0f;
#pragma unroll
    for (int w = 0; w < BN / WN; ++w) {
      const float mw = red[(w * BM + tid) * 2];
      if (mw != -INFINITY) se += red[(w * BM + tid) * 2 + 1] * __builtin_amdgcn_exp2f((mw - mx) * L2E);
    }
    pmax[(m0 + tid) * nvt + tn] = mx;
    psum[(m0 + tid) * nvt + tn] = se;
  }
}

// LM head + cross-entropy partials on full tiles with direct global -> LDS
// loads: 256 tokens x 256 vocabulary columns per block, 2 x NWN waves of 128
// tokens x 256 / NWN columns each, v_mfma_f32_32x32x16_bf16 with the
// embedding rows as the first operand, so the accumulator is the transpose
// of the logits: a lane owns one token and 16 of its columns per 32 x 32
// tile, and a token's max and sum of exp over the block's columns reduce in
// registers, across the two lane halves and, through LDS, across the 4 waves
// along the vocabulary.  Operands stream through STAGES stages of BK bf16
// columns (a stage row is 2 BK bytes); 16-byte chunk c of row r sits at
// chunk c ^ sw(r), so the fragment reads of 16 consecutive rows hit distinct
// banks.  K assignment: in sub-step ks, lane half h supplies chunk
// h * (2 BK / 32) + ks of its row for both operands.
// Requires M % 256 == 0, V % 256 == 0, d % BK == 0.
template <int STAGES, int BK, int NWN>
__global__ void __launch_bounds__(128 * NWN) k_lmhead_dma(const uint16_t* __restrict__ x,
                                                          const uint16_t* __restrict__ E, int64_t M,
                                                          int64_t d, int64_t V,
                                                          const int32_t* __restrict__ labels,
                                                          float* pmax, float* psum, float* lab,
                                                          int64_t nvt) {
  constexpr int BM = 256, BN = 256, WM = 128, WN = BN / NWN, NT = 128 * NWN;
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int ROWB = 2 * BK, CPR = ROWB / 16;   // bytes and 16-byte chunks per stage row
  constexpr int OPB = BM * ROWB;                  // bytes per operand per stage
  constexpr int KS = CPR / 2;                     // MFMA sub-steps per stage
  constexpr int IPW = BM * CPR / NT;              // loads per operand per wave per stage
  static_assert(CPR == 8 || CPR == 4, "stage width");
  static_assert(STAGES >= 2 && STAGES * 2 * OPB + BN / WN * BM * 8 <= 152 * 1024, "LDS");
  __shared__ __attribute__((aligned(1024))) uint8_t lds[STAGES * 2 * OPB];
  __shared__ float red[BN / WN][BM][2];           // per wave column: token max and sum of exp
  __shared__ int32_t lbl[BM];
  auto sw = [](int row) __attribute__((always_inline)) {
    return CPR == 8 ? ((row >> 1) & 7) : ((row >> 2) & 3);
  };

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm = wid / (BN / WN), wn = wid % (BN / WN);
  const int64_t ntiles = (M / BM) * nvt;
  const int nk = (int)(d / BK);

  // load j of wave w fills the 64 LDS chunks (w * IPW + j) * 64 .. + 63 of an operand:
  // RPL rows of CPR chunks.  The chunk swizzle of those rows depends on j only through
  // its parity, so two per-lane sources per operand serve every load (the rest of the
  // offset is wave-uniform).
  constexpr int RPL = 64 / CPR;                   // rows per 1 KB load
  static_assert(IPW % 2 == 0, "loads per wave");
  const uint8_t* asrc[2];
  const uint8_t* bsrc[2];
  // tile it of the grouped (XCD-aware) order: its origin and the load sources
  auto tile = [&](int64_t it, int64_t& m0, int64_t& n0) __attribute__((always_inline)) {
    int64_t tm, tn;
    tile_of_linear(xcd_linear(it, ntiles), M / BM, nvt, tm, tn);
    m0 = tm * BM;
    n0 = tn * BN;
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int row = (wid * IPW + p) * RPL + lane / CPR, lc = (lane % CPR) ^ sw(row);
      asrc[p] = reinterpret_cast<const uint8_t*>(x) + (m0 + row) * d * 2 + 16 * lc;
      bsrc[p] = reinterpret_cast<const uint8_t*>(E) + (n0 + row) * d * 2 + 16 * lc;
    }
  };
  const uint32_t wbase = __builtin_amdgcn_readfirstlane(wid) * IPW * 1024u;
  auto Ast = [&](int st) { return lds + st * 2 * OPB; };
  auto issue = [&](int kt, int st) __attribute__((always_inline)) {
    const int64_t koff = (int64_t)kt * ROWB;
    const uint32_t ab = lds_offset(Ast(st)) + wbase, bb = ab + OPB;
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const int64_t roff = (int64_t)(j & ~1) * RPL * d * 2 + koff;
      dma16(asrc[j & 1] + roff, ab + 1024u * j);
      dma16(bsrc[j & 1] + roff, bb + 1024u * j);
    }
  };

  typedef uint32_t v4u __attribute__((ext_vector_type(4)));
  const int h = lane >> 5;
  const int arow0 = wm * WM + (lane & 31), brow0 = wn * WN + (lane & 31);
  v16f acc[TM][TN];
  auto compute = [&](const uint8_t* As, const uint8_t* Bs) __attribute__((always_inline)) {
    v8bf af[2][TM], bfr[2][TN];
    auto frag = [&](int ks, int slot) __attribute__((always_inline)) {
      const int c = h * KS + ks;
#pragma unroll
      for (int a = 0; a < TM; ++a) {
        const int row = arow0 + 32 * a;
        af[slot][a] = __builtin_bit_cast(
            v8bf, *reinterpret_cast<const v4u*>(As + row * ROWB + 16 * (c ^ sw(row))));
      }
#pragma unroll
      for (int b = 0; b < TN; ++b) {
        const int row = brow0 + 32 * b;
        bfr[slot][b] = __builtin_bit_cast(
            v8bf, *reinterpret_cast<const v4u*>(Bs + row * ROWB + 16 * (c ^ sw(row))));
      }
    };
    frag(0, 0);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int cur = ks & 1;
      if (ks + 1 < KS) frag(ks + 1, cur ^ 1);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b)   // embedding rows first: acc holds logits^T
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[cur][b], af[cur][a], acc[a][b], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Blocks walk the tiles it = blockIdx.x, + gridDim.x, ...  The first stages of the next
  // tile are issued right after the last barrier of the current one (the ring is free
  // then), so their loads land while the current tile's epilogue runs.
  int64_t it = blockIdx.x;
  if (it >= ntiles) return;                       // whole block
  int64_t m0, n0;
  tile(it, m0, n0);
  for (int i = tid; i < BM; i += NT) lbl[i] = labels[m0 + i];
#pragma unroll
  for (int st = 0; st < STAGES - 1; ++st)
    if (st < nk) issue(st, st);
  while (true) {
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int b = 0; b < TN; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;
    // prologue: stages 0 .. STAGES-2 issued, stage 0 complete
    if (nk >= STAGES - 1) wait_vmcnt_le<(STAGES - 2) * 2 * IPW>(); else __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      const int st = kt % STAGES;
      const bool more = kt + STAGES - 1 < nk;
      if (more) issue(kt + STAGES - 1, (kt + STAGES - 1) % STAGES);   // the stage freed at kt-1
      compute(Ast(st), Ast(st) + OPB);
      if (more) wait_vmcnt_le<(STAGES - 2) * 2 * IPW>(); else __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
    }
    const int64_t cm0 = m0, cn0 = n0, ctn = cn0 / BN;
    const int64_t nit = it + gridDim.x;
    if (nit < ntiles) {                           // next tile's first stages
      tile(nit, m0, n0);
#pragma unroll
      for (int st = 0; st < STAGES - 1; ++st)
        if (st < nk) issue(st, st);
    }

    // ---- epilogue: per token, max and sum of exp over the block's 256 columns ----
    const float L2E = 1.4426950408889634f;
#pragma unroll
    for (int a = 0; a < TM; ++a) {
      const int li = wm * WM + 32 * a + (lane & 31);
      const int lb = lbl[li];
      float mx = -INFINITY;
#pragma unroll
      for (int b = 0; b < TN; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, acc[a][b][r]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      float se = 0.0f;
#pragma unroll
      for (int b = 0; b < TN; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          se += __builtin_amdgcn_exp2f((acc[a][b][r] - mx) * L2E);
          const int64_t col = cn0 + wn * WN + 32 * b + 8 * (r >> 2) + 4 * h + (r & 3);
          if (col == lb) lab[cm0 + li] = acc[a][b][r];
        }
      se += __shfl_xor(se, 32, 64);
      if (h == 0) {
        red[wn][li][0] = mx;
        red[wn][li][1] = se;
      }
    }
    __syncthreads();
    if (tid < BM) {
      float mx = -INFINITY;
#pragma unroll
      for (int w = 0; w < BN / WN; ++w) mx = fmaxf(mx, red[w][tid][0]);
      float se = 0.0f;
#pragma unroll
      for (int w = 0; w < BN / WN; ++w)
        se += red[w][tid][1] * __builtin_amdgcn_exp2f((red[w][tid][0] - mx) * L2E);
      pmax[(cm0 + tid) * nvt + ctn] = mx;
      psum[(cm0 + tid) * nvt + ctn] = se;
    }
    if (nit >= ntiles) break;
    it = nit;
    // the load sources again (computed afresh rather than held through the epilogue)
    int64_t itr = it;
    asm volatile("" : "+s"(itr));
    tile(itr, m0, n0);
    __syncthreads();                              // red and lbl read by every wave
    for (int i = tid; i < BM; i += NT) lbl[i] = labels[m0 + i];
  }
}

// Row loss = logsumexp - label logit; the last position of each sequence has
// no label (0).  One wave per row over the vocabulary-tile partials.
__global__ void __launch_bounds__(256) k_ce_combine(const float* pmax, const float* psum,
                                                    const float* lab, int64_t M, int64_t nvt, int S,
                                                    float* row_loss) {
  const int64_t m = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (m >= M) return;
  float mx = -INFINITY;
  for (int64_t t = lane; t < nvt; t += 64) mx = fmaxf(mx, pmax[m * nvt + t]);
  mx = wmax(mx);
  float s = 0.0f;
  for (int64_t t = lane; t < nvt; t += 64) {
    const float pm = pmax[m * nvt + t];
    if (pm != -INFINITY) s += psum[m * nvt + t] * expf(pm - mx);
  }
  s = wsum(s);
  if (lane == 0) {
    const bool labelled = (m % S) != S - 1;
    row_loss[m] = labelled ? (mx + logf(s)) - lab[m] : 0.0f;
  }
}

// Mean over the labelled positions, fp64 accumulation in a fixed order.
__global__ void __launch_bounds__(256) k_loss_mean(const float* row_loss, int64_t M, int64_t count,
                                                   float* out_f32, double* out_f64) {
  __shared__ double lds[256];
  double acc = 0.0;
  for (int64_t i = threadIdx.x; i < M; i += 256) acc += (double)row_loss[i];
  lds[threadIdx.x] = acc;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off) lds[threadIdx.x] += lds[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double mean = lds[0] / (double)count;
    if (out_f64) *out_f64 = mean;
    if (out_f32) *out_f32 = (float)mean;
  }
}

// Next-token label of every position (-1 at the last position of a sequence); an
// id outside [0, V) becomes label 0 and sets bit 8 of the deferred error word.
__global__ void k_labels(const int32_t* tok, int64_t M, int S, int64_t V, int32_t* labels,
                         int32_t* err) {
  const int64_t m = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (m >= M) return;
  int32_t t = -1;
  if ((m % S) != S - 1) {
    t = tok[m + 1];
    if (t < 0 || (int64_t)t >= V) {
      atomicOr(err, 8);
      t = 0;
    }
  }
  labels[m] = t;
}

}  // namespace tmz

// ===========================================================================
// Model runtime
// ===========================================================================
using namespace tmz;

struct termezo_model {
  termezo_ctx* ctx = nullptr;
  hipStream_t stream = nullptr;   // the context's stream, or the model's own (destroy never reads ctx)
  bool own_stream = false;        // forwards run on a stream of their own (ordered after the
                                  // context's work at entry, joined back by termezo_model_join)
  hipEvent_t ev_in = nullptr, ev_out = nullptr;
  bool use_snap = false;          // read the context's codes snapshot instead of its current codes
  termezo_model_config cfg{};
  const void* emb = nullptr;
  const void* normw = nullptr;    // RMSNorm weights [2 n_blocks + 1][d] (null: one)
  int hd = 0;
  int64_t cap_M = 0;
  int cap_S = 0;
  void *h = nullptr, *q = nullptr, *k = nullptr, *v = nullptr, *vt = nullptr, *attn = nullptr,
       *g = nullptr, *u = nullptr, *xf = nullptr;
  int8_t* xq = nullptr;
  float* xs = nullptr;
  int32_t* xrs = nullptr;                    // per-token sums of the quantised activations
  float *pmax = nullptr, *psum = nullptr, *lab = nullptr, *row = nullptr;
  int32_t* labels = nullptr;
  float *rope_c = nullptr, *rope_s = nullptr;
  double* loss64 = nullptr;
  float* loss32 = nullptr;
  // optional event timing of the matrix-core kernels (class 0: BitLinear
  // GEMM, 1: attention, 2: LM head + cross-entropy partials)
  struct Span {
    hipEvent_t a, b;
    int cls;
    double ops;
  };
  bool timing = false;
  std::vector<Span> spans;
  size_t used = 0;
};

namespace {

void mfree(void*& p) {
  if (p) (void)hipFree(p);
  p = nullptr;
}

int span_begin(termezo_model* m, int cls, double ops, hipStream_t s) {
  if (!m->timing) return -1;
  if (m->used == m->spans.size()) {
    termezo_model::Span sp{};
    if (hipEventCreate(&sp.a) != hipSuccess || hipEventCreate(&sp.b) != hipSuccess) return -1;
    m->spans.push_back(sp);
  }
  termezo_model::Span& sp = m->spans[m->used];
  sp.cls = cls;
  sp.ops = ops;
  if (hipEventRecord(sp.a, s) != hipSuccess) return -1;
  return (int)m->used++;
}

void span_end(termezo_model* m, int idx, hipStream_t s) {
  if (idx >= 0) (void)hipEventRecord(m->spans[idx].b, s);
}

// A span whose events the launch itself sets to its kernel's start and end (GEMMs).
LaunchEvents span_kernel(termezo_model* m, int cls, double ops) {
  LaunchEvents ev;
  if (!m->timing) return ev;
  if (m->used == m->spans.size()) {
    termezo_model::Span sp{};
    if (hipEventCreate(&sp.a) != hipSuccess || hipEventCreate(&sp.b) != hipSuccess) return ev;
    m->spans.push_back(sp);
  }
  termezo_model::Span& sp = m->spans[m->used++];
  sp.cls = cls;
  sp.ops = ops;
  ev.start = sp.a;
  ev.stop = sp.b;
  return ev;
}

void model_free_buffers(termezo_model* m) {
  mfree(m->h); mfree(m->q); mfree(m->k); mfree(m->v); mfree(m->vt); mfree(m->attn); mfree(m->g);
  mfree(m->u);
  mfree(m->xf);
  void* p;
  p = m->xq; mfree(p); m->xq = nullptr;
  p = m->xs; mfree(p); m->xs = nullptr;
  p = m->xrs; mfree(p); m->xrs = nullptr;
  p = m->pmax; mfree(p); m->pmax = nullptr;
  p = m->psum; mfree(p); m->psum = nullptr;
  p = m->lab; mfree(p); m->lab = nullptr;
  p = m->row; mfree(p); m->row = nullptr;
  p = m->labels; mfree(p); m->labels = nullptr;
  p = m->rope_c; mfree(p); m->rope_c = nullptr;
  p = m->rope_s; mfree(p); m->rope_s = nullptr;
  p = m->loss64; mfree(p); m->loss64 = nullptr;
  p = m->loss32; mfree(p); m->loss32 = nullptr;
  m->cap_M = 0;
  m->cap_S = 0;
}

termezo_status model_reserve(termezo_model* m, int64_t M, int S) {
  if (M <= m->cap_M && S == m->cap_S) return TERMEZO_OK;
  model_free_buffers(m);
  const termezo_model_config& c = m->cfg;
  const size_t es = c.act_dtype == TERMEZO_BF16 ? 2 : 4;
  const int64_t dq = (int64_t)c.n_heads * m->hd, dkv = (int64_t)c.n_kv_heads * m->hd;
  const int64_t kmax = std::max<int64_t>(std::max<int64_t>(c.d_model, dq), c.d_ffn);
  const int64_t nvt = c.act_dtype == TERMEZO_BF16 ? (c.vocab + kLmTile - 1) / kLmTile
                                                  : (c.vocab + kVT - 1) / kVT;
  hipError_t e = hipSuccess;
  auto A = [&](void** p, size_t bytes) {
    if (e == hipSuccess) e = hipMalloc(p, bytes > 0 ? bytes : 1);
  };
  A(&m->h, M * c.d_model * es);
  A(&m->q, M * dq * es);
  A(&m->k, M * dkv * es);
  A(&m->v, M * dkv * es);
  A(&m->vt, M * dkv * es);
  A(&m->attn, M * dq * es);
  A(&m->g, M * c.d_ffn * es);
  A(&m->u, M * c.d_ffn * es);
  A(&m->xf, M * c.d_model * es);
  A((void**)&m->xq, M * kmax);
  A((void**)&m->xs, M * 4);
  A((void**)&m->xrs, M * 4);
  A((void**)&m->pmax, M * nvt * 4);
  A((void**)&m->psum, M * nvt * 4);
  A((void**)&m->lab, M * 4);
  A((void**)&m->row, M * 4);
  A((void**)&m->labels, M * 4);
  A((void**)&m->rope_c, (size_t)S * (m->hd / 2) * 4);
  A((void**)&m->rope_s, (size_t)S * (m->hd / 2) * 4);
  A((void**)&m->loss64, 8);
  A((void**)&m->loss32, 4);
  if (e != hipSuccess) {
    model_free_buffers(m);
    return e == hipErrorOutOfMemory ? TERMEZO_ERR_OOM : TERMEZO_ERR_DEVICE;
  }
  // rotary table: angle p * base^(-2i/hd), evaluated in fp64 and rounded to fp32
  const int half = m->hd / 2;
  std::vector<float> cs((size_t)S * half), sn((size_t)S * half);
  for (int p = 0; p < S; ++p)
    for (int i = 0; i < half; ++i) {
      const double ang = (double)p * std::pow((double)c.rope_base, -2.0 * i / (double)m->hd);
      cs[(size_t)p * half + i] = (float)std::cos(ang);
      sn[(size_t)p * half + i] = (float)std::sin(ang);
    }
  e = hipMemcpy(m->rope_c, cs.data(), cs.size() * 4, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(m->rope_s, sn.data(), sn.size() * 4, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    model_free_buffers(m);
    return TERMEZO_ERR_DEVICE;
  }
  m->cap_M = M;
  m->cap_S = S;
  return TERMEZO_OK;
}

hipError_t run_attention(termezo_model* m, int B, int S, hipStream_t st) {
  const termezo_model_config& c = m->cfg;
  const int64_t M = (int64_t)B * S;
  if (c.act_dtype == TERMEZO_F32) {
    hipLaunchKernelGGL(k_attn_f32, dim3((unsigned)M, c.n_heads), dim3(256), S * sizeof(float), st,
                       (const float*)m->q, (const float*)m->k, (const float*)m->v, (float*)m->attn,
                       S, c.n_heads, c.n_kv_heads, m->hd, 1.0f / std::sqrt((float)m->hd));
    return hipGetLastError();
  }
  const float sl2 = (float)(1.4426950408889634 / std::sqrt((double)m->hd));
  dim3 pgrid((unsigned)((S + 63) / 64), (unsigned)(B * c.n_kv_heads));
  dim3 grid((unsigned)((S + 127) / 128), c.n_heads, B);
#define TMZ_ATTN(HDV)                                                                        \
  hipLaunchKernelGGL(k_kv_prep<HDV>, pgrid, dim3(256), 0, st, (uint16_t*)m->k,                  \
                     (const uint16_t*)m->v, (uint16_t*)m->vt, S, c.n_kv_heads, m->rope_c,      \
                     m->rope_s);                                                              \
  hipLaunchKernelGGL(k_attn_bf16<HDV>, grid, dim3(512), 0, st, (const uint16_t*)m->q,          \
                     (const uint16_t*)m->k, (const uint16_t*)m->vt, (uint16_t*)m->attn, S,     \
                     c.n_heads, c.n_kv_heads, sl2, m->rope_c, m->rope_s)
  const int G = c.n_heads / c.n_kv_heads;
  const bool gqa = (m->hd == 64 || m->hd == 96 || m->hd == 128) &&
                   (G == 1 || G == 2 || G == 4 || G == 8) &&
                   S % 64 == 0 && S % (256 / G) == 0;
  if (gqa) {
    const int nbh = B * c.n_kv_heads, nqt = S / (256 / G);
    if (m->hd == 128)
      hipLaunchKernelGGL(k_kv_prep<128>, pgrid, dim3(256), 0, st, (uint16_t*)m->k,
                         (const uint16_t*)m->v, (uint16_t*)m->vt, S, c.n_kv_heads, m->rope_c,
                         m->rope_s);
    else if (m->hd == 96)
      hipLaunchKernelGGL(k_kv_prep<96>, pgrid, dim3(256), 0, st, (uint16_t*)m->k,
                         (const uint16_t*)m->v, (uint16_t*)m->vt, S, c.n_kv_heads, m->rope_c,
                         m->rope_s);
    else
      hipLaunchKernelGGL(k_kv_prep<64>, pgrid, dim3(256), 0, st, (uint16_t*)m->k,
                         (const uint16_t*)m->v, (uint16_t*)m->vt, S, c.n_kv_heads, m->rope_c,
                         m->rope_s);
#define TMZ_GQA(HDV, GV)                                                                      \
  hipLaunchKernelGGL((k_attn_gqa<HDV, GV>), dim3((unsigned)(nqt * nbh)), dim3(512), 0, st,      \
                     (const uint16_t*)m->q, (const uint16_t*)m->k, (const uint16_t*)m->vt,     \
                     (uint16_t*)m->attn, S, c.n_kv_heads, nbh, nqt, sl2, m->rope_c, m->rope_s)
    switch (m->hd * 16 + G) {
      case 128 * 16 + 1: TMZ_GQA(128, 1); break;
      case 128 * 16 + 2: TMZ_GQA(128, 2); break;
      case 128 * 16 + 4: TMZ_GQA(128, 4); break;
      case 128 * 16 + 8: TMZ_GQA(128, 8); break;
      case 96 * 16 + 1: TMZ_GQA(96, 1); break;
      case 96 * 16 + 2: TMZ_GQA(96, 2); break;
      case 96 * 16 + 4: TMZ_GQA(96, 4); break;
      case 96 * 16 + 8: TMZ_GQA(96, 8); break;
      case 64 * 16 + 1: TMZ_GQA(64, 1); break;
      case 64 * 16 + 2: TMZ_GQA(64, 2); break;
      case 64 * 16 + 4: TMZ_GQA(64, 4); break;
      case 64 * 16 + 8: TMZ_GQA(64, 8); break;
      default: return hipErrorInvalidValue;
    }
#undef TMZ_GQA
    return hipGetLastError();
  }
  switch (m->hd) {
    case 64: TMZ_ATTN(64); break;
    case 96: TMZ_ATTN(96); break;
    case 128: TMZ_ATTN(128); break;
    default: return hipErrorInvalidValue;
  }
#undef TMZ_ATTN
  return hipGetLastError();
}

}  // namespace

extern "C" {

termezo_status termezo_model_create(termezo_ctx* ctx, const termezo_model_config* cfg,
                                    const void* embedding, termezo_model** out) {
  if (!out) return TERMEZO_ERR_INVALID_ARG;
  *out = nullptr;
  if (!ctx || !cfg || !embedding) return TERMEZO_ERR_INVALID_ARG;
  const termezo_model_config& c = *cfg;
  if (c.n_blocks <= 0 || c.d_model <= 0 || c.n_heads <= 0 || c.n_kv_heads <= 0 ||
      c.d_ffn <= 0 || c.vocab <= 0 || c.d_model % c.n_heads != 0 || c.n_heads % c.n_kv_heads != 0)
    return TERMEZO_ERR_INVALID_ARG;
  if (c.act_dtype != TERMEZO_F32 && c.act_dtype != TERMEZO_BF16) return TERMEZO_ERR_INVALID_ARG;
  if (!(c.norm_eps > 0.0f) || !(c.rope_base > 1.0f)) return TERMEZO_ERR_INVALID_ARG;
  const int hd = c.d_model / c.n_heads;
  if (hd % 2 != 0 || c.d_model % 16 != 0 || c.d_ffn % 16 != 0) return TERMEZO_ERR_INVALID_ARG;
  if (c.act_dtype == TERMEZO_BF16 && hd != 64 && hd != 96 && hd != 128)
    return TERMEZO_ERR_INVALID_ARG;
  if (std::max(c.d_model, c.d_ffn) > 64 * 8 * kRowChunks || (c.d_model / c.n_heads) % 16 != 0)
    return TERMEZO_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(embedding) & 15u) != 0) return TERMEZO_ERR_INVALID_ARG;
  if (ctx->L != 7 * c.n_blocks) return TERMEZO_ERR_INVALID_ARG;
  const int64_t dq = (int64_t)c.n_heads * hd, dkv = (int64_t)c.n_kv_heads * hd;
  const int64_t shp[7][2] = {{dq, c.d_model}, {dkv, c.d_model}, {dkv, c.d_model}, {c.d_model, dq},
                             {c.d_ffn, c.d_model}, {c.d_ffn, c.d_model}, {c.d_model, c.d_ffn}};
  for (int l = 0; l < ctx->L; ++l)
    if (ctx->layers[l].d_out != shp[l % 7][0] || ctx->layers[l].d_in != shp[l % 7][1])
      return TERMEZO_ERR_INVALID_ARG;
  termezo_model* m = new (std::nothrow) termezo_model();
  if (!m) return TERMEZO_ERR_OOM;
  m->ctx = ctx;
  m->stream = ctx->stream;
  m->cfg = c;
  m->emb = embedding;
  m->hd = hd;
  *out = m;
  return TERMEZO_OK;
}

termezo_status termezo_model_set_timing(termezo_model* m, int32_t enable) {
  if (!m) return TERMEZO_ERR_INVALID_ARG;
  if (hipStreamSynchronize(m->stream) != hipSuccess) return TERMEZO_ERR_DEVICE;
  m->timing = enable != 0;
  m->used = 0;
  return TERMEZO_OK;
}

termezo_status termezo_model_timing(termezo_model* m, int32_t cls, double* ms, int64_t* launches,
                                    double* ops) {
  if (!m || cls < 0 || cls > 2) return TERMEZO_ERR_INVALID_ARG;
  if (hipStreamSynchronize(m->stream) != hipSuccess) return TERMEZO_ERR_DEVICE;
  double t = 0.0, o = 0.0;
  int64_t n = 0;
  for (size_t i = 0; i < m->used; ++i) {
    const termezo_model::Span& sp = m->spans[i];
    if (sp.cls != cls) continue;
    float e = 0.0f;
    if (hipEventElapsedTime(&e, sp.a, sp.b) != hipSuccess) return TERMEZO_ERR_DEVICE;
    t += e;
    o += sp.ops;
    ++n;
  }
  if (ms) *ms = t;
  if (launches) *launches = n;
  if (ops) *ops = o;
  return TERMEZO_OK;
}

termezo_status termezo_model_set_norm_weights(termezo_model* m, const void* norm_weights) {
  if (!m) return TERMEZO_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(norm_weights) & 15u) != 0) {
    m->ctx->last_error = "model_set_norm_weights: pointer must be 16-byte aligned";
    return TERMEZO_ERR_INVALID_ARG;
  }
  m->normw = norm_weights;
  return TERMEZO_OK;
}

void termezo_model_destroy(termezo_model* m) {
  if (!m) return;
  (void)hipStreamSynchronize(m->stream);
  for (auto& sp : m->spans) {
    (void)hipEventDestroy(sp.a);
    (void)hipEventDestroy(sp.b);
  }
  if (m->ev_in) (void)hipEventDestroy(m->ev_in);
  if (m->ev_out) (void)hipEventDestroy(m->ev_out);
  model_free_buffers(m);
  delete m;
}

termezo_status termezo_model_set_stream(termezo_model* m, void* hip_stream) {
  if (!m) return TERMEZO_ERR_INVALID_ARG;
  termezo_ctx* c = m->ctx;
  hipStream_t s = hip_stream ? static_cast<hipStream_t>(hip_stream) : c->stream;
  if (s != c->stream && !m->ev_in) {
    if (hipEventCreateWithFlags(&m->ev_in, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&m->ev_out, hipEventDisableTiming) != hipSuccess) {
      c->last_error = "model_set_stream: event creation";
      return TERMEZO_ERR_DEVICE;
    }
  }
  if (hipStreamSynchronize(m->stream) != hipSuccess) return TERMEZO_ERR_DEVICE;
  m->stream = s;
  m->own_stream = s != c->stream;
  return TERMEZO_OK;
}

termezo_status termezo_model_use_snapshot(termezo_model* m, int32_t on) {
  if (!m) return TERMEZO_ERR_INVALID_ARG;
  m->use_snap = on != 0;
  return TERMEZO_OK;
}

termezo_status termezo_model_join(termezo_model* m) {
  if (!m) return TERMEZO_ERR_INVALID_ARG;
  if (!m->own_stream) return TERMEZO_OK;
  termezo_ctx* c = m->ctx;
  if (hipEventRecord(m->ev_out, m->stream) != hipSuccess ||
      hipStreamWaitEvent(c->stream, m->ev_out, 0) != hipSuccess) {
    c->last_error = "model_join: event record / wait";
    return TERMEZO_ERR_DEVICE;
  }
  return TERMEZO_OK;
}

termezo_status termezo_model_loss(termezo_model* m, const int32_t* tokens, int32_t batch,
                                  int32_t seq, float* loss_dev, float* row_loss_dev,
                                  float* loss_host) {
  if (!m || !tokens || batch <= 0 || seq < 2) return TERMEZO_ERR_INVALID_ARG;
  termezo_ctx* c = m->ctx;
  if (m->use_snap ? !c->snap_valid : !c->codes_valid) {
    c->last_error = m->use_snap ? "model_loss: no codes snapshot" :
                                  "model_loss: no current codes (perturb first)";
    return TERMEZO_ERR_STATE;
  }
  const termezo_model_config& cf = m->cfg;
  const int64_t M = (int64_t)batch * seq;
  termezo_status st = model_reserve(m, M, seq);
  if (st != TERMEZO_OK) return st;
  hipStream_t s = m->stream;
  if (m->own_stream &&   // everything queued on the context's stream so far comes first
      (hipEventRecord(m->ev_in, c->stream) != hipSuccess ||
       hipStreamWaitEvent(s, m->ev_in, 0) != hipSuccess)) {
    c->last_error = "model_loss: event record / wait";
    return TERMEZO_ERR_DEVICE;
  }
  const uint32_t* codes = m->use_snap ? c->d_codes_snap : c->d_codes;
  const float* betas = m->use_snap ? c->d_beta_snap : c->d_beta_cur;
  const bool bf = cf.act_dtype == TERMEZO_BF16;
  // full-precision parameters: a registered theta tensor is read at its current
  // (possibly perturbed) values
  auto current = [&](const void* p) -> const void* {
    if (!p || c->theta_sign == 0) return p;
    for (const ThetaHost& t : c->theta)
      if (t.data == p) return c->theta_sign > 0 ? t.plus : t.minus;
    return p;
  };
  const void* emb = current(m->emb);
  const void* nrm = current(m->normw);
  const int64_t d = cf.d_model, F = cf.d_ffn, dq = (int64_t)cf.n_heads * m->hd,
                dkv = (int64_t)cf.n_kv_heads * m->hd;
  const int64_t nvt = bf ? (cf.vocab + kLmTile - 1) / kLmTile : (cf.vocab + kVT - 1) / kVT;
  hipError_t e = hipSuccess;
  auto chk = [&](hipError_t x) {
    if (e == hipSuccess) e = x;
  };
  const termezo_dtype adt = cf.act_dtype;

  if (bf)
    hipLaunchKernelGGL(k_embed<uint16_t>, dim3((unsigned)M), dim3(256), 0, s, tokens,
                       (const uint16_t*)emb, d, (int64_t)cf.vocab, (uint16_t*)m->h, c->d_err);
  else
    hipLaunchKernelGGL(k_embed<float>, dim3((unsigned)M), dim3(256), 0, s, tokens,
                       (const float*)emb, d, (int64_t)cf.vocab, (float*)m->h, c->d_err);
  chk(hipGetLastError());
  hipLaunchKernelGGL(k_labels, dim3((unsigned)((M + 255) / 256)), dim3(256), 0, s, tokens, M, seq,
                     (int64_t)cf.vocab, m->labels, c->d_err);
  const unsigned rowg = (unsigned)((M + 3) / 4);
  // RMSNorm (weight row wr of the norm weights, one when there are none), then
  // the quantiser, or stored (the LM-head input)
  auto rmsq = [&](int8_t* xq, float* xs, void* xf, int wr) {
#define TMZ_NORM(T, MD, W)                                                                   \
  row_launch<MD, T, W>(rowg, s, (const T*)m->h,                                              \
                       nrm ? (const T*)nrm + (int64_t)wr * d : (const T*)nullptr, M, d,      \
                       cf.norm_eps, xq, xs, m->xrs, (T*)xf, c->n_cu)
    if (bf) {
      if (xf) {
        if (nrm) TMZ_NORM(uint16_t, kRowNormStore, true); else TMZ_NORM(uint16_t, kRowNormStore, false);
      } else {
        if (nrm) TMZ_NORM(uint16_t, kRowNormQuant, true); else TMZ_NORM(uint16_t, kRowNormQuant, false);
      }
    } else {
      if (xf) {
        if (nrm) TMZ_NORM(float, kRowNormStore, true); else TMZ_NORM(float, kRowNormStore, false);
      } else {
        if (nrm) TMZ_NORM(float, kRowNormQuant, true); else TMZ_NORM(float, kRowNormQuant, false);
      }
    }
#undef TMZ_NORM
    chk(hipGetLastError());
  };
  for (int blk = 0; blk < cf.n_blocks; ++blk) {
    const int l0 = 7 * blk;
    const LayerHost* Ls = &c->layers[l0];
    // attention sub-block
    rmsq(m->xq, m->xs, nullptr, 2 * blk);
    GemmOut o3 = {};
    o3.nseg = 3;
    o3.y[0] = m->q; o3.ld[0] = dq; o3.beta[0] = betas + l0;
    o3.y[1] = m->k; o3.ld[1] = dkv; o3.beta[1] = betas + l0 + 1;
    o3.y[2] = m->v; o3.ld[2] = dkv; o3.beta[2] = betas + l0 + 2;
    o3.nstart[0] = 0; o3.nstart[1] = dq; o3.nstart[2] = dq + dkv; o3.nstart[3] = dq + 2 * dkv;
    chk(launch_gemm_i8(m->xq, m->xs, m->xrs, codes + Ls[0].code_off, M, d, dq + 2 * dkv, o3, adt,
                       kGemmStore, nullptr, c->n_cu, s,
                       span_kernel(m, 0, 2.0 * M * d * (dq + 2 * dkv))));
    if (!bf) {   // bf16: the rotation is applied inside the attention kernel
      const unsigned rg =
          (unsigned)std::min<int64_t>(8192, (M * cf.n_heads * (m->hd / 2) + 255) / 256);
      hipLaunchKernelGGL(k_rope<float>, dim3(rg), dim3(256), 0, s, (float*)m->q, M, cf.n_heads,
                         m->hd, seq, m->rope_c, m->rope_s);
      hipLaunchKernelGGL(k_rope<float>, dim3(rg), dim3(256), 0, s, (float*)m->k, M,
                         cf.n_kv_heads, m->hd, seq, m->rope_c, m->rope_s);
      chk(hipGetLastError());
    }
    const int sp = span_begin(m, 1, 4.0 * batch * cf.n_heads * m->hd * (0.5 * seq * (seq + 1.0)), s);
    chk(run_attention(m, batch, seq, s));
    span_end(m, sp, s);
    if (bf)
      row_launch<kRowQuant, uint16_t>(rowg, s, (const uint16_t*)m->attn, (const uint16_t*)nullptr,
                                      M, dq, 0.0f, m->xq, m->xs, m->xrs, (uint16_t*)nullptr,
                                      c->n_cu);
    else
      row_launch<kRowQuant, float>(rowg, s, (const float*)m->attn, (const float*)nullptr, M, dq,
                                   0.0f, m->xq, m->xs, m->xrs, (float*)nullptr);
    chk(hipGetLastError());
    GemmOut oo = {};
    oo.nseg = 1;
    oo.y[0] = m->h; oo.ld[0] = d; oo.beta[0] = betas + l0 + 3;
    oo.nstart[0] = 0; oo.nstart[1] = d;
    chk(launch_gemm_i8(m->xq, m->xs, m->xrs, codes + Ls[3].code_off, M, dq, d, oo, adt, kGemmResidual,
                       nullptr, c->n_cu, s,
                       span_kernel(m, 0, 2.0 * M * dq * d)));
    // MLP sub-block
    rmsq(m->xq, m->xs, nullptr, 2 * blk + 1);
    GemmOut o2 = {};
    o2.nseg = 2;
    o2.y[0] = m->g; o2.ld[0] = F; o2.beta[0] = betas + l0 + 4;
    o2.y[1] = m->u; o2.ld[1] = F; o2.beta[1] = betas + l0 + 5;
    o2.nstart[0] = 0; o2.nstart[1] = F; o2.nstart[2] = 2 * F;
    // gate|up with the SwiGLU in the epilogue where the full-tile path applies (the
    // product lands in g), else the two projections and the SwiGLU row kernel
    const bool fused = gemm_swiglu_ok(M, d, 2 * F, adt);
    chk(launch_gemm_i8(m->xq, m->xs, m->xrs, codes + Ls[4].code_off, M, d, 2 * F, o2, adt,
                       fused ? kGemmSwiGLU : kGemmStore, nullptr, c->n_cu, s,
                       span_kernel(m, 0, 2.0 * M * d * 2 * F)));
    if (fused)
      row_launch<kRowQuant, uint16_t>(rowg, s, (const uint16_t*)m->g, (const uint16_t*)nullptr, M,
                                      F, 0.0f, m->xq, m->xs, m->xrs, (uint16_t*)nullptr, c->n_cu);
    else if (bf)
      row_launch<kRowSwiGLU, uint16_t>(rowg, s, (const uint16_t*)m->g, (const uint16_t*)m->u, M,
                                       F, 0.0f, m->xq, m->xs, m->xrs, (uint16_t*)nullptr);
    else
      row_launch<kRowSwiGLU, float>(rowg, s, (const float*)m->g, (const float*)m->u, M, F, 0.0f,
                                    m->xq, m->xs, m->xrs, (float*)nullptr);
    chk(hipGetLastError());
    GemmOut od = {};
    od.nseg = 1;
    od.y[0] = m->h; od.ld[0] = d; od.beta[0] = betas + l0 + 6;
    od.nstart[0] = 0; od.nstart[1] = d;
    chk(launch_gemm_i8(m->xq, m->xs, m->xrs, codes + Ls[6].code_off, M, F, d, od, adt, kGemmResidual,
                       nullptr, c->n_cu, s,
                       span_kernel(m, 0, 2.0 * M * F * d)));
  }
  rmsq(nullptr, nullptr, m->xf, 2 * cf.n_blocks);
  const LaunchEvents ev_lm = span_kernel(m, 2, 2.0 * M * d * cf.vocab);
  if (bf) {
    const unsigned nb = (unsigned)(nvt * ((M + kLmTile - 1) / kLmTile));
    // the direct-load kernel walks its tiles with one block per compute unit
    const unsigned nbp = c->n_cu > 0 && nb > (unsigned)c->n_cu ? (unsigned)c->n_cu : nb;
    if (M % kLmTile == 0 && cf.vocab % kLmTile == 0 && d % 64 == 0)
      hipExtLaunchKernelGGL((k_lmhead_dma<kLmDmaStages, kLmDmaBK, kLmDmaNWN>), dim3(nbp),
                            dim3(128 * kLmDmaNWN), 0, s, ev_lm.start, ev_lm.stop, 0,
                            (const uint16_t*)m->xf, (const uint16_t*)emb, M, d, (int64_t)cf.vocab,
                            m->labels, m->pmax, m->psum, m->lab, nvt);
    else
      hipExtLaunchKernelGGL(k_lmhead_bf16<false>, dim3(nb), dim3(512), 0, s, ev_lm.start,
                            ev_lm.stop, 0, (const uint16_t*)m->xf, (const uint16_t*)emb, M, d,
                            (int64_t)cf.vocab, m->labels, m->pmax, m->psum, m->lab, nvt);
  }
  else
    hipExtLaunchKernelGGL(k_lmhead_f32, dim3((unsigned)nvt, (unsigned)((M + 1) / 2)), dim3(256), 0,
                          s, ev_lm.start, ev_lm.stop, 0, (const float*)m->xf, (const float*)emb, M,
                          d, (int64_t)cf.vocab, m->labels, m->pmax, m->psum, m->lab, nvt);
  chk(hipGetLastError());
  float* rows = row_loss_dev ? row_loss_dev : m->row;
  hipLaunchKernelGGL(k_ce_combine, dim3((unsigned)((M + 3) / 4)), dim3(256), 0, s, m->pmax,
                     m->psum, m->lab, M, nvt, seq, rows);
  hipLaunchKernelGGL(k_loss_mean, dim3(1), dim3(256), 0, s, rows, M,
                     (int64_t)batch * (seq - 1), loss_dev ? loss_dev : m->loss32, m->loss64);
  chk(hipGetLastError());
  if (e != hipSuccess) {
    c->last_error = std::string("model_loss: ") + hipGetErrorString(e);
    return e == hipErrorOutOfMemory ? TERMEZO_ERR_OOM : TERMEZO_ERR_DEVICE;
  }
  if (loss_host) {
    double v = 0.0;
    if (hipMemcpyAsync(&v, m->loss64, 8, hipMemcpyDeviceToHost, s) != hipSuccess)
      return TERMEZO_ERR_DEVICE;
    if (m->own_stream && hipStreamSynchronize(s) != hipSuccess) return TERMEZO_ERR_DEVICE;
    const termezo_status ds = termezo_sync(c);     // waits; reports deferred errors
    if (ds != TERMEZO_OK) return ds;
    *loss_host = (float)v;
  }
  return TERMEZO_OK;
}

}  // extern "C"
