// BitLinear forward on gfx950: per-token absmax int8 activation quantisation
// and the int8 x ternary contraction on the int8 matrix cores
// (v_mfma_i32_32x32x32_i8), int32 accumulation, per-row rescale epilogue.
#include "tmz_device.h"
#include "tmz_internal.h"

namespace tmz {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

// ---------------------------------------------------------------------------
// Activation quantisation, one block per token row:
//   a = max |x|, s = 127 / max(a, 1e-5), x_q = clamp(rne(x s), -128, 127).
// ---------------------------------------------------------------------------
__device__ __forceinline__ void load4(const float* p, float v[4]) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
}
__device__ __forceinline__ void load4(const uint16_t* p, float v[4]) {
  const uint2 a = *reinterpret_cast<const uint2*>(p);
  v[0] = __uint_as_float(a.x << 16);
  v[1] = __uint_as_float(a.x & 0xFFFF0000u);
  v[2] = __uint_as_float(a.y << 16);
  v[3] = __uint_as_float(a.y & 0xFFFF0000u);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

__device__ __forceinline__ int32_t quant_byte(float x, float s) {
  float q = __builtin_rintf(x * s);
  q = fminf(fmaxf(q, -128.0f), 127.0f);
  return (int32_t)q;
}

template <typename T>
__global__ void __launch_bounds__(256) k_act_quant(const T* __restrict__ x, int64_t K,
                                                   int8_t* __restrict__ xq, float* __restrict__ s) {
  __shared__ float red[4];
  const int64_t m = blockIdx.x;
  const T* row = x + m * K;
  float a = 0.0f;
  for (int64_t k = (int64_t)threadIdx.x * 4; k < K; k += 256 * 4) {
    float v[4];
    load4(row + k, v);
    a = fmaxf(a, fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
  }
  a = wave_max(a);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = a;
  __syncthreads();
  a = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  const float sc = __fdiv_rn(127.0f, fmaxf(a, 1e-5f));
  if (threadIdx.x == 0) s[m] = sc;
  uint32_t* out = reinterpret_cast<uint32_t*>(xq + m * K);
  for (int64_t k = (int64_t)threadIdx.x * 4; k < K; k += 256 * 4) {
    float v[4];
    load4(row + k, v);
    const uint32_t b0 = (uint32_t)quant_byte(v[0], sc) & 0xFFu;
    const uint32_t b1 = (uint32_t)quant_byte(v[1], sc) & 0xFFu;
    const uint32_t b2 = (uint32_t)quant_byte(v[2], sc) & 0xFFu;
    const uint32_t b3 = (uint32_t)quant_byte(v[3], sc) & 0xFFu;
    out[k / 4] = b0 | (b1 << 8) | (b2 << 16) | (b3 << 24);
  }
}

// ---------------------------------------------------------------------------
// Tiled int8 GEMM  acc = x_q c^T  with 2-bit codes unpacked into LDS.
// Block tile 128 x 128 x 64, 4 waves in a 2 x 2 grid, each wave 64 x 64 made
// of 2 x 2 tiles of v_mfma_i32_32x32x32_i8.  Within each 32-wide K step,
// lane l supplies the 16 bytes at k = 16 (l / 32) .. +15 of row l % 32 for
// both operands, so A and B agree on the K assignment.
// Accumulator layout (32 x 32, 16 values per lane): column l % 32,
// row 8 (r / 4) + 4 (l / 32) + (r % 4).
// ---------------------------------------------------------------------------
constexpr int kBM = 128, kBN = 128, kBK = 64;
constexpr int kLdsStride = 80;   // bytes per LDS row (64 data + 16 pad)

__device__ __forceinline__ float load_act(const float* p) { return *p; }
__device__ __forceinline__ float load_act(const uint16_t* p) { return bf16_to_f32(*p); }
__device__ __forceinline__ void store_act(float* p, float v) { *p = v; }
__device__ __forceinline__ void store_act(uint16_t* p, float v) { *p = f32_to_bf16_rne(v); }
__device__ __forceinline__ float round_act(const float*, float v) { return v; }
__device__ __forceinline__ float round_act(const uint16_t*, float v) {
  return bf16_to_f32(f32_to_bf16_rne(v));
}

template <typename TY, int MODE>
__global__ void __launch_bounds__(256) k_gemm_i8(const int8_t* __restrict__ xq,
                                                 const float* __restrict__ s,
                                                 const uint32_t* __restrict__ codes, int64_t M,
                                                 int64_t K, int64_t N, GemmOut out,
                                                 int32_t* __restrict__ acc_out) {
  __shared__ __attribute__((aligned(16))) int8_t As[kBM * kLdsStride];
  __shared__ __attribute__((aligned(16))) int8_t Bs[kBN * kLdsStride];
  __shared__ float rrow[kMaxSeg][kBM];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wid = tid >> 6;
  const int wm = wid >> 1, wn = wid & 1;
  const int64_t m0 = (int64_t)blockIdx.y * kBM, n0 = (int64_t)blockIdx.x * kBN;
  const int64_t KW = K / 16;  // code words per row

  for (int i = tid; i < kMaxSeg * kBM; i += 256) {
    const int sg = i / kBM, r = i % kBM;
    const int64_t m = m0 + r;
    rrow[sg][r] = (sg < out.nseg && m < M) ? __fdiv_rn(*out.beta[sg], s[m]) : 0.0f;
  }

  v16i acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0;

  for (int64_t k0 = 0; k0 < K; k0 += kBK) {
    // ---- stage A: 128 rows x 64 bytes ----
#pragma unroll
    for (int it = 0; it < 2; ++it) {
      const int c = tid + 256 * it;
      const int row = c >> 2, c16 = c & 3;
      const int64_t m = m0 + row, k = k0 + 16 * c16;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (m < M && k < K) v = *reinterpret_cast<const uint4*>(xq + m * K + k);
      *reinterpret_cast<uint4*>(As + row * kLdsStride + 16 * c16) = v;
    }
    // ---- stage B: 128 rows x 4 code words, unpacked to int8 ----
#pragma unroll
    for (int it = 0; it < 2; ++it) {
      const int c = tid + 256 * it;
      const int row = c >> 2, wi = c & 3;
      const int64_t n = n0 + row, kw = k0 / 16 + wi;
      uint32_t word = 0;
      if (n < N && kw < KW) word = codes[n * KW + kw];
      uint4 v;
      v.x = unpack_group(word, 0);
      v.y = unpack_group(word, 1);
      v.z = unpack_group(word, 2);
      v.w = unpack_group(word, 3);
      *reinterpret_cast<uint4*>(Bs + row * kLdsStride + 16 * wi) = v;
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int kb = 32 * ks + 16 * (lane >> 5);
      v4i af[2], bf[2];
#pragma unroll
      for (int a = 0; a < 2; ++a) {
        const int row = wm * 64 + a * 32 + (lane & 31);
        af[a] = *reinterpret_cast<const v4i*>(As + row * kLdsStride + kb);
      }
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int row = wn * 64 + b * 32 + (lane & 31);
        bf[b] = *reinterpret_cast<const v4i*>(Bs + row * kLdsStride + kb);
      }
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[a], bf[b], acc[a][b], 0, 0, 0);
    }
    __syncthreads();
  }

  // ---- epilogue: y = float(acc) * (beta_seg / s_m); segments split N ----
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int64_t n = n0 + wn * 64 + b * 32 + (lane & 31);
    if (n >= N) continue;
    int sg = 0;
    if (out.nseg > 1 && n >= out.nstart[1]) sg = 1;
    if (out.nseg > 2 && n >= out.nstart[2]) sg = 2;
    TY* y = reinterpret_cast<TY*>(out.y[sg]);
    const int64_t ld = out.ld[sg];
    const int64_t nl = n - out.nstart[sg];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int li = wm * 64 + a * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const int64_t m = m0 + li;
        if (m < M) {
          const int32_t v = acc[a][b][r];
          const float yv = (float)v * rrow[sg][li];
          TY* p = y + m * ld + nl;
          if (MODE == kGemmStore) {
            store_act(p, yv);
          } else {  // residual: h <- round(h + round(y))
            store_act(p, load_act(p) + round_act(p, yv));
          }
          if (acc_out) acc_out[m * N + n] = v;
        }
      }
  }
}

// ===========================================================================
hipError_t launch_act_quant(const void* x, termezo_dtype xdt, int64_t M, int64_t K, int8_t* xq,
                            float* s, hipStream_t st) {
  if (xdt == TERMEZO_F32)
    hipLaunchKernelGGL(k_act_quant<float>, dim3(M), dim3(256), 0, st, (const float*)x, K, xq, s);
  else
    hipLaunchKernelGGL(k_act_quant<uint16_t>, dim3(M), dim3(256), 0, st, (const uint16_t*)x, K, xq,
                       s);
  return hipGetLastError();
}

hipError_t launch_gemm_i8(const int8_t* xq, const float* s, const uint32_t* codes, int64_t M,
                          int64_t K, int64_t N, const GemmOut& out, termezo_dtype ydt, int mode,
                          int32_t* acc, hipStream_t st) {
  dim3 grid((unsigned)((N + kBN - 1) / kBN), (unsigned)((M + kBM - 1) / kBM));
  if (ydt == TERMEZO_F32) {
    if (mode == kGemmStore)
      hipLaunchKernelGGL((k_gemm_i8<float, kGemmStore>), grid, dim3(256), 0, st, xq, s, codes, M, K,
                         N, out, acc);
    else
      hipLaunchKernelGGL((k_gemm_i8<float, kGemmResidual>), grid, dim3(256), 0, st, xq, s, codes, M,
                         K, N, out, acc);
  } else {
    if (mode == kGemmStore)
      hipLaunchKernelGGL((k_gemm_i8<uint16_t, kGemmStore>), grid, dim3(256), 0, st, xq, s, codes, M,
                         K, N, out, acc);
    else
      hipLaunchKernelGGL((k_gemm_i8<uint16_t, kGemmResidual>), grid, dim3(256), 0, st, xq, s, codes,
                         M, K, N, out, acc);
  }
  return hipGetLastError();
}

hipError_t launch_bitlinear_gemm(const int8_t* xq, const float* s, const uint32_t* codes,
                                 const float* beta_dev, int64_t M, int64_t K, int64_t N, void* y,
                                 termezo_dtype ydt, int32_t* acc, hipStream_t st) {
  GemmOut out = {};
  out.nseg = 1;
  out.y[0] = y;
  out.ld[0] = N;
  out.beta[0] = beta_dev;
  out.nstart[0] = 0;
  out.nstart[1] = N;
  return launch_gemm_i8(xq, s, codes, M, K, N, out, ydt, kGemmStore, acc, st);
}

}  // namespace tmz
