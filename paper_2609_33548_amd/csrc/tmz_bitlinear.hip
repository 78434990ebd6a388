// BitLinear forward on gfx950: per-token absmax int8 activation quantisation
// and the int8 x ternary contraction on the int8 matrix cores
// (v_mfma_i32_32x32x32_i8), int32 accumulation, per-row rescale epilogue.
#include <hip/hip_ext.h>

#include "tmz_device.h"
#include "tmz_internal.h"

namespace tmz {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// Activation quantisation, one block per token row:
//   a = max |x|, s = 127 / max(a, 1e-5), x_q = clamp(rne(x s), -128, 127),
// and the row's sum of x_q (int32, for the offset weight encoding of the
// full-tile GEMM).
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

// Rows of up to kActRegs * 4 * 256 values are held in registers (one read of
// x); longer rows are read twice.
constexpr int kActRegs = 8;

template <typename T>
__global__ void __launch_bounds__(256) k_act_quant(const T* __restrict__ x, int64_t K,
                                                   int8_t* __restrict__ xq, float* __restrict__ s,
                                                   int32_t* __restrict__ rs) {
  __shared__ float red[4];
  __shared__ int ired[4];
  const int64_t m = blockIdx.x;
  const T* row = x + m * K;
  uint32_t* out = reinterpret_cast<uint32_t*>(xq + m * K);
  const bool held = K <= (int64_t)kActRegs * 4 * 256;
  float v[kActRegs][4];
  float a = 0.0f;
  if (held) {
#pragma unroll
    for (int i = 0; i < kActRegs; ++i) {
      const int64_t k = ((int64_t)i * 256 + threadIdx.x) * 4;
      if (k < K) {
        load4(row + k, v[i]);
      } else {
        v[i][0] = v[i][1] = v[i][2] = v[i][3] = 0.0f;
      }
      a = fmaxf(a, fmaxf(fmaxf(fabsf(v[i][0]), fabsf(v[i][1])), fmaxf(fabsf(v[i][2]), fabsf(v[i][3]))));
    }
  } else {
    for (int64_t k = (int64_t)threadIdx.x * 4; k < K; k += 256 * 4) {
      float w[4];
      load4(row + k, w);
      a = fmaxf(a, fmaxf(fmaxf(fabsf(w[0]), fabsf(w[1])), fmaxf(fabsf(w[2]), fabsf(w[3]))));
    }
  }
  a = wave_max(a);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = a;
  __syncthreads();
  a = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  const float sc = __fdiv_rn(127.0f, fmaxf(a, 1e-5f));
  if (threadIdx.x == 0) s[m] = sc;
  int qs = 0;                                        // this thread's sum of x_q
  auto pack = [&](const float* w) __attribute__((always_inline)) {
    const int32_t q0 = quant_byte(w[0], sc), q1 = quant_byte(w[1], sc);
    const int32_t q2 = quant_byte(w[2], sc), q3 = quant_byte(w[3], sc);
    qs += q0 + q1 + q2 + q3;
    return ((uint32_t)q0 & 0xFFu) | (((uint32_t)q1 & 0xFFu) << 8) | (((uint32_t)q2 & 0xFFu) << 16) |
           (((uint32_t)q3 & 0xFFu) << 24);
  };
  if (held) {
#pragma unroll
    for (int i = 0; i < kActRegs; ++i) {
      const int64_t k = ((int64_t)i * 256 + threadIdx.x) * 4;
      if (k < K) out[k / 4] = pack(v[i]);
    }
  } else {
    for (int64_t k = (int64_t)threadIdx.x * 4; k < K; k += 256 * 4) {
      float w[4];
      load4(row + k, w);
      out[k / 4] = pack(w);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) qs += __shfl_xor(qs, off, 64);
  if ((threadIdx.x & 63) == 0) ired[threadIdx.x >> 6] = qs;
  __syncthreads();
  if (threadIdx.x == 0) rs[m] = ired[0] + ired[1] + ired[2] + ired[3];
}

// ---------------------------------------------------------------------------
// Tiled int8 GEMM  acc = x_q c^T  with the 2-bit codes unpacked into LDS.
//
// Block tile BM x BN x 64; the waves form a (BM/WM) x (BN/WN) grid and each
// owns a WM x WN sub-tile made of v_mfma_i32_32x32x32_i8 tiles (int32
// accumulators in AGPRs).  LDS holds two stages (double buffer, one barrier per
// K step); the global loads of step i+2 are issued while step i is computed.
// Within each 32-wide K step lane l supplies the 16 bytes at k = 16 (l / 32)
// of row l % 32 for both operands, so A and B agree on the K assignment.
// Accumulator layout (32 x 32, 16 values per lane): column l % 32,
// row 8 (r / 4) + 4 (l / 32) + (r % 4).
// LDS rows are 64 data bytes + 16 pad (80 B stride: the 16-byte fragment reads of
// consecutive rows fall in distinct banks).
// ---------------------------------------------------------------------------
// Block tile BM x BN with a K step of BK = 128; 8 waves in a 2 x 4 grid, each
// owning a 128 x 64 sub-tile of v_mfma_i32_32x32x32_i8 tiles (int32
// accumulators).  Two LDS stages (one barrier per K step); the global loads of
// step k+2 are issued after step k's MFMAs and stored to LDS after step k+1's.
// Within each 32-wide K sub-step, lane l supplies the 16 bytes at
// k = 16 (l / 32) of row l % 32 for both operands, so A and B agree on the K
// assignment.  Accumulator layout (32 x 32, 16 values per lane): column l % 32,
// row 8 (r / 4) + 4 (l / 32) + (r % 4).  LDS rows are 128 data bytes + 16 pad
// (144 B: 16-byte fragment reads of 16 consecutive rows hit distinct banks).
// FULL = every tile is in bounds (M % BM = N % BN = K % BK = 0): no predication.
// ---------------------------------------------------------------------------
constexpr int kBK = 128;
constexpr int kLdsStride = kBK + 16;

__device__ __forceinline__ void store_act(float* p, float v) { *p = v; }
__device__ __forceinline__ void store_act(uint16_t* p, float v) {
  *reinterpret_cast<__bf16*>(p) = (__bf16)v;
}
__device__ __forceinline__ float load_act(const float* p) { return *p; }
__device__ __forceinline__ float load_act(const uint16_t* p) { return bf16_to_f32(*p); }
__device__ __forceinline__ float round_act(const float*, float v) { return v; }
__device__ __forceinline__ float round_act(const uint16_t*, float v) { return (float)(__bf16)v; }
// Both values rounded to the activation type (bf16: one packed conversion).
__device__ __forceinline__ void round_act2(const float*, float&, float&) {}
__device__ __forceinline__ void round_act2(const uint16_t*, float& a, float& b) {
  const uint32_t p = pack_bf16x2(a, b);
  a = __uint_as_float(p << 16);
  b = __uint_as_float(p & 0xFFFF0000u);
}

// Four consecutive activations: one 8-byte (bf16) or 16-byte (fp32) access.
__device__ __forceinline__ void store4(float* p, const float v[4]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void store4(uint16_t* p, const float v[4]) {
  *reinterpret_cast<uint2*>(p) = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
}
// h + y for a 16-byte unit of outputs, rounded to the output type.
__device__ __forceinline__ v4u add_units(v4u h, v4u y, const float*) {
  v4u r;
#pragma unroll
  for (int i = 0; i < 4; ++i) r[i] = __float_as_uint(__uint_as_float(h[i]) + __uint_as_float(y[i]));
  return r;
}
__device__ __forceinline__ v4u add_units(v4u h, v4u y, const uint16_t*) {
  v4u r;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    r[i] = pack_bf16x2(__uint_as_float(h[i] << 16) + __uint_as_float(y[i] << 16),
                       __uint_as_float(h[i] & 0xFFFF0000u) + __uint_as_float(y[i] & 0xFFFF0000u));
  return r;
}
__device__ __forceinline__ void load4v(const float* p, float v[4]) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
}
__device__ __forceinline__ void load4v(const uint16_t* p, float v[4]) {
  const uint2 a = *reinterpret_cast<const uint2*>(p);
  v[0] = __uint_as_float(a.x << 16);
  v[1] = __uint_as_float(a.x & 0xFFFF0000u);
  v[2] = __uint_as_float(a.y << 16);
  v[3] = __uint_as_float(a.y & 0xFFFF0000u);
}

template <int BM, int BN, int WM, int WN, bool FULL, typename TY, int MODE>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64)
    k_gemm_i8(const int8_t* __restrict__ xq, const float* __restrict__ s,
              const uint32_t* __restrict__ codes, int64_t M, int64_t K, int64_t N, GemmOut out,
              int32_t* __restrict__ acc_out) {
  constexpr int NT = (BM / WM) * (BN / WN) * 64;
  constexpr int TM = WM / 32, TN = WN / 32;         // MFMA tiles per wave
  constexpr int CPR = kBK / 16;                     // 16-byte chunks per row
  constexpr int A_CH = BM * CPR / NT;               // A chunks per thread per stage
  constexpr int WPR = kBK / 16;                     // code words per row per stage
  constexpr int B_WORDS = BN * WPR / NT;            // code words per thread per stage
  static_assert(A_CH >= 1 && B_WORDS >= 1 && B_WORDS <= 4 && WPR % B_WORDS == 0, "tiling");
  constexpr int STAGE = (BM + BN) * kLdsStride;
  __shared__ __attribute__((aligned(16))) int8_t smem[2 * STAGE];
  __shared__ float rrow[kMaxSeg][BM];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wid = tid >> 6;
  const int wm = wid / (BN / WN), wn = wid % (BN / WN);
  int64_t tm, tn;
  tile_of_block((M + BM - 1) / BM, (N + BN - 1) / BN, tm, tn);
  const int64_t m0 = tm * BM, n0 = tn * BN;
  const int64_t KW = K / 16;                        // code words per row
  const int nk = (int)((K + kBK - 1) / kBK);

  for (int i = tid; i < kMaxSeg * BM; i += NT) {
    const int sg = i / BM, r = i % BM;
    const int64_t m = m0 + r;
    rrow[sg][r] = (sg < out.nseg && m < M) ? __fdiv_rn(*out.beta[sg], s[m]) : 0.0f;
  }

  const int brow = (tid * B_WORDS) / WPR, bw0 = (tid * B_WORDS) % WPR;
  const int8_t* abase = xq + m0 * K;
  const uint32_t* bbase = codes + (n0 + brow) * KW + bw0;

  v4u ra[A_CH];
  uint32_t rb[B_WORDS];
  auto gload = [&](int kt) __attribute__((always_inline)) {
    const int64_t k0 = (int64_t)kt * kBK;
#pragma unroll
    for (int it = 0; it < A_CH; ++it) {
      const int c = tid + NT * it;
      const int row = c / CPR, col = c % CPR;
      if (FULL || (m0 + row < M && k0 + 16 * col < K))
        ra[it] = *reinterpret_cast<const v4u*>(abase + row * K + k0 + 16 * col);
      else
        ra[it] = v4u{0u, 0u, 0u, 0u};
    }
    const int64_t kw0 = k0 / 16;
    if constexpr (FULL && B_WORDS == 4) {
      const v4u v = *reinterpret_cast<const v4u*>(bbase + kw0);
      rb[0] = v.x;
      rb[1] = v.y;
      rb[2] = v.z;
      rb[3] = v.w;
    } else if constexpr (FULL && B_WORDS == 2) {
      const uint2 v = *reinterpret_cast<const uint2*>(bbase + kw0);
      rb[0] = v.x;
      rb[1] = v.y;
    } else {
#pragma unroll
      for (int j = 0; j < B_WORDS; ++j)
        rb[j] = (FULL || (n0 + brow < N && kw0 + bw0 + j < KW)) ? bbase[kw0 + j] : 0u;
    }
  };
  auto lstore = [&](int buf) __attribute__((always_inline)) {
    int8_t* As = smem + buf * STAGE;
    int8_t* Bs = As + BM * kLdsStride;
#pragma unroll
    for (int it = 0; it < A_CH; ++it) {
      const int c = tid + NT * it;
      *reinterpret_cast<v4u*>(As + (c / CPR) * kLdsStride + 16 * (c % CPR)) = ra[it];
    }
#pragma unroll
    for (int j = 0; j < B_WORDS; ++j) {
      uint32_t o[4];
      unpack_word(rb[j], o);
      const v4u v = {o[0], o[1], o[2], o[3]};
      *reinterpret_cast<v4u*>(Bs + brow * kLdsStride + 16 * (bw0 + j)) = v;
    }
  };

  v16i acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0;

  gload(0);
  lstore(0);
  if (nk > 1) gload(1);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int8_t* As = smem + (kt & 1) * STAGE;
    const int8_t* Bs = As + BM * kLdsStride;
#pragma unroll
    for (int ks = 0; ks < kBK / 32; ++ks) {
      const int kb = 32 * ks + 16 * (lane >> 5);
      v4i af[TM], bf[TN];
#pragma unroll
      for (int a = 0; a < TM; ++a)
        af[a] = *reinterpret_cast<const v4i*>(As + (wm * WM + a * 32 + (lane & 31)) * kLdsStride + kb);
#pragma unroll
      for (int b = 0; b < TN; ++b)
        bf[b] = *reinterpret_cast<const v4i*>(Bs + (wn * WN + b * 32 + (lane & 31)) * kLdsStride + kb);
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[a], bf[b], acc[a][b], 0, 0, 0);
    }
    if (kt + 1 < nk) {
      lstore((kt + 1) & 1);
      if (kt + 2 < nk) gload(kt + 2);
    }
    __syncthreads();
  }

  // ---- epilogue: y = float(acc) * (beta_seg / s_m); segments split N ----
  const int rl = wm * WM + 4 * (lane >> 5);          // lane's first local row
#pragma unroll
  for (int b = 0; b < TN; ++b) {
    const int64_t n = n0 + wn * WN + b * 32 + (lane & 31);
    if (!FULL && n >= N) continue;
    int sg = 0;
    if (out.nseg > 1 && n >= out.nstart[1]) sg = 1;
    if (out.nseg > 2 && n >= out.nstart[2]) sg = 2;
    const int64_t ld = out.ld[sg];
    TY* colp = reinterpret_cast<TY*>(out.y[sg]) + (n - out.nstart[sg]) + (m0 + rl) * ld;
    const float* rr = &rrow[sg][rl];
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ro = a * 32 + 8 * (r >> 2) + (r & 3);
        if (FULL || m0 + rl + ro < M) {
          const int32_t v = acc[a][b][r];
          const float yv = (float)v * rr[ro];
          TY* p = colp + (int64_t)ro * ld;
          if (MODE == kGemmStore) {
            store_act(p, yv);
          } else {  // residual: h <- round(h + round(y))
            store_act(p, load_act(p) + round_act(p, yv));
          }
          if (acc_out) acc_out[(m0 + rl + ro) * N + n] = v;
        }
      }
  }
}

// ---------------------------------------------------------------------------
// Full-tile GEMM with direct global -> LDS loads (global_load_lds_dwordx4:
// lane i of a wave writes its 16 bytes at the wave's LDS base + 16 i, no VGPRs)
// into a ring of NST stages of BK = 128 or 256 K values each; the loads of
// step k + NST - 1 are issued as step k starts, so they have NST - 1 steps of
// compute to land, and one barrier per step publishes them.
//   A stage: BM rows x BK bytes; 16-byte chunk c of row r stored at chunk
//            c ^ swz(r) (128: (r >> 1) & 7; 256: r & 15).
//   B stage: BN rows x BK / 4 bytes of packed 2-bit codes; 16-byte unit u of
//            row r stored at unit u ^ bswz(r) (128: bit 2 ^ bit 3 of r;
//            256: (r >> 2) & 3).
// The swizzles keep the 16-byte fragment reads of 8 or 16 consecutive rows on
// distinct banks.  8 waves as 2 x 4, WM x WN per wave,
// v_mfma_i32_32x32x32_i8 with the activations as the first operand and the codes
// as the second (the matrix cores run measurably faster with the few-bit code
// values in the second operand), so a lane's accumulator column is one output
// feature and its 16 registers are 16 tokens.
// K assignment: in sub-step ks (32 wide) of a K step of KS = BK / 32 sub-steps,
// lane l supplies the 16 values at k = 16 (KS (l / 32) + ks) for both operands,
// so one 16-byte read gives a lane the codes of four sub-steps.  The codes of sub-step ks+1 are
// unpacked between the MFMAs of sub-step ks.  The accumulators start at minus the
// activation row sums (the codes enter as w + 1); the per-token output scales
// beta' / s_m are tabulated in LDS after the main loop.
//
// Tiles are 256 x 256 (128 x 64 per wave).  When the last round of tiles
// would fill at most half of the compute units, its tiles are instead cut
// into four 128 x 128 tiles (64 x 32 per wave), so the tail takes about a
// quarter of a round instead of a whole one.  K step 256 (two stages of 80 KB,
// the whole LDS) when K allows, else 128 (three stages).
// Requires M % 256 == 0, N % 256 == 0, K % BK == 0.
// ---------------------------------------------------------------------------
template <int BK>
__device__ __forceinline__ int aswz(int row) {
  return BK == 256 ? (row & 15) : ((row >> 1) & 7);
}
template <int BK>
__device__ __forceinline__ int bswz(int row) {
  return BK == 256 ? ((row >> 2) & 3) : (((row >> 2) ^ (row >> 3)) & 1);
}

__device__ __forceinline__ v4i unpack16(uint32_t w) {
  uint32_t o[4];
  unpack_word(w, o);
  return v4i{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
}

// The 16 codes of a word as the int8 values w + 1 (0, 1, 2 for w = -1, 0, +1), the
// operand of the full-tile GEMM: acc' = sum_k x_q (w + 1) and acc = acc' - sum_k x_q,
// exactly, in int32.  The offset values switch far fewer operand bits than
// two's-complement -1 (0xFF), and the matrix cores draw less power on them (the
// same GEMM measured 5% faster in the decoder step).  Same selector scheme as
// unpack_word: bytes 0, 1, 2 of the low table for groups 0 and 2; for groups 1
// and 3 selectors 0, 4, 8: byte 0 of the low table, byte 0 of the high table and
// the (clear) sign of the low table's byte 1.
__device__ __forceinline__ v4i unpack16_off1(uint32_t w) {
  const uint32_t y = w >> 4;
  return v4i{(int)__builtin_amdgcn_perm(0u, 0x00000201u, w & 0x03030303u),
             (int)__builtin_amdgcn_perm(0x02u, 0x00000001u, w & 0x0C0C0C0Cu),
             (int)__builtin_amdgcn_perm(0u, 0x00000201u, y & 0x03030303u),
             (int)__builtin_amdgcn_perm(0x02u, 0x00000001u, y & 0x0C0C0C0Cu)};
}

constexpr int kDmaBM = 256, kDmaBN = 256;
template <int BK, int NST>
constexpr int dma_lds_bytes(int BM, int BN) { return NST * (BM * BK + BN * BK / 4); }

template <int BM, int BN, int WM, int WN, typename TY, int MODE, int BK, int NST>
__device__ __forceinline__ void gemm_tile_dma(const int8_t* __restrict__ xq,
                                              const uint32_t* __restrict__ codes, int64_t K,
                                              int64_t N, const GemmOut& out, int32_t* acc_out,
                                              int64_t m0, int64_t n0, int8_t* lds,
                                              const float* __restrict__ s,
                                              const int32_t* __restrict__ rs) {
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int AROW = BK;                        // bytes per A row per stage (no pad)
  constexpr int BROW = BK / 4;                    // bytes of packed codes per B row per stage
  constexpr int ACH = BK / 16;                    // 16-byte chunks per A row
  constexpr int BU = BROW / 16;                   // 16-byte units per B row
  constexpr int ASTAGE = BM * AROW, BSTAGE = BN * BROW;
  constexpr int KS = BK / 32;                     // MFMA sub-steps per K step
  constexpr int HK = KS / 4;                      // 16-byte code reads per lane per fragment
  constexpr int NW = (BM / WM) * (BN / WN);       // waves per block
  constexpr int ARPI = 1024 / AROW;               // A rows per 1 KB load instruction
  constexpr int BRPI = 1024 / BROW;               // B rows per 1 KB load instruction
  constexpr int AJ = BM / (ARPI * NW);            // A loads per wave per stage
  constexpr int BW = BN / BRPI < NW ? BN / BRPI : NW;      // waves holding distinct B rows
  constexpr int BJ = BN / BRPI > NW ? BN / (BRPI * NW) : 1;  // B loads per wave per stage
  constexpr int DJ = AJ + BJ;                     // direct loads per wave per stage
  static_assert(AJ >= 1 && BM % (ARPI * NW) == 0 && (BN / BRPI <= NW || BN % (BRPI * NW) == 0) &&
                    DJ * (NST - 1) < 64 && (BK == 128 || BK == 256), "tile");
  const int tid = threadIdx.x;
  const int lane = tid & 63, wid = tid >> 6;
  const int wm = wid / (BN / WN), wn = wid % (BN / WN);
  const int64_t KW = K / 16;
  const int nk = (int)(K / BK);

  // Per-lane global sources.  A: wave w fills 1 KB chunks AJ w .. AJ w + AJ-1
  // (ARPI rows each); lane i -> row ARPI j + i / ACH, physical chunk i % ACH.
  // B: wave w fills the BRPI-row blocks BJ (w % BW) .. + BJ-1, BU lanes
  // (physical units) per row (with BW < NW several waves write the same bytes).
  const int8_t* asrc[AJ];
#pragma unroll
  for (int j = 0; j < AJ; ++j) {
    const int row = ARPI * (AJ * wid + j) + lane / ACH;
    const int chunk = (lane % ACH) ^ aswz<BK>(row);
    asrc[j] = xq + (m0 + row) * K + 16 * chunk;
  }
  const int bw = wid % BW;
  const uint32_t* bsrc[BJ];
#pragma unroll
  for (int j = 0; j < BJ; ++j) {
    const int brow_l = BRPI * (BJ * bw + j) + lane / BU;
    int64_t crow = n0 + brow_l;                   // code row of tile row brow_l
    if constexpr (MODE == kGemmSwiGLU) {
      // column 64 p + c holds gate row 32 p + c (c < 32) or up row F + 32 p + c - 32, so
      // a wave's column blocks b = 0 and 1 hold the gate and the up values of the same
      // 32 features in the same lanes
      const int64_t p = crow >> 6, c = crow & 63;
      crow = c < 32 ? 32 * p + c : (N >> 1) + 32 * p + (c - 32);
    }
    bsrc[j] = codes + crow * KW + 4 * ((lane % BU) ^ bswz<BK>(brow_l));
  }

  static_assert(MODE != kGemmSwiGLU || WN == 64, "SwiGLU: gate and up blocks of one wave");
  // the segments' beta', for the epilogue's table of output scales
  float bet[kMaxSeg];
#pragma unroll
  for (int sg = 0; sg < kMaxSeg; ++sg) bet[sg] = sg < out.nseg ? *out.beta[sg] : 0.0f;

  const uint32_t wa = __builtin_amdgcn_readfirstlane(wid);   // wave-uniform
  const uint32_t wb = __builtin_amdgcn_readfirstlane(bw);
  auto issue = [&](int kt, int8_t* Ad, uint32_t* Bd) __attribute__((always_inline)) {
    const int64_t koff = (int64_t)kt * BK;
    const uint32_t abase = lds_offset(Ad) + 1024u * AJ * wa;
#pragma unroll
    for (int j = 0; j < AJ; ++j) dma16(asrc[j] + koff, abase + 1024u * j);
    const uint32_t bbase = lds_offset(Bd) + 1024u * BJ * wb;
#pragma unroll
    for (int j = 0; j < BJ; ++j) dma16(bsrc[j] + koff / 16, bbase + 1024u * j);
  };

  // Accumulator register r of tile (a, b) is token wm WM + 32 a + 8 (r / 4) + 4 h + r % 4
  // and feature column wn WN + 32 b + n of the block (n = lane % 32, h = lane / 32).  It
  // starts at -sum_k x_q of its token, so it ends at sum_k x_q (w + 1) - sum_k x_q =
  // sum_k x_q w.
  const int h = lane >> 5, n = lane & 31;
  v16i acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a) {
    const int32_t* rp = rs + m0 + wm * WM + 32 * a + 4 * h;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const v4i r4 = *reinterpret_cast<const v4i*>(rp + 8 * q);
#pragma unroll
      for (int b = 0; b < TN; ++b)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[a][b][4 * q + j] = -r4[j];
    }
  }

  const int arow0 = wm * WM + (lane & 31);        // A fragment row of this lane (a = 0)
  const int brow0 = wn * WN + (lane & 31);
  // Fragments live across K steps: the first A fragments and the packed codes of the
  // next stage are read right after the barrier that ends a stage, ahead of that
  // stage's last MFMA sub-step (whose operands are already in registers), so their LDS
  // latency and the first code unpacking fall under MFMAs instead of stalling both
  // waves of each SIMD at every stage boundary.
  v4i af[2][TM];
  v4i bq[HK][TN], bfc[TN], bfn[TN];
  auto afrag = [&](const int8_t* As, int ks, int slot) __attribute__((always_inline)) {
    const int c = (ACH / 2) * h + ks;                // logical 16-byte chunk
#pragma unroll
    for (int a = 0; a < TM; ++a) {
      const int row = arow0 + 32 * a;
      af[slot][a] = *reinterpret_cast<const v4i*>(As + row * AROW + 16 * (c ^ aswz<BK>(row)));
    }
  };
  // the packed codes of a stage and its first A fragments
  auto first = [&](const int8_t* As, const uint32_t* Bs) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < HK; ++q)
#pragma unroll
      for (int b = 0; b < TN; ++b) {
        const int row = brow0 + 32 * b;
        bq[q][b] = *reinterpret_cast<const v4i*>(Bs + row * (BROW / 4) +
                                                 4 * ((HK * h + q) ^ bswz<BK>(row)));
      }
    afrag(As, 0, 0);
  };
  auto mfmas = [&](int slot) __attribute__((always_inline)) {
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int b = 0; b < TN; ++b)   // activations first, codes second: acc holds Y
        acc[a][b] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[slot][a], bfc[b], acc[a][b], 0, 0, 0);
  };
  // sub-steps 0 .. KS-2 of a stage (reading the fragments of the next sub-step during
  // each); the operands of sub-step KS-1 are left in af[(KS-1) & 1] and bfc
  auto steps = [&](const int8_t* As) __attribute__((always_inline)) {
#pragma unroll
    for (int b = 0; b < TN; ++b) bfc[b] = unpack16_off1((uint32_t)bq[0][b][0]);
#pragma unroll
    for (int ks = 0; ks + 1 < KS; ++ks) {
      const int cur = ks & 1;
      afrag(As, ks + 1, cur ^ 1);
#pragma unroll
      for (int b = 0; b < TN; ++b) bfn[b] = unpack16_off1((uint32_t)bq[(ks + 1) / 4][b][(ks + 1) % 4]);
      mfmas(cur);
      __builtin_amdgcn_sched_group_barrier(0x100, TM, 0);      // next A fragments (LDS reads)
#pragma unroll
      for (int i = 0; i < TM * TN; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);     // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);     // then unpack work (VALU)
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int b = 0; b < TN; ++b) bfc[b] = bfn[b];
    }
  };

  auto Ast = [&](int st) { return lds + st * ASTAGE; };
  auto Bst = [&](int st) { return reinterpret_cast<uint32_t*>(lds + NST * ASTAGE + st * BSTAGE); };
  // prologue: stages 0 .. NST-2 in flight, stage 0 complete before the loop
#pragma unroll
  for (int p = 0; p < NST - 1; ++p)
    if (p < nk) issue(p, Ast(p), Bst(p));
  if (NST == 3 && nk > 1) wait_vmcnt_le<DJ>(); else __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  first(Ast(0), Bst(0));
  int cur = 0;
  for (int kt = 0; kt < nk; ++kt) {
    const int nxt = cur == 0 ? NST - 1 : cur - 1;     // (kt + NST - 1) % NST
    const int nst = cur == NST - 1 ? 0 : cur + 1;      // stage of step kt + 1
    // the buffer of step kt - 1: every wave finished reading it before the last barrier
    if (kt + NST - 1 < nk) issue(kt + NST - 1, Ast(nxt), Bst(nxt));
    steps(Ast(cur));
#pragma unroll
    for (int b = 0; b < TN; ++b)   // the last sub-step's codes unpacked before the barrier
      asm volatile("" : "+v"(bfc[b]));
    // the loads of step kt + 1 have landed (NST = 3: those of kt + 2 may still be in flight)
    if (NST == 3 && kt + 2 < nk) wait_vmcnt_le<DJ>(); else __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (kt + 1 < nk) first(Ast(nst), Bst(nst));
    mfmas((KS - 1) & 1);                              // the last sub-step of step kt
    __builtin_amdgcn_sched_barrier(0);
    cur = nst;
  }

  // ---- epilogue.  Each wave stages one 32-token slice (MFMA row tile a) of its
  // outputs row-major in a private LDS region (the ring is free after the last
  // barrier), then writes whole 16-byte units, so a store instruction covers
  // 64 / UPR tokens of UPR * 16 contiguous bytes each instead of scattered
  // 2-byte values.  Unit u of staged row r sits at unit u ^ (r % UPR).  The LDS
  // writes and reads of one wave need no barrier: a wave's LDS operations are
  // ordered.  The output scales beta' / s_m of the block's tokens (one per segment)
  // are computed once per block into a table after the staging regions.
  constexpr int OW = MODE == kGemmSwiGLU ? WN / 2 : WN;   // outputs per staged row
  constexpr int UB = 16 / (int)sizeof(TY);                // outputs per 16-byte unit
  constexpr int UPR = OW / UB;                            // units per staged row
  constexpr int RB = OW * (int)sizeof(TY);                // bytes per staged row
  constexpr int RPL = 32 * UPR / 64;                      // units read per lane
  static_assert(NW * 32 * RB + kMaxSeg * BM * 4 <= NST * (ASTAGE + BSTAGE) && RPL >= 1 &&
                    UPR <= 16, "epilogue staging");
  int8_t* wl = lds + wid * 32 * RB;
  float* fac = reinterpret_cast<float*>(lds + NW * 32 * RB);   // [segment][BM]
#pragma unroll
  for (int sg = 0; sg < kMaxSeg; ++sg)
    if (sg < out.nseg)
      for (int t = tid; t < BM; t += NW * 64) fac[sg * BM + t] = __fdiv_rn(bet[sg], s[m0 + t]);
  __syncthreads();
  // the output scales of the lane's 16 tokens of slice a
  auto load_fac = [&](int a, int sg, float f[16]) __attribute__((always_inline)) {
    const float* p = fac + sg * BM + wm * WM + 32 * a + 4 * h;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 v = *reinterpret_cast<const float4*>(p + 8 * q);
      f[4 * q] = v.x; f[4 * q + 1] = v.y; f[4 * q + 2] = v.z; f[4 * q + 3] = v.w;
    }
  };
  // Stage the lane's 16 values (its tokens) of output column c.  bf16: the values of
  // two consecutive tokens are packed, the lane pair (n, n ^ 1) swaps halves (one DPP
  // move), and each lane writes one token's two adjacent outputs (the even lane the
  // first token, the odd lane the second).
  const uint32_t psel = (n & 1) ? 0x03020706u : 0x05040100u;
  auto stage16 = [&](int c, const float v[16]) __attribute__((always_inline)) {
    if constexpr (sizeof(TY) == 2) {
      const int fc = c & ~1;
#pragma unroll
      for (int r = 0; r < 16; r += 2) {
        const uint32_t p = pack_bf16x2(v[r], v[r + 1]);
        const uint32_t o = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)p, 0xB1, 0xF, 0xF, false);
        const int row = 8 * (r >> 2) + 4 * h + (r & 3) + (n & 1);
        *reinterpret_cast<uint32_t*>(wl + row * RB + 16 * ((fc / UB) ^ (row % UPR)) + 2 * (fc % UB)) =
            __builtin_amdgcn_perm(o, p, psel);
      }
    } else {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 8 * (r >> 2) + 4 * h + (r & 3);
        *reinterpret_cast<float*>(wl + row * RB + 16 * ((c / UB) ^ (row % UPR)) + 4 * (c % UB)) = v[r];
      }
    }
  };
  const int64_t fbase = MODE == kGemmSwiGLU ? (n0 + wn * WN) / 2 : n0 + wn * WN;
  // output unit i (of RPL) of slice a of this lane
  auto unit_ptr = [&](int a, int i) __attribute__((always_inline)) {
    const int c = 64 * i + lane, row = c / UPR, u = c % UPR;
    const int64_t tok = m0 + wm * WM + 32 * a + row;
    const int64_t f = fbase + (int64_t)u * UB;
    int sg = 0;
    if constexpr (MODE != kGemmSwiGLU) {
      if (out.nseg > 1 && f >= out.nstart[1]) sg = 1;
      if (out.nseg > 2 && f >= out.nstart[2]) sg = 2;
    }
    return reinterpret_cast<v4u*>(reinterpret_cast<TY*>(out.y[sg]) + tok * out.ld[sg] +
                                  (f - out.nstart[sg]));
  };
  // residual inputs: all of a lane's units loaded up front (at most 16 units, else
  // one slice at a time) so their latency overlaps the staging
  constexpr int HPRE = MODE == kGemmResidual ? (TM * RPL <= 8 ? TM : 1) : 0;
  v4u hin[HPRE > 0 ? HPRE : 1][RPL];
  if constexpr (HPRE == TM) {
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int i = 0; i < RPL; ++i) hin[a][i] = *unit_ptr(a, i);
  }
#pragma unroll
  for (int a = 0; a < TM; ++a) {
    if constexpr (HPRE == 1) {
#pragma unroll
      for (int i = 0; i < RPL; ++i) hin[0][i] = *unit_ptr(a, i);
    }
    if constexpr (MODE == kGemmSwiGLU) {
      // block 0: gate, block 1: up values of feature fbase + n
      float fg[16], fu[16], v[16];
      load_fac(a, 0, fg);
      load_fac(a, 1, fu);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float g = (float)acc[a][0][r] * fg[r], u = (float)acc[a][1][r] * fu[r];
        round_act2((TY*)nullptr, g, u);
        v[r] = silu_mul(g, u);
      }
      stage16(n, v);
    } else {
#pragma unroll
      for (int b = 0; b < TN; ++b) {
        const int64_t nb = n0 + wn * WN + b * 32;
        const int sg = (out.nseg > 2 && nb >= out.nstart[2]) ? 2 : (out.nseg > 1 && nb >= out.nstart[1]) ? 1 : 0;
        float f[16], v[16];
        load_fac(a, sg, f);
#pragma unroll
        for (int r = 0; r < 16; ++r)   // rounded to the output type by the staging store
          v[r] = (float)acc[a][b][r] * f[r];
        stage16(32 * b + n, v);
        if (acc_out) {   // int32 accumulators (parity only), straight from the registers
#pragma unroll
          for (int r = 0; r < 16; ++r)
            acc_out[(m0 + wm * WM + 32 * a + 8 * (r >> 2) + 4 * h + (r & 3)) * N + nb + n] = acc[a][b][r];
        }
      }
    }
    // read back whole units and write them to the outputs
#pragma unroll
    for (int i = 0; i < RPL; ++i) {
      const int c = 64 * i + lane, row = c / UPR, u = c % UPR;
      const v4u v = *reinterpret_cast<const v4u*>(wl + row * RB + 16 * (u ^ (row % UPR)));
      v4u* p = unit_ptr(a, i);
      if constexpr (MODE == kGemmResidual)   // h <- round(h + y), y already rounded
        *p = add_units(hin[HPRE == TM ? a : 0][i], v, (TY*)nullptr);
      else
        *p = v;
    }
  }
}

// Blocks [0, full) take 256 x 256 tiles [0, full) of the grouped order (XCD
// aware); the following blocks take the four 128 x 128 quarters of each tile
// in [full, T).
template <typename TY, int MODE, int BK>
__global__ void __launch_bounds__(512)
    k_gemm_i8_dma(const int8_t* __restrict__ xq, const float* __restrict__ s,
                  const int32_t* __restrict__ rs, const uint32_t* __restrict__ codes, int64_t M, int64_t K, int64_t N, GemmOut out,
                  int64_t full, int32_t* __restrict__ acc_out) {
  constexpr int NST = BK == 256 ? 2 : 3;
  __shared__ __attribute__((aligned(1024))) int8_t lds[dma_lds_bytes<BK, NST>(kDmaBM, kDmaBN)];
  const int64_t nb_m = M / kDmaBM, nb_n = N / kDmaBN;
  const bool quarter = (int64_t)blockIdx.x >= full;
  int64_t t, tm, tn;
  int q = 0;
  if (!quarter) {
    t = xcd_linear(blockIdx.x, full);
  } else {
    const int64_t i = (int64_t)blockIdx.x - full;
    t = full + i / 4;
    q = (int)(i % 4);
  }
  tile_of_linear(t, nb_m, nb_n, tm, tn);
  const int64_t m0 = tm * kDmaBM + (quarter ? 128 * (q >> 1) : 0);
  const int64_t n0 = tn * kDmaBN + (quarter ? 128 * (q & 1) : 0);
  if (!quarter)
    gemm_tile_dma<256, 256, 128, 64, TY, MODE, BK, NST>(xq, codes, K, N, out, acc_out, m0, n0, lds, s,
                                                        rs);
  else
    gemm_tile_dma<128, 128, 64, 32, TY, MODE, BK, NST>(xq, codes, K, N, out, acc_out, m0, n0, lds, s,
                                                       rs);
}

// Two blocks per compute unit: 128 x 256 tiles of 4 waves (128 x 64 per wave, the
// same per-wave work as the 256 x 256 tile) with a 72 KB ring, so that one
// block's barriers, prologue and epilogue overlap the other block's MFMAs and a
// block left alone on a compute unit at the end of the grid runs at its full rate.
constexpr int kHalfBM = 128, kHalfBN = 256;

template <typename TY, int MODE>
__global__ void __launch_bounds__(256, 2)
    k_gemm_i8_dma_h(const int8_t* __restrict__ xq, const float* __restrict__ s,
                    const int32_t* __restrict__ rs, const uint32_t* __restrict__ codes, int64_t M, int64_t K, int64_t N, GemmOut out,
                    int32_t* __restrict__ acc_out) {
  __shared__ __attribute__((aligned(1024))) int8_t lds[dma_lds_bytes<128, 3>(kHalfBM, kHalfBN)];
  int64_t tm, tn;
  tile_of_block(M / kHalfBM, N / kHalfBN, tm, tn);
  gemm_tile_dma<kHalfBM, kHalfBN, 128, 64, TY, MODE, 128, 3>(xq, codes, K, N, out, acc_out,
                                                             tm * kHalfBM, tn * kHalfBN, lds, s, rs);
}

// ---------------------------------------------------------------------------
// Small-M BitLinear (M <= kGemvMaxM): one block of 8 waves per 16 output
// features, so even M = 1 spreads the code stream over N / 16 blocks.
// v_mfma_i32_16x16x64_i8 with the codes as the first operand (16 features x
// 64 k) and a group of 16 tokens as the second.  K is cut in chunks of 256
// (16 code words per feature); in a chunk, lane l loads the 4 words
// 4 (l / 16) .. 4 (l / 16) + 3 of feature l % 16 (one 16-byte load) and MFMA j
// takes word j, i.e. k = 16 (4 (l / 16) + j) .. + 15, with the 16 int8
// activations of token l % 16 at the same k.  Chunks are dealt round-robin to
// the 8 waves; their int32 partial sums meet in LDS.
// Accumulator (16 x 16, 4 values per lane): token l % 16, features
// 4 (l / 16) .. 4 (l / 16) + 3.  Segment boundaries are multiples of 16.
// ---------------------------------------------------------------------------
constexpr int kGemvMaxM = 128;

template <typename TY, int MODE, bool CVEC, int G, int CPW>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(4)))
    k_gemv_i8(const int8_t* __restrict__ xq, const float* __restrict__ s,
              const uint32_t* __restrict__ codes, int64_t M, int64_t K, int64_t N, GemmOut out,
              int yvec, int32_t* __restrict__ acc_out) {
  constexpr int NW = 8;
  static_assert(16 * G <= kGemvMaxM, "token groups");
  __shared__ int32_t red[NW][G][4][64];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int64_t n0 = (int64_t)blockIdx.x * 16;
  const int64_t KW = K / 16;
  const int nchunk = (int)((KW + 15) / 16);
  const int ng = (int)((M + 15) / 16);
  const int fr = lane & 15, g = lane >> 4;
  const bool row_ok = n0 + fr < N;
  const uint32_t* crow = codes + (row_ok ? n0 + fr : 0) * KW;
  // Every load below reads a clamped in-bounds address and out-of-range values are
  // zeroed afterwards; the only branches around loads are wave-uniform, so all the
  // loads of a pass are in flight together.
  v4i acc[G];
#pragma unroll
  for (int tg = 0; tg < G; ++tg) acc[tg] = v4i{0, 0, 0, 0};
  // code words of chunk c (zero outside the matrix)
  auto cload = [&](int c, uint32_t* cw) __attribute__((always_inline)) {
    const int64_t w0 = (int64_t)c * 16 + 4 * g;        // first code word of this lane
    if (CVEC) {                                        // KW % 4 == 0: 4 words or none
      const v4u v = *reinterpret_cast<const v4u*>(crow + (w0 < KW ? w0 : 0));
      const bool ok = row_ok && w0 < KW;
#pragma unroll
      for (int j = 0; j < 4; ++j) cw[j] = ok ? v[j] : 0u;
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t v = crow[w0 + j < KW ? w0 + j : 0];
        cw[j] = (row_ok && w0 + j < KW) ? v : 0u;
      }
    }
  };
  // activations of token group tg at this lane's 4 k chunks of chunk c (zero outside)
  auto xload = [&](int c, int tg, v4i* b) __attribute__((always_inline)) {
    const int64_t kb = ((int64_t)c * 16 + 4 * g) * 16;
    const int64_t m = 16 * tg + fr;
    const int8_t* xr = xq + (m < M ? m : 0) * K;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t k = kb + 16 * j;
      b[j] = *reinterpret_cast<const v4i*>(xr + (k < K ? k : 0));
      if (!(m < M && k < K)) b[j] = v4i{0, 0, 0, 0};
    }
  };
  auto mfma4 = [&](const v4i* a, const v4i* b, v4i& acc_) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < 4; ++j) acc_ = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[j], b[j], acc_, 0, 0, 0);
  };
  // Passes of up to CPW chunks per wave (CPW * 2048 k per pass): every code load of a
  // pass is issued first, then the activations of each token group, so a pass costs
  // one memory round trip.  Chunk indices are wave-uniform: chunks beyond the matrix
  // issue no loads and contribute nothing.
  for (int c0 = wid; c0 < nchunk; c0 += CPW * NW) {
    uint32_t cw[CPW][4];
#pragma unroll
    for (int i = 0; i < CPW; ++i) {
      if (c0 + NW * i < nchunk) {
        cload(c0 + NW * i, cw[i]);
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) cw[i][j] = 0u;
      }
    }
#pragma unroll
    for (int tg = 0; tg < G; ++tg) {
      if (tg < ng) {
        v4i b[CPW][4];
#pragma unroll
        for (int i = 0; i < CPW; ++i)
          if (c0 + NW * i < nchunk) xload(c0 + NW * i, tg, b[i]);
#pragma unroll
        for (int i = 0; i < CPW; ++i) {
          if (c0 + NW * i < nchunk) {
            v4i a4[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) a4[j] = unpack16(cw[i][j]);
            mfma4(a4, b[i], acc[tg]);
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
#pragma unroll
  for (int tg = 0; tg < G; ++tg)
    if (tg < ng)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[wid][tg][i][lane] = acc[tg][i];
  __syncthreads();

  for (int tg = wid; tg < ng; tg += NW) {             // one wave per token group
    const int64_t m = 16 * tg + fr;
    if (m >= M) continue;
    int32_t v[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int32_t t = 0;
#pragma unroll
      for (int w = 0; w < NW; ++w) t += red[w][tg][i][lane];
      v[i] = t;
    }
    const int64_t n = n0 + 4 * g;
    if (n >= N) continue;
    int sg = 0;
    if (out.nseg > 1 && n >= out.nstart[1]) sg = 1;
    if (out.nseg > 2 && n >= out.nstart[2]) sg = 2;
    const float rr = __fdiv_rn(*out.beta[sg], s[m]);
    TY* p = reinterpret_cast<TY*>(out.y[sg]) + m * out.ld[sg] + (n - out.nstart[sg]);
    float y4[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) y4[i] = (float)v[i] * rr;
    if (yvec && n + 3 < N) {
      if (MODE == kGemmStore) {
        store4(p, y4);
      } else {
        float h4[4];
        load4v(p, h4);
#pragma unroll
        for (int i = 0; i < 4; ++i) y4[i] = h4[i] + round_act(p, y4[i]);
        store4(p, y4);
      }
    } else {
      for (int i = 0; i < 4 && n + i < N; ++i) {
        if (MODE == kGemmStore)
          store_act(p + i, y4[i]);
        else
          store_act(p + i, load_act(p + i) + round_act(p + i, y4[i]));
      }
    }
    if (acc_out)
      for (int i = 0; i < 4 && n + i < N; ++i) acc_out[m * N + n + i] = v[i];
  }
}

// ---------------------------------------------------------------------------
// One token (M = 1) with the activation quantisation fused in: every block reads the
// whole activation row (at most 8192 values), forms a = max |x| and
// s = 127 / max(a, 1e-5) and quantises the row into LDS exactly as k_act_quant does,
// then runs the contraction of k_gemv_i8 for its 16 output features (token 0 of the
// 16-token MFMA group).  One launch per call instead of two; the code words are
// loaded first so that their latency overlaps the row's.
// ---------------------------------------------------------------------------
constexpr int kGemv1MaxK = 8192;

__device__ __forceinline__ void load8x(const float* p, float v[8]) {
  load4(p, v);
  load4(p + 4, v + 4);
}
__device__ __forceinline__ void load8x(const uint16_t* p, float v[8]) {
  const uint4 a = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    v[2 * j] = __uint_as_float(w[j] << 16);
    v[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
  }
}

template <typename TX, typename TY, bool CVEC>
__global__ void __launch_bounds__(512)
    k_gemv1_fused(const TX* __restrict__ x, const uint32_t* __restrict__ codes, int64_t K,
                  int64_t N, const float* __restrict__ beta, TY* __restrict__ y, int yvec) {
  constexpr int NW = 8;
  constexpr int CPW = kGemv1MaxK / (256 * NW);        // 256-k chunks per wave at most
  constexpr int XI = kGemv1MaxK / (8 * 512);           // 8-value items of the row per thread
  __shared__ __attribute__((aligned(16))) int8_t xql[kGemv1MaxK];
  __shared__ int32_t red[NW][4][64];
  __shared__ float amx[NW];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int64_t n0 = (int64_t)blockIdx.x * 16;
  const int64_t KW = K / 16;
  const int nchunk = (int)((KW + 15) / 16);
  const int fr = lane & 15, g = lane >> 4;
  const bool row_ok = n0 + fr < N;
  const uint32_t* crow = codes + (row_ok ? n0 + fr : 0) * KW;
  // this wave's code words (chunks wid, wid + NW, ...), zero outside the matrix
  uint32_t cw[CPW][4];
#pragma unroll
  for (int i = 0; i < CPW; ++i) {
    const int64_t w0 = (int64_t)(wid + NW * i) * 16 + 4 * g;
    if (CVEC) {
      const v4u v = *reinterpret_cast<const v4u*>(crow + (w0 < KW ? w0 : 0));
      const bool ok = row_ok && w0 < KW;
#pragma unroll
      for (int j = 0; j < 4; ++j) cw[i][j] = ok ? v[j] : 0u;
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t v = crow[w0 + j < KW ? w0 + j : 0];
        cw[i][j] = (row_ok && w0 + j < KW) ? v : 0u;
      }
    }
  }
  // the activation row: max |x|, then the quantised row into LDS
  float xv[XI][8];
  float a = 0.0f;
#pragma unroll
  for (int it = 0; it < XI; ++it) {
    const int64_t k = ((int64_t)it * 512 + tid) * 8;
    if (k < K) {
      load8x(x + k, xv[it]);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) xv[it][j] = 0.0f;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) a = fmaxf(a, fabsf(xv[it][j]));
  }
  a = wave_max(a);
  if (lane == 0) amx[wid] = a;
  __syncthreads();
#pragma unroll
  for (int w = 0; w < NW; ++w) a = fmaxf(a, amx[w]);
  const float sc = __fdiv_rn(127.0f, fmaxf(a, 1e-5f));
#pragma unroll
  for (int it = 0; it < XI; ++it) {
    const int64_t k = ((int64_t)it * 512 + tid) * 8;
    if (k < K) {
      uint32_t w[2];
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        uint32_t b = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) b |= ((uint32_t)quant_byte(xv[it][4 * h2 + j], sc) & 0xFFu) << (8 * j);
        w[h2] = b;
      }
      *reinterpret_cast<uint2*>(xql + k) = make_uint2(w[0], w[1]);
    }
  }
  __syncthreads();
  // contraction: token fr of the MFMA group is the row for fr == 0, zero otherwise
  v4i acc = v4i{0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < CPW; ++i) {
    const int c = wid + NW * i;
    if (c < nchunk) {                                   // wave-uniform
      const int64_t kb = ((int64_t)c * 16 + 4 * g) * 16;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t k = kb + 16 * j;
        v4i b = *reinterpret_cast<const v4i*>(xql + (k < K ? k : 0));
        if (!(fr == 0 && k < K)) b = v4i{0, 0, 0, 0};
        acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(unpack16(cw[i][j]), b, acc, 0, 0, 0);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) red[wid][i][lane] = acc[i];
  __syncthreads();
  if (wid == 0 && fr == 0) {                            // lanes 0, 16, 32, 48: features 4 g ..
    const int64_t n = n0 + 4 * g;
    if (n < N) {
      const float rr = __fdiv_rn(*beta, sc);
      float y4[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int32_t v = 0;
#pragma unroll
        for (int w = 0; w < NW; ++w) v += red[w][i][lane];
        y4[i] = (float)v * rr;
      }
      if (yvec && n + 3 < N) {
        store4(y + n, y4);
      } else {
        for (int i = 0; i < 4 && n + i < N; ++i) store_act(y + n + i, y4[i]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Two to sixteen tokens with the activation quantisation fused in.  Every block
// issues its code loads first, then reads all M activation rows (half a wave per
// row, the row held in registers), forms each row's a = max |x| and
// s = 127 / max(a, 1e-5) with a half-wave reduction and quantises the rows into LDS
// with the operations of k_act_quant, then contracts its FG groups of 16 output
// features as k_gemv_i8 does (one 16-token MFMA group, activations read from LDS).
// One launch per call instead of two, and no x_q, scale or row-sum buffers.  Every
// block quantises all M rows itself (VALU work that grows with M K), so the launcher
// takes this kernel only for small M K, and two feature groups per block where one
// would need more than a round of blocks.  Rows are held packed (bf16: 8 values per
// 16 bytes) up to KMAX values, at most ROWS rows; LDS rows are padded by 16 bytes so
// the 16 token rows of a fragment read fall in distinct banks.
// ---------------------------------------------------------------------------
constexpr int kGemvFusedMaxM = 16;
constexpr int64_t kGemvFusedMaxMK = 16 * 2560;      // rows x values quantised per block

template <typename TX> struct RowChunk;            // 8 activations as loaded
template <> struct RowChunk<uint16_t> {
  uint4 v;
  __device__ __forceinline__ void load(const uint16_t* p) { v = *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ void zero() { v = make_uint4(0u, 0u, 0u, 0u); }
  __device__ __forceinline__ void launder() {
    asm volatile("" : "+v"(v.x), "+v"(v.y), "+v"(v.z), "+v"(v.w));
  }
  __device__ __forceinline__ void get(float o[8]) const {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      o[2 * j] = __uint_as_float(w[j] << 16);
      o[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
    }
  }
};
template <> struct RowChunk<float> {
  float4 a, b;
  __device__ __forceinline__ void load(const float* p) {
    a = *reinterpret_cast<const float4*>(p);
    b = *reinterpret_cast<const float4*>(p + 4);
  }
  __device__ __forceinline__ void zero() { a = b = make_float4(0.f, 0.f, 0.f, 0.f); }
  __device__ __forceinline__ void launder() {}
  __device__ __forceinline__ void get(float o[8]) const {
    o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
    o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
  }
};

template <typename TX, typename TY, bool CVEC, int KMAX, int ROWS, int FG>
__global__ void __launch_bounds__(512)
    k_gemv_fused(const TX* __restrict__ x, const uint32_t* __restrict__ codes, int64_t M,
                 int64_t K, int64_t N, const float* __restrict__ beta, TY* __restrict__ y,
                 int yvec) {
  constexpr int NW = 8;
  constexpr int CPW = (KMAX + 256 * NW - 1) / (256 * NW);  // 256-k chunks per wave at most
  constexpr int XI = KMAX / (8 * 32);                       // 8-value chunks of a row per lane
  constexpr int LROW = KMAX + 16;                           // LDS row stride in bytes
  static_assert(KMAX % 256 == 0 && ROWS <= 2 * NW && FG <= NW, "row layout");
  __shared__ __attribute__((aligned(16))) int8_t xql[ROWS * LROW];
  __shared__ int32_t red[NW][FG][4][64];
  __shared__ float scl[ROWS];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int64_t n0 = (int64_t)blockIdx.x * 16 * FG;
  const int64_t KW = K / 16;
  const int nchunk = (int)((KW + 15) / 16);
  const int fr = lane & 15, g = lane >> 4;
  // this wave's code words (chunks wid, wid + NW, ...) of each feature group, zero
  // outside the matrix
  uint32_t cw[FG][CPW][4];
#pragma unroll
  for (int f = 0; f < FG; ++f) {
    const bool row_ok = n0 + 16 * f + fr < N;
    const uint32_t* crow = codes + (row_ok ? n0 + 16 * f + fr : 0) * KW;
#pragma unroll
    for (int i = 0; i < CPW; ++i) {
      const int64_t w0 = (int64_t)(wid + NW * i) * 16 + 4 * g;
      if (CVEC) {
        const v4u v = *reinterpret_cast<const v4u*>(crow + (w0 < KW ? w0 : 0));
        const bool ok = row_ok && w0 < KW;
#pragma unroll
        for (int j = 0; j < 4; ++j) cw[f][i][j] = ok ? v[j] : 0u;
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint32_t v = crow[w0 + j < KW ? w0 + j : 0];
          cw[f][i][j] = (row_ok && w0 + j < KW) ? v : 0u;
        }
      }
    }
  }
  // token row r = 2 wid + (lane / 32), chunk (it * 32 + lane % 32) of 8 values
  const int r = 2 * wid + (lane >> 5), j32 = lane & 31;
  const bool rok = r < M && r < ROWS;          // the launcher keeps M <= ROWS
  const TX* xr = x + (rok ? r : 0) * K;
  RowChunk<TX> xv[XI];
  float a = 0.0f;
#pragma unroll
  for (int it = 0; it < XI; ++it) {
    const int64_t k = ((int64_t)it * 32 + j32) * 8;
    if (rok && k < K) xv[it].load(xr + k); else xv[it].zero();
    float v[8];
    xv[it].get(v);
#pragma unroll
    for (int t = 0; t < 8; ++t) a = fmaxf(a, fabsf(v[t]));
  }
#pragma unroll
  for (int off = 16; off > 0; off >>= 1) a = fmaxf(a, __shfl_xor(a, off, 32));
  const float sc = __fdiv_rn(127.0f, fmaxf(a, 1e-5f));
  if (rok) {
    if (j32 == 0) scl[r] = sc;
#pragma unroll
    for (int it = 0; it < XI; ++it) {
      const int64_t k = ((int64_t)it * 32 + j32) * 8;
      if (k < K) {
        float v[8];
        xv[it].launder();                               // keep the row packed until here
        xv[it].get(v);
        uint32_t w[2];
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) {
          uint32_t b = 0;
#pragma unroll
          for (int t = 0; t < 4; ++t) b |= ((uint32_t)quant_byte(v[4 * h2 + t], sc) & 0xFFu) << (8 * t);
          w[h2] = b;
        }
        *reinterpret_cast<uint2*>(xql + r * LROW + k) = make_uint2(w[0], w[1]);
      }
    }
  }
  __syncthreads();
  // contraction: token fr of the MFMA group (token rows at or beyond M only feed their
  // own accumulator column, which is never stored)
  v4i acc[FG];
#pragma unroll
  for (int f = 0; f < FG; ++f) acc[f] = v4i{0, 0, 0, 0};
  const int8_t* xl = xql + (fr < ROWS ? fr : 0) * LROW;
#pragma unroll
  for (int i = 0; i < CPW; ++i) {
    const int c = wid + NW * i;
    if (c < nchunk) {                                   // wave-uniform
      const int64_t kb = ((int64_t)c * 16 + 4 * g) * 16;
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int64_t k = kb + 16 * jj;
        v4i b = *reinterpret_cast<const v4i*>(xl + (k < K ? k : 0));
        if (!(k < K)) b = v4i{0, 0, 0, 0};
#pragma unroll
        for (int f = 0; f < FG; ++f)
          acc[f] = __builtin_amdgcn_mfma_i32_16x16x64_i8(unpack16(cw[f][i][jj]), b, acc[f], 0, 0, 0);
      }
    }
  }
#pragma unroll
  for (int f = 0; f < FG; ++f)
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wid][f][i][lane] = acc[f][i];
  __syncthreads();
  if (wid < FG && fr < M) {                             // wave f: token fr, features 4 g ..
    const int64_t n = n0 + 16 * wid + 4 * g;
    if (n < N) {
      const float rr = __fdiv_rn(*beta, scl[fr]);
      float y4[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int32_t v = 0;
#pragma unroll
        for (int w = 0; w < NW; ++w) v += red[w][wid][i][lane];
        y4[i] = (float)v * rr;
      }
      TY* yr = y + (int64_t)fr * N;
      if (yvec && n + 3 < N) {
        store4(yr + n, y4);
      } else {
        for (int i = 0; i < 4 && n + i < N; ++i) store_act(yr + n + i, y4[i]);
      }
    }
  }
}

// Rows of up to 4096 values for up to 16 tokens; longer bf16 rows (up to 8192 values) for
// at most kGemvFusedLongRows tokens, the rows the long-row instantiation holds in LDS.
constexpr int kGemvFusedLongRows = 5;
bool gemv_fused_ok(int64_t M, int64_t K, termezo_dtype xdt) {
  return M >= 2 && M <= kGemvFusedMaxM && M * K <= kGemvFusedMaxMK &&
         (K <= 4096 || (xdt == TERMEZO_BF16 && K <= 8192 && M <= kGemvFusedLongRows));
}

hipError_t launch_gemv_fused(const void* x, termezo_dtype xdt, const uint32_t* codes,
                             const float* beta_dev, int64_t M, int64_t K, int64_t N, void* y,
                             termezo_dtype ydt, int n_cu, hipStream_t st) {
  if (!gemv_fused_ok(M, K, xdt) || K % 16 != 0) return hipErrorInvalidValue;
  const bool cvec = (K / 16) % 4 == 0 && reinterpret_cast<uintptr_t>(codes) % 16 == 0;
  const int yvec =
      N % 4 == 0 && reinterpret_cast<uintptr_t>(y) % (ydt == TERMEZO_F32 ? 16 : 8) == 0;
  const bool two = (N + 15) / 16 > (n_cu > 0 ? n_cu : 256);   // two feature groups per block
  const dim3 grid((unsigned)(two ? (N + 31) / 32 : (N + 15) / 16));
#define TMZ_GF(TX, TY, CV, KM, RW, FGV)                                                         \
  hipLaunchKernelGGL((k_gemv_fused<TX, TY, CV, KM, RW, FGV>), grid, dim3(512), 0, st,           \
                     (const TX*)x, codes, M, K, N, beta_dev, (TY*)y, yvec)
#define TMZ_GFG(TX, TY, CV, KM, RW)                                     \
  do {                                                                  \
    if (two) TMZ_GF(TX, TY, CV, KM, RW, 2); else TMZ_GF(TX, TY, CV, KM, RW, 1); \
  } while (0)
#define TMZ_GFY(TX, CV, KM, RW)                                                               \
  do {                                                                                        \
    if (ydt == TERMEZO_F32) TMZ_GFG(TX, float, CV, KM, RW); else TMZ_GFG(TX, uint16_t, CV, KM, RW); \
  } while (0)
  if (xdt == TERMEZO_F32) {
    if (cvec) TMZ_GFY(float, true, 4096, 16); else TMZ_GFY(float, false, 4096, 16);
  } else if (K <= 4096) {
    if (cvec) TMZ_GFY(uint16_t, true, 4096, 16); else TMZ_GFY(uint16_t, false, 4096, 16);
  } else {
    if (cvec) TMZ_GFY(uint16_t, true, 8192, kGemvFusedLongRows);
    else TMZ_GFY(uint16_t, false, 8192, kGemvFusedLongRows);
  }
#undef TMZ_GFY
#undef TMZ_GFG
#undef TMZ_GF
  return hipGetLastError();
}

bool gemv1_fused_ok(int64_t M, int64_t K) { return M == 1 && K <= kGemv1MaxK; }

hipError_t launch_gemv1_fused(const void* x, termezo_dtype xdt, const uint32_t* codes,
                              const float* beta_dev, int64_t K, int64_t N, void* y,
                              termezo_dtype ydt, hipStream_t st) {
  if (K > kGemv1MaxK || K % 16 != 0) return hipErrorInvalidValue;
  const bool cvec = (K / 16) % 4 == 0 && reinterpret_cast<uintptr_t>(codes) % 16 == 0;
  const int yvec = reinterpret_cast<uintptr_t>(y) % (ydt == TERMEZO_F32 ? 16 : 8) == 0;
  const dim3 grid((unsigned)((N + 15) / 16));
#define TMZ_G1(TX, TY, CV)                                                                     \
  hipLaunchKernelGGL((k_gemv1_fused<TX, TY, CV>), grid, dim3(512), 0, st, (const TX*)x, codes, K, \
                     N, beta_dev, (TY*)y, yvec)
#define TMZ_G1X(TX, CV)                                        \
  do {                                                          \
    if (ydt == TERMEZO_F32) TMZ_G1(TX, float, CV); else TMZ_G1(TX, uint16_t, CV); \
  } while (0)
  if (xdt == TERMEZO_F32) {
    if (cvec) TMZ_G1X(float, true); else TMZ_G1X(float, false);
  } else {
    if (cvec) TMZ_G1X(uint16_t, true); else TMZ_G1X(uint16_t, false);
  }
#undef TMZ_G1X
#undef TMZ_G1
  return hipGetLastError();
}

// ===========================================================================
hipError_t launch_act_quant(const void* x, termezo_dtype xdt, int64_t M, int64_t K, int8_t* xq,
                            float* s, int32_t* rs, hipStream_t st) {
  if (xdt == TERMEZO_F32)
    hipLaunchKernelGGL(k_act_quant<float>, dim3(M), dim3(256), 0, st, (const float*)x, K, xq, s, rs);
  else
    hipLaunchKernelGGL(k_act_quant<uint16_t>, dim3(M), dim3(256), 0, st, (const uint16_t*)x, K, xq,
                       s, rs);
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN, bool FULL>
static hipError_t launch_tile(const int8_t* xq, const float* s, const uint32_t* codes, int64_t M,
                              int64_t K, int64_t N, const GemmOut& out, termezo_dtype ydt, int mode,
                              int32_t* acc, hipStream_t st, LaunchEvents ev) {
  constexpr int NT = (BM / WM) * (BN / WN) * 64;
  dim3 grid((unsigned)(((N + BN - 1) / BN) * ((M + BM - 1) / BM)));
  if (ydt == TERMEZO_F32) {
    if (mode == kGemmStore)
      hipExtLaunchKernelGGL((k_gemm_i8<BM, BN, WM, WN, FULL, float, kGemmStore>), grid, dim3(NT), 0,
                            st, ev.start, ev.stop, 0, xq, s, codes, M, K, N, out, acc);
    else
      hipExtLaunchKernelGGL((k_gemm_i8<BM, BN, WM, WN, FULL, float, kGemmResidual>), grid, dim3(NT),
                            0, st, ev.start, ev.stop, 0, xq, s, codes, M, K, N, out, acc);
  } else {
    if (mode == kGemmStore)
      hipExtLaunchKernelGGL((k_gemm_i8<BM, BN, WM, WN, FULL, uint16_t, kGemmStore>), grid, dim3(NT),
                            0, st, ev.start, ev.stop, 0, xq, s, codes, M, K, N, out, acc);
    else
      hipExtLaunchKernelGGL((k_gemm_i8<BM, BN, WM, WN, FULL, uint16_t, kGemmResidual>), grid,
                            dim3(NT), 0, st, ev.start, ev.stop, 0, xq, s, codes, M, K, N, out, acc);
  }
  return hipGetLastError();
}

// Tile choice: the small-M kernel up to kGemvMaxM tokens.  When every tile is in bounds
// and the outputs allow 4-wide stores, the direct-to-LDS kernels: 128 x 256 tiles, two
// blocks per compute unit (k_gemm_i8_dma_h), when the 256 x 256 grid is below one round
// of the n_cu compute units or spans at least three rounds, and always for the SwiGLU
// gate|up product; otherwise 256 x 256 tiles of 8 waves (128 x 64 per wave, two waves per
// SIMD) with the last round cut into 128 x 128 quarter tiles when it would fill at most
// half of the compute units (n_cu = 0: never).  Other shapes: the register-staged
// kernel, 256 x 256 blocks of 8 waves when the grid fills the chip, 128 x 128 blocks of 4
// waves otherwise.
bool gemm_swiglu_ok(int64_t M, int64_t K, int64_t N, termezo_dtype ydt) {
  return ydt == TERMEZO_BF16 && M % kDmaBM == 0 && N % kDmaBN == 0 && K % kBK == 0 && M > 0 &&
         K > 0;
}

// Two blocks per compute unit (128 x 256 tiles) measured faster than the 256 x 256
// grid with a quarter-tile tail when the 256 x 256 grid is below one round of compute
// units (M = 2048: 1.2-1.4x) or spans at least three rounds (gate|up at the 2B shape:
// 1.04-1.07x), and slower in between (1.25 and 1.9 rounds: 0.9x).
static bool use_half_tiles(int64_t M, int64_t T, int n_cu) {
  return n_cu > 0 && M % kHalfBM == 0 && (T < n_cu || T >= 3 * (int64_t)n_cu);
}

// Launch plan of the full-tile path: blocks [0, full) take 256 x 256 tiles, the rest take
// quarters of the remaining ones.
static int64_t dma_full_tiles(int64_t T, int n_cu) {
  int64_t full = T;
  if (n_cu > 0 && T > n_cu) {
    const int64_t rem = T % n_cu;
    if (rem > 0 && 2 * rem <= n_cu) full = T - rem;
  }
  return full;
}

hipError_t launch_gemm_i8(const int8_t* xq, const float* s, const int32_t* rs, const uint32_t* codes,
                          int64_t M,
                          int64_t K, int64_t N, const GemmOut& out, termezo_dtype ydt, int mode,
                          int32_t* acc, int n_cu, hipStream_t st, LaunchEvents ev) {
  // the full-tile paths read the row sums, four tokens per 16-byte load
  if (M > kGemvMaxM && (!rs || reinterpret_cast<uintptr_t>(rs) % 16 != 0)) return hipErrorInvalidValue;
  if (mode == kGemmSwiGLU) {
    if (!gemm_swiglu_ok(M, K, N, ydt) || out.nseg != 2 || out.nstart[1] * 2 != N || acc ||
        out.ld[0] % 8 != 0 || reinterpret_cast<uintptr_t>(out.y[0]) % 16 != 0)
      return hipErrorInvalidValue;
    // always the two-blocks-per-CU tiles: their waves are 64 columns wide, the gate and
    // the up block of 32 features each
    const int64_t T = (M / kHalfBM) * (N / kHalfBN);
    hipExtLaunchKernelGGL((k_gemm_i8_dma_h<uint16_t, kGemmSwiGLU>), dim3((unsigned)T), dim3(256), 0,
                          st, ev.start, ev.stop, 0, xq, s, rs, codes, M, K, N, out, acc);
    return hipGetLastError();
  }
  if (M <= kGemvMaxM) {
    bool seg16 = true;
    for (int i = 1; i < out.nseg; ++i) seg16 = seg16 && out.nstart[i] % 16 == 0;
    if (seg16) {
      const int cvec = (K / 16) % 4 == 0 && reinterpret_cast<uintptr_t>(codes) % 16 == 0;
      const uintptr_t vec = ydt == TERMEZO_F32 ? 16 : 8;   // 4-element store width
      int yvec = 1;
      for (int i = 0; i < out.nseg; ++i)
        yvec = yvec && out.ld[i] % 4 == 0 && reinterpret_cast<uintptr_t>(out.y[i]) % vec == 0;
      dim3 grid((unsigned)((N + 15) / 16));
      // up to 16 tokens: one token group, 8192 k per pass; more: 8 groups, 4096 k
#define TMZ_GEMV(TY, MD, CV)                                                                    \
  do {                                                                                          \
    if (M <= 16)                                                                                \
      hipExtLaunchKernelGGL((k_gemv_i8<TY, MD, CV, 1, 4>), grid, dim3(512), 0, st, ev.start,    \
                            ev.stop, 0, xq, s, codes, M, K, N, out, yvec, acc);                 \
    else                                                                                        \
      hipExtLaunchKernelGGL((k_gemv_i8<TY, MD, CV, kGemvMaxM / 16, 2>), grid, dim3(512), 0, st, \
                            ev.start, ev.stop, 0, xq, s, codes, M, K, N, out, yvec, acc);       \
  } while (0)
      const bool f32 = ydt == TERMEZO_F32, store = mode == kGemmStore;
      if (cvec) {
        if (f32) { if (store) TMZ_GEMV(float, kGemmStore, true); else TMZ_GEMV(float, kGemmResidual, true); }
        else { if (store) TMZ_GEMV(uint16_t, kGemmStore, true); else TMZ_GEMV(uint16_t, kGemmResidual, true); }
      } else {
        if (f32) { if (store) TMZ_GEMV(float, kGemmStore, false); else TMZ_GEMV(float, kGemmResidual, false); }
        else { if (store) TMZ_GEMV(uint16_t, kGemmStore, false); else TMZ_GEMV(uint16_t, kGemmResidual, false); }
      }
#undef TMZ_GEMV
      return hipGetLastError();
    }
  }
  const int64_t big_blocks = ((M + 255) / 256) * ((N + 255) / 256);
  bool seg32 = true;
  for (int i = 1; i < out.nseg; ++i) seg32 = seg32 && out.nstart[i] % 32 == 0;
  const int64_t ue = ydt == TERMEZO_F32 ? 4 : 8;       // outputs per 16-byte unit
  for (int i = 0; i < out.nseg; ++i)
    seg32 = seg32 && out.ld[i] % ue == 0 && reinterpret_cast<uintptr_t>(out.y[i]) % 16 == 0;
  const bool dma = M % 256 == 0 && N % 256 == 0 && K % kBK == 0 && seg32;
  if (big_blocks >= 256 || (dma && n_cu > 0)) {
    if (dma) {
      const int64_t T = big_blocks;
      if (use_half_tiles(M, T, n_cu)) {
        dim3 gh((unsigned)(2 * T));
#define TMZ_HALF(TY, MD) \
  hipExtLaunchKernelGGL((k_gemm_i8_dma_h<TY, MD>), gh, dim3(256), 0, st, ev.start, ev.stop, 0, xq, s, rs, \
                        codes, M, K, N, out, acc)
        if (ydt == TERMEZO_F32) {
          if (mode == kGemmStore) TMZ_HALF(float, kGemmStore); else TMZ_HALF(float, kGemmResidual);
        } else {
          if (mode == kGemmStore) TMZ_HALF(uint16_t, kGemmStore); else TMZ_HALF(uint16_t, kGemmResidual);
        }
#undef TMZ_HALF
        return hipGetLastError();
      }
      // fewer full tiles than compute units: every tile as four 128 x 128 quarters
      const int64_t full = T < n_cu ? 0 : dma_full_tiles(T, n_cu);
      dim3 grid((unsigned)(full + 4 * (T - full)));
#define TMZ_DMA(TY, MD, BK) \
  hipExtLaunchKernelGGL((k_gemm_i8_dma<TY, MD, BK>), grid, dim3(512), 0, st, ev.start, ev.stop, 0, xq, s, \
                        rs, codes, M, K, N, out, full, acc)
#define TMZ_DMA_K(TY, MD) \
  do {                                                 \
    if (K % 256 == 0) TMZ_DMA(TY, MD, 256); else TMZ_DMA(TY, MD, 128); \
  } while (0)
      if (ydt == TERMEZO_F32) {
        if (mode == kGemmStore) TMZ_DMA_K(float, kGemmStore); else TMZ_DMA_K(float, kGemmResidual);
      } else {
        if (mode == kGemmStore) TMZ_DMA_K(uint16_t, kGemmStore); else TMZ_DMA_K(uint16_t, kGemmResidual);
      }
#undef TMZ_DMA_K
#undef TMZ_DMA
      return hipGetLastError();
    }
    return launch_tile<256, 256, 128, 64, false>(xq, s, codes, M, K, N, out, ydt, mode, acc, st, ev);
  }
  return launch_tile<128, 128, 64, 64, false>(xq, s, codes, M, K, N, out, ydt, mode, acc, st, ev);
}

hipError_t launch_bitlinear_gemm(const int8_t* xq, const float* s, const int32_t* rs,
                                 const uint32_t* codes,
                                 const float* beta_dev, int64_t M, int64_t K, int64_t N, void* y,
                                 termezo_dtype ydt, int32_t* acc, int n_cu, hipStream_t st) {
  GemmOut out = {};
  out.nseg = 1;
  out.y[0] = y;
  out.ld[0] = N;
  out.beta[0] = beta_dev;
  out.nstart[0] = 0;
  out.nstart[1] = N;
  return launch_gemm_i8(xq, s, rs, codes, M, K, N, out, ydt, kGemmStore, acc, n_cu, st);
}

}  // namespace tmz
