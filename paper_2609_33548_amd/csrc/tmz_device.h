// Device-side helpers for the TerMeZO kernels (gfx950).
//
// Everything here is exact integer work or a fixed sequence of correctly
// rounded fp32 operations (the library is compiled with -ffp-contract=off and
// correctly rounded fp32 division/sqrt), so results are reproducible bit for
// bit on any implementation that follows the same definitions.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tmz {

typedef float v2f __attribute__((ext_vector_type(2)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));

// Two floats to a packed pair of bf16 (RNE), low half = a: one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v2f{a, b}, v2bf));
}

// ---------------------------------------------------------------------------
// Counter-based generator: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11).
// Key = 64-bit seed; counter = (q_lo, q_hi, stream, 0).
// ---------------------------------------------------------------------------
struct U4 {
  uint32_t a, b, c, d;
};

__device__ __forceinline__ U4 philox10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                       uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    // full 64-bit products (one v_mad_u64_u32 each instead of a mul_hi / mul_lo pair)
    const uint64_t pA = (uint64_t)0xD2511F53u * c0, pB = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t hA = (uint32_t)(pA >> 32), lA = (uint32_t)pA;
    const uint32_t hB = (uint32_t)(pB >> 32), lB = (uint32_t)pB;
    const uint32_t n0 = hB ^ c1 ^ k0;
    const uint32_t n2 = hA ^ c3 ^ k1;
    c0 = n0;
    c1 = lB;
    c2 = n2;
    c3 = lA;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return U4{c0, c1, c2, c3};
}

// ---------------------------------------------------------------------------
// Natural log for Box-Muller radii, u in (0, 1]: u = m 2^e with
// m in [sqrt(1/2), sqrt(2)); ln m = 2 atanh((m-1)/(m+1)) by its Taylor series
// through the 11th power; ln2 split in an exact high part and a low part.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float ln_unit(float u) {
  uint32_t bits = __float_as_uint(u);
  int ex = int(bits >> 23) - 127;
  uint32_t mant = bits & 0x7FFFFFu;
  uint32_t mb = mant | 0x3F800000u;
  if (mant > 0x3504F3u) {
    mb -= 0x00800000u;
    ex += 1;
  }
  const float m = __uint_as_float(mb);
  const float f = __fdiv_rn(m - 1.0f, m + 1.0f);
  const float f2 = 2.0f * f;
  const float t = f * f;
  float p = fmaf(0x1.745d18p-4f, t, 0x1.c71c72p-4f);  // 1/11, 1/9
  p = fmaf(p, t, 0x1.24924ap-3f);                     // 1/7
  p = fmaf(p, t, 0x1.99999ap-3f);                     // 1/5
  p = fmaf(p, t, 0x1.555556p-2f);                     // 1/3
  const float lm = fmaf(f2 * t, p, f2);
  const float e = (float)ex;
  return fmaf(e, 0x1.62e000p-1f, fmaf(e, 0x1.0bfbe8p-15f, lm));
}

// sin and cos of 2 pi j / 2^24 for a 24-bit integer j: exact reduction to
// the nearest quarter turn, Taylor series of sin(pi r), cos(pi r) on
// |r| <= 1/4, then the quadrant rotation.
__device__ __forceinline__ void sincos_turn24(uint32_t j, float& s, float& c) {
  const uint32_t quad = (j + 0x200000u) >> 22;
  const float r = (float)(int32_t)(j - (quad << 22)) * 0x1p-23f;
  const float t = r * r;
  float ps = fmaf(-0x1.e30750p-8f, t, 0x1.507834p-4f);
  ps = fmaf(ps, t, -0x1.32d2ccp-1f);
  ps = fmaf(ps, t, 0x1.466bc6p+1f);
  ps = fmaf(ps, t, -0x1.4abbcep+2f);
  const float sr = fmaf(r * t, ps, fmaf(r, 0x1.921fb6p+1f, r * -0x1.777a5cp-24f));
  float pc = fmaf(0x1.f9d38ap-10f, t, -0x1.a6d1f2p-6f);
  pc = fmaf(pc, t, 0x1.e1f506p-3f);
  pc = fmaf(pc, t, -0x1.55d3c8p+0f);
  pc = fmaf(pc, t, 0x1.03c1f0p+2f);
  pc = fmaf(pc, t, -0x1.3bd3ccp+2f);
  const float cr = fmaf(t, pc, 1.0f);
  switch (quad & 3u) {
    case 0: s = sr;  c = cr;  break;
    case 1: s = cr;  c = -sr; break;
    case 2: s = -sr; c = -cr; break;
    default: s = -cr; c = sr; break;
  }
}

// Correctly rounded square root of a non-negative normal fp32 x (or of +-0).
// The hardware estimate s is within one ulp; with its neighbours s- and s+,
// the exact residuals x - s- s and x - s+ s (one fma each) decide whether x lies
// below the square of the midpoint (s- + s)/2 or above that of (s + s+)/2 --
// no fp32 x can fall between s- s and that midpoint square, so the tests are
// exact.
__device__ __forceinline__ float sqrt_rn(float x) {
  if (x == 0.0f) return x;               // IEEE: sqrt(+-0) = +-0
  float s = __builtin_amdgcn_sqrtf(x);
  const float sm = __uint_as_float(__float_as_uint(s) - 1u);
  const float sp = __uint_as_float(__float_as_uint(s) + 1u);
  if (fmaf(-sm, s, x) <= 0.0f)
    s = sm;
  else if (fmaf(-sp, s, x) > 0.0f)
    s = sp;
  return s;
}

// One Box-Muller pair from two 32-bit words: radius from xr, angle from xa.
__device__ __forceinline__ void box_muller(uint32_t xr, uint32_t xa, float& zc, float& zs) {
  const float u1 = (float)((xr >> 8) + 1u) * 0x1p-24f;
  const float rad = sqrt_rn(-2.0f * ln_unit(u1));
  float s, c;
  sincos_turn24(xa >> 8, s, c);
  zc = rad * c;
  zs = rad * s;
}

// z for one global id (stream 0 = perturbation directions).
__device__ __forceinline__ float gauss_at(uint64_t seed, uint64_t gid) {
  const uint64_t q = gid >> 2;
  const U4 x = philox10((uint32_t)q, (uint32_t)(q >> 32), 0u, 0u, (uint32_t)seed,
                        (uint32_t)(seed >> 32));
  const uint32_t lane = (uint32_t)gid & 3u;
  const uint32_t xr = lane < 2 ? x.a : x.c;
  const uint32_t xa = lane < 2 ? x.b : x.d;
  float zc, zs;
  box_muller(xr, xa, zc, zs);
  return (lane & 1u) ? zs : zc;
}

// z for a run of global ids: ids of one quad share their Philox call and ids
// of one pair share their Box-Muller evaluation (the same operations as
// gauss_at, so the values are identical).
struct GaussCache {
  uint64_t quad = ~0ull, pair = ~0ull;
  U4 x = {0u, 0u, 0u, 0u};
  float zc = 0.0f, zs = 0.0f;
  __device__ __forceinline__ float get(uint64_t seed, uint64_t gid) {
    const uint64_t p = gid >> 1;
    if (p != pair) {
      const uint64_t q = gid >> 2;
      if (q != quad) {
        x = philox10((uint32_t)q, (uint32_t)(q >> 32), 0u, 0u, (uint32_t)seed, (uint32_t)(seed >> 32));
        quad = q;
      }
      const bool hi = (gid & 2u) != 0;
      box_muller(hi ? x.c : x.a, hi ? x.d : x.b, zc, zs);
      pair = p;
    }
    return (gid & 1u) ? zs : zc;
  }
};

// ---------------------------------------------------------------------------
// Fixed-point |w|: floor(|w| * 2^36) taken from the fp32 bit pattern.
// Valid for |w| < 4 (then the result is below 2^38).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint64_t fix_abs(float w) {
  const uint32_t a = __float_as_uint(w) & 0x7FFFFFFFu;
  const int e = int(a >> 23);
  if (e == 0) return 0ull;                       // zero / subnormal: < 2^-126
  const uint64_t m = (uint64_t)((a & 0x7FFFFFu) | 0x800000u);
  const int sh = e - 114;                        // |w| 2^36 = m 2^(e - 114)
  if (sh >= 0) return m << sh;
  if (sh <= -24) return 0ull;
  return m >> (-sh);
}

// |w| < 4 and finite (4.0f = 0x40800000).
__device__ __forceinline__ bool in_fix_range(float w) {
  return (__float_as_uint(w) & 0x7FFFFFFFu) < 0x40800000u;
}

// ---------------------------------------------------------------------------
// bfloat16 helpers (storage format of bf16 latents and activations).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float v) {
  uint32_t b = __float_as_uint(v);
  if ((b & 0x7F800000u) == 0x7F800000u) {        // inf / nan
    if (b & 0x7FFFFFu) b |= 0x00400000u;
    return (uint16_t)(b >> 16);
  }
  b += 0x7FFFu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}

// ---------------------------------------------------------------------------
// Ternary code and its 2-bit packing.
// Code values: 0 -> 0b00, +1 -> 0b01, -1 -> 0b10.
// A 32-bit word holds 16 codes of one row along d_in; the code at offset
// j = 4 i + b (i, b in 0..3) sits at bits [8 b + 2 i, 8 b + 2 i + 1], so that
// (word >> 2i) & 0x03030303 puts codes 4i..4i+3 in the low bits of bytes 0..3.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t ternary_code(float w, float tau) {
  return w > tau ? 1u : (w < -tau ? 2u : 0u);
}

__device__ __forceinline__ int code_shift(int j) { return 8 * (j & 3) + 2 * (j >> 2); }

// Expand the four codes of group i (offsets 4i..4i+3) to four int8 lanes.
__device__ __forceinline__ uint32_t unpack_group(uint32_t word, int i) {
  const uint32_t sel = (word >> (2 * i)) & 0x03030303u;
  // byte selector 0 -> 0x00, 1 -> 0x01, 2 -> 0xFF
  return __builtin_amdgcn_perm(0u, 0xFFFF0100u, sel);
}

// All 16 codes of a word as four int8 lanes of four (offsets 0..15) with one
// shift: groups 0 and 2 (bits 0-1 of each byte of w and w >> 4) are byte
// selectors 0, 1, 2 into 0x00, 0x01, 0xFF; groups 1 and 3 (bits 2-3), masked in
// place, are selectors 0, 4, 8: byte 0 of the low table (0x00), byte 0 of the
// high table (0x01) and the sign of the low table's byte 1 (0xFF).
__device__ __forceinline__ void unpack_word(uint32_t w, uint32_t out[4]) {
  const uint32_t y = w >> 4;
  out[0] = __builtin_amdgcn_perm(0u, 0x00FF0100u, w & 0x03030303u);
  out[1] = __builtin_amdgcn_perm(0x01u, 0x00008000u, w & 0x0C0C0C0Cu);
  out[2] = __builtin_amdgcn_perm(0u, 0x00FF0100u, y & 0x03030303u);
  out[3] = __builtin_amdgcn_perm(0x01u, 0x00008000u, y & 0x0C0C0C0Cu);
}

// Block order: consecutive workgroups are dealt round-robin to the 8 XCDs
// (each with its own L2).  The linear id is remapped so that each XCD gets a
// contiguous range of tiles, walked in groups of kGroupM block-rows (N
// fastest inside a group), so tiles resident on one XCD share A rows and code
// columns in that XCD's L2.
constexpr int kXcd = 8;
constexpr int kGroupM = 4;

__device__ __forceinline__ int64_t xcd_linear(int64_t b, int64_t total) {
  const int64_t xcd = b % kXcd, local = b / kXcd;
  const int64_t full = total / kXcd, rem = total % kXcd;
  return xcd * full + min(xcd, rem) + local;
}

__device__ __forceinline__ void tile_of_linear(int64_t lb, int64_t nb_m, int64_t nb_n, int64_t& tm,
                                               int64_t& tn) {
  const int64_t span = (int64_t)kGroupM * nb_n;
  const int64_t g = lb / span, in = lb % span;
  const int64_t gm = min((int64_t)kGroupM, nb_m - g * kGroupM);
  tm = g * kGroupM + in % gm;
  tn = in / gm;
}

__device__ __forceinline__ void tile_of_block(int64_t nb_m, int64_t nb_n, int64_t& tm, int64_t& tn) {
  tile_of_linear(xcd_linear(blockIdx.x, nb_m * nb_n), nb_m, nb_n, tm, tn);
}

// silu(g) * u as the decoder evaluates it (hardware exp2 and reciprocal), shared by the
// SwiGLU row kernel and the SwiGLU GEMM epilogue so the two give identical results.
__device__ __forceinline__ float silu_mul(float g, float u) {
  const float sg = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(g * -1.4426950408889634f));
  return g * sg * u;
}

// ---------------------------------------------------------------------------
// Direct global -> LDS loads (gfx950 global_load_lds_dwordx4).
// ---------------------------------------------------------------------------
// One 16-byte-per-lane direct global -> LDS load; lds_base is the wave's
// destination (LDS byte offset, wave-uniform).  Issued as inline assembly so
// that its completion is tracked only by the caller's explicit vmcnt waits
// (the compiler would otherwise wait conservatively).
__device__ __forceinline__ void dma16(const void* gptr, uint32_t lds_base) {
  asm volatile(
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, off"
      :
      : "v"(gptr), "s"(lds_base)
      : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

template <int N>
__device__ __forceinline__ void wait_vmcnt_le() {
  // s_waitcnt vmcnt(N): vmcnt in bits [3:0] and [15:14]; expcnt, lgkmcnt left at their maxima
  static_assert(N >= 0 && N < 16, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (0x7 << 4) | (0xF << 8));
}

}  // namespace tmz
