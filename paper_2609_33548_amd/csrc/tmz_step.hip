// Streaming and sparse kernels of the TerMeZO step on gfx950:
//   absmean sums and thresholds (Sec. 3, eq. quant),
//   global radix selection of the boundary band (eq. distance, eq. selection_init),
//   stable compaction of the active index lists,
//   seed-regenerated perturbation with exact |w'| sum deltas (Algorithm 1),
//   dense requantisation to packed 2-bit codes and sparse code patching,
//   masked update and shrink-only set update (Algorithm 1, eq. selection_).
#include "tmz_device.h"
#include "tmz_internal.h"

namespace tmz {

// ---------------------------------------------------------------------------
// Latent loads: 16 consecutive elements (64 B fp32 or 32 B bf16) as fp32.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void load16(const float* p, float v[16]) {
  const float4* q = reinterpret_cast<const float4*>(p);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float4 a = q[i];
    v[4 * i + 0] = a.x;
    v[4 * i + 1] = a.y;
    v[4 * i + 2] = a.z;
    v[4 * i + 3] = a.w;
  }
}

__device__ __forceinline__ void load16(const uint16_t* p, float v[16]) {
  const uint4* q = reinterpret_cast<const uint4*>(p);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const uint4 a = q[i];
    const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[8 * i + 2 * j + 0] = __uint_as_float(w[j] << 16);
      v[8 * i + 2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
    }
  }
}

__device__ __forceinline__ float load1(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float load1(const uint16_t* p, int64_t i) { return bf16_to_f32(p[i]); }
__device__ __forceinline__ void store1(float* p, int64_t i, float v) { p[i] = v; }
__device__ __forceinline__ void store1(uint16_t* p, int64_t i, float v) { p[i] = f32_to_bf16_rne(v); }
__device__ __forceinline__ float storage_round(const float*, float v) { return v; }
__device__ __forceinline__ float storage_round(const uint16_t*, float v) {
  return bf16_to_f32(f32_to_bf16_rne(v));
}

// ---------------------------------------------------------------------------
// Wave / block reductions (wave64).
// ---------------------------------------------------------------------------
__device__ __forceinline__ unsigned long long wave_sum_u64(unsigned long long v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)v, off, 64);
    const uint32_t hi = __shfl_xor((uint32_t)(v >> 32), off, 64);
    v += ((unsigned long long)hi << 32) | lo;
  }
  return v;
}

__device__ __forceinline__ long long wave_sum_i64(long long v) {
  return (long long)wave_sum_u64((unsigned long long)v);
}

// Block-wide sum of a u64 (blockDim.x == 256).  All threads must call.
__device__ unsigned long long block_sum_u64(unsigned long long v, unsigned long long* lds4) {
  v = wave_sum_u64(v);
  const int wid = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (lane == 0) lds4[wid] = v;
  __syncthreads();
  unsigned long long r = lds4[0] + lds4[1] + lds4[2] + lds4[3];
  __syncthreads();
  return r;
}

// Exclusive prefix sum over a 256-thread block of int64 values; returns the
// exclusive prefix and writes the block total to *total.
__device__ long long block_excl_scan_i64(long long v, long long* lds, long long* total) {
  const int tid = threadIdx.x;
  lds[tid] = v;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {
    long long add = tid >= off ? lds[tid - off] : 0;
    __syncthreads();
    lds[tid] += add;
    __syncthreads();
  }
  const long long incl = lds[tid];
  *total = lds[255];
  __syncthreads();
  return incl - v;
}

// Layer of active-list position j: largest l with act_off[l] <= j (L layers).
__device__ __forceinline__ int layer_of(const int64_t* act_off, int L, int64_t j) {
  int lo = 0, hi = L - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (act_off[mid] <= j) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Flush a per-lane (layer, delta) partial into S[layer]: one atomic per wave
// when every active lane holds the same layer, per-lane atomics otherwise.
__device__ __forceinline__ void flush_delta(long long* S, int layer, long long d, bool valid) {
  const unsigned long long vm = __ballot(valid);
  if (vm == 0ull) return;
  const int first = __shfl(layer, __builtin_ffsll((long long)vm) - 1, 64);
  const bool uniform = __ballot(valid && layer != first) == 0ull;
  if (uniform) {
    const long long t = wave_sum_i64(valid ? d : 0);
    if ((threadIdx.x & 63) == 0 && t != 0)
      atomicAdd((unsigned long long*)&S[first], (unsigned long long)t);
  } else if (valid && d != 0) {
    atomicAdd((unsigned long long*)&S[layer], (unsigned long long)d);
  }
}

// ---------------------------------------------------------------------------
// Fixed-point |w| sums, one contiguous range of tiles per block.
// ---------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) k_abs_sum(DevState st, int64_t* S_out, int64_t tpb) {
  __shared__ unsigned long long red[4];
  const int64_t t0 = (int64_t)blockIdx.x * tpb;
  const int64_t t1 = min(st.T, t0 + tpb);
  unsigned long long acc = 0;
  int cur = -1;
  bool bad = false;
  for (int64_t t = t0; t < t1; ++t) {
    const int l = st.tile_layer[t];
    if (l != cur) {
      if (cur >= 0) {
        const unsigned long long s = block_sum_u64(acc, red);
        if (threadIdx.x == 0 && s) atomicAdd((unsigned long long*)&S_out[cur], s);
      }
      acc = 0;
      cur = l;
    }
    const int64_t start = st.tile_start[t];
    const int64_t cnt = min((int64_t)kTile, st.n[l] - start);
    const T* w = reinterpret_cast<const T*>(st.w[l]) + start;
    for (int64_t e = (int64_t)threadIdx.x * 16; e < cnt; e += 256 * 16) {
      float v[16];
      load16(w + e, v);
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        bad |= !in_fix_range(v[j]);
        acc += fix_abs(v[j]);
      }
    }
  }
  if (cur >= 0) {
    const unsigned long long s = block_sum_u64(acc, red);
    if (threadIdx.x == 0 && s) atomicAdd((unsigned long long*)&S_out[cur], s);
  }
  if (bad) atomicOr(st.err, 1);
}

// tau = fp32(0.5 (S 2^-36 / n + delta)), beta = fp32(S 2^-36 / n + delta).
__global__ void k_thresholds(const int64_t* S, const int64_t* n, float delta, float* tau,
                             float* beta, int L) {
  const int l = blockIdx.x * blockDim.x + threadIdx.x;
  if (l >= L) return;
  const double gamma = ((double)S[l] * 0x1p-36) / (double)n[l];
  const double b = gamma + (double)delta;
  beta[l] = (float)b;
  tau[l] = (float)(0.5 * b);
}

__global__ void k_fill_u64(unsigned long long* p, int64_t n, unsigned long long v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

__global__ void k_copy_i64(int64_t* dst, const int64_t* src, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

// ---------------------------------------------------------------------------
// Radix selection of xi0 over the distance keys.  d >= 0, so its fp32 bit
// pattern is a monotone uint32 key.  Pass p histograms 11/11/10 bits of the
// keys whose higher bits equal the prefix fixed by the earlier passes.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t dist_key(float w, float tau) {
  return __float_as_uint(fabsf(fabsf(w) - tau));
}

template <typename T>
__global__ void __launch_bounds__(256) k_hist(DevState st, int pass, const SelectState* sel,
                                              unsigned long long* hist, int64_t tpb) {
  __shared__ uint32_t h[kHistBins];
  for (int i = threadIdx.x; i < kHistBins; i += 256) h[i] = 0;
  __syncthreads();
  const uint32_t prefix = sel->prefix;
  const int64_t t0 = (int64_t)blockIdx.x * tpb;
  const int64_t t1 = min(st.T, t0 + tpb);
  for (int64_t t = t0; t < t1; ++t) {
    const int l = st.tile_layer[t];
    const float tau = st.tau[l];
    const int64_t start = st.tile_start[t];
    const int64_t cnt = min((int64_t)kTile, st.n[l] - start);
    const T* w = reinterpret_cast<const T*>(st.w[l]) + start;
    for (int64_t e = (int64_t)threadIdx.x * 16; e < cnt; e += 256 * 16) {
      float v[16];
      load16(w + e, v);
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const uint32_t key = dist_key(v[j], tau);
        if (pass == 0) {
          atomicAdd(&h[key >> 21], 1u);
        } else if (pass == 1) {
          if ((key >> 21) == (prefix >> 21)) atomicAdd(&h[(key >> 10) & 0x7FFu], 1u);
        } else {
          if ((key >> 10) == (prefix >> 10)) atomicAdd(&h[key & 0x3FFu], 1u);
        }
      }
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kHistBins; i += 256)
    if (h[i]) atomicAdd(&hist[i], (unsigned long long)h[i]);
}

// Find the bucket holding the k0-th key, extend the prefix, clear the histogram.
__global__ void k_select_bucket(SelectState* sel, unsigned long long* hist, int pass) {
  if (threadIdx.x == 0) {
    const unsigned long long need = sel->k0 - sel->less;
    unsigned long long c = 0;
    uint32_t b = 0;
    const uint32_t nb = pass == 2 ? 1024u : 2048u;
    for (b = 0; b < nb; ++b) {
      if (c + hist[b] >= need) break;
      c += hist[b];
    }
    sel->less += c;
    const int shift = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
    sel->prefix |= b << shift;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kHistBins; i += blockDim.x) hist[i] = 0;
}

__global__ void k_select_init(SelectState* sel, unsigned long long k0) {
  sel->k0 = k0;
  sel->less = 0;
  sel->prefix = 0;
  sel->pad = 0;
}

// ---------------------------------------------------------------------------
// Mask compaction: per-tile counts, single-block scan, ordered write.
// ---------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) k_mask_count(DevState st, const SelectState* sel,
                                                    uint32_t* tile_cnt) {
  __shared__ unsigned long long red[4];
  const uint32_t xi = sel->prefix;
  for (int64_t t = blockIdx.x; t < st.T; t += gridDim.x) {
    const int l = st.tile_layer[t];
    const float tau = st.tau[l];
    const int64_t start = st.tile_start[t];
    const int64_t cnt = min((int64_t)kTile, st.n[l] - start);
    const T* w = reinterpret_cast<const T*>(st.w[l]) + start;
    uint32_t nl = 0, ne = 0;
    for (int64_t e = (int64_t)threadIdx.x * 16; e < cnt; e += 256 * 16) {
      float v[16];
      load16(w + e, v);
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const uint32_t key = dist_key(v[j], tau);
        nl += key < xi;
        ne += key == xi;
      }
    }
    const unsigned long long s = block_sum_u64(((unsigned long long)ne << 32) | nl, red);
    if (threadIdx.x == 0) {
      tile_cnt[2 * t] = (uint32_t)s;
      tile_cnt[2 * t + 1] = (uint32_t)(s >> 32);
    }
  }
}

// One block of 256 threads: per tile, equal-keys-before and output offsets;
// per layer, the first output position.
__global__ void __launch_bounds__(256) k_mask_scan(const SelectState* sel, const uint32_t* tile_cnt,
                                                   const int32_t* tile_layer, int64_t T, int L,
                                                   int inclusive, int64_t* tile_out,
                                                   int64_t* tile_eqb, int64_t* act_off) {
  __shared__ long long lds[256];
  const int64_t need = (int64_t)(sel->k0 - sel->less);  // equal keys to admit (exact-k)
  const int64_t per = (T + 255) / 256;
  const int64_t a = min(T, (int64_t)threadIdx.x * per), b = min(T, a + per);
  long long tot;
  long long eq = 0;
  for (int64_t t = a; t < b; ++t) eq += tile_cnt[2 * t + 1];
  long long eqb = block_excl_scan_i64(eq, lds, &tot);
  long long sel_sum = 0;
  for (int64_t t = a; t < b; ++t) {
    const long long e = tile_cnt[2 * t + 1];
    const long long q = inclusive ? e : max(0ll, min(e, (long long)need - eqb));
    tile_eqb[t] = eqb;
    sel_sum += (long long)tile_cnt[2 * t] + q;
    eqb += e;
  }
  long long off = block_excl_scan_i64(sel_sum, lds, &tot);
  for (int64_t t = a; t < b; ++t) {
    const long long e = tile_cnt[2 * t + 1];
    const long long q = inclusive ? e : max(0ll, min(e, (long long)need - tile_eqb[t]));
    tile_out[t] = off;
    if (t == 0 || tile_layer[t] != tile_layer[t - 1]) act_off[tile_layer[t]] = off;
    off += (long long)tile_cnt[2 * t] + q;
  }
  if (threadIdx.x == 0) act_off[L] = tot;
}

// Ordered write: every thread owns 32 consecutive elements of the tile.
template <typename T>
__global__ void __launch_bounds__(256) k_mask_write(DevState st, const SelectState* sel,
                                                    const uint32_t* tile_cnt,
                                                    const int64_t* tile_out,
                                                    const int64_t* tile_eqb, int inclusive,
                                                    uint32_t* act) {
  __shared__ long long lds[256];
  const uint32_t xi = sel->prefix;
  const int64_t need = (int64_t)(sel->k0 - sel->less);
  for (int64_t t = blockIdx.x; t < st.T; t += gridDim.x) {
    const int l = st.tile_layer[t];
    const float tau = st.tau[l];
    const int64_t start = st.tile_start[t];
    const int64_t cnt = min((int64_t)kTile, st.n[l] - start);
    const T* w = reinterpret_cast<const T*>(st.w[l]) + start;
    const int64_t e0 = (int64_t)threadIdx.x * 32;
    uint32_t lmask = 0, emask = 0;
    for (int h = 0; h < 2; ++h) {
      const int64_t e = e0 + 16 * h;
      if (e < cnt) {
        float v[16];
        load16(w + e, v);
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const uint32_t key = dist_key(v[j], tau);
          lmask |= (uint32_t)(key < xi) << (16 * h + j);
          emask |= (uint32_t)(key == xi) << (16 * h + j);
        }
      }
    }
    long long tot;
    const long long packed = ((long long)__popc(emask) << 32) | __popc(lmask);
    const long long pre = block_excl_scan_i64(packed, lds, &tot);
    long long lb = pre & 0xFFFFFFFFll, eb = pre >> 32;
    const long long etile = tile_cnt[2 * t + 1];
    const long long quota = inclusive ? etile : max(0ll, min(etile, (long long)need - tile_eqb[t]));
    const int64_t base = tile_out[t];
    for (int j = 0; j < 32; ++j) {
      const uint32_t bit = 1u << j;
      if (lmask & bit) {
        act[base + lb + min(eb, quota)] = (uint32_t)(start + e0 + j);
        ++lb;
      } else if (emask & bit) {
        if (eb < quota) act[base + lb + eb] = (uint32_t)(start + e0 + j);
        ++eb;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Dense requantisation of every layer with its current threshold.
// ---------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) k_requant(DevState st, int64_t tpb) {
  const int64_t t0 = (int64_t)blockIdx.x * tpb;
  const int64_t t1 = min(st.T, t0 + tpb);
  for (int64_t t = t0; t < t1; ++t) {
    const int l = st.tile_layer[t];
    const float tau = st.tau_cur[l];
    const int64_t start = st.tile_start[t];
    const int64_t cnt = min((int64_t)kTile, st.n[l] - start);
    const T* w = reinterpret_cast<const T*>(st.w[l]) + start;
    uint32_t* out = st.codes + st.code_off[l] + start / 16;
    for (int64_t e = (int64_t)threadIdx.x * 16; e < cnt; e += 256 * 16) {
      float v[16];
      load16(w + e, v);
      uint32_t word = 0;
#pragma unroll
      for (int j = 0; j < 16; ++j) word |= ternary_code(v[j], tau) << code_shift(j);
      out[e / 16] = word;
    }
  }
}

// ---------------------------------------------------------------------------
// Perturbation at the actives: w' = fma(se, z, w), stored compactly; the
// exact change of the fixed-point |w| sum goes to S_cur (initialised to
// S_clean by the caller).  Each thread walks kRun consecutive entries.
// ---------------------------------------------------------------------------
constexpr int kRun = 4;

template <typename T>
__global__ void __launch_bounds__(256) k_perturb_delta(DevState st, const uint32_t* act,
                                                       const int64_t* act_off, uint64_t seed,
                                                       float se, float* wp) {
  const int64_t k = act_off[st.L];
  const int64_t j0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * kRun;
  int l = j0 < k ? layer_of(act_off, st.L, j0) : 0;
  long long acc = 0;
  bool bad = false, any = false;
  for (int r = 0; r < kRun; ++r) {
    const int64_t j = j0 + r;
    if (j >= k) break;
    if (act_off[l + 1] <= j) {              // the run crosses into a later layer
      if (any) atomicAdd((unsigned long long*)&st.S_cur[l], (unsigned long long)acc);
      acc = 0;
      while (act_off[l + 1] <= j) ++l;
    }
    const uint32_t i = act[j];
    const float wv = load1(reinterpret_cast<const T*>(st.w[l]), i);
    const float v = se != 0.0f ? fmaf(se, gauss_at(seed, (uint64_t)(st.gid0[l] + i)), wv) : wv;
    wp[j] = v;
    bad |= !in_fix_range(v);
    acc += (long long)fix_abs(v) - (long long)fix_abs(wv);
    any = true;
  }
  flush_delta((long long*)st.S_cur, l, acc, any);
  if (bad) atomicOr(st.err, 1);
}

// Sparse code patch at the actives with the current threshold.
__global__ void __launch_bounds__(256) k_patch_codes(DevState st, const uint32_t* act,
                                                     const int64_t* act_off, const float* wp) {
  const int64_t k = act_off[st.L];
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= k) return;
  const int l = layer_of(act_off, st.L, j);
  const uint32_t i = act[j];
  uint32_t* word = st.codes + st.code_off[l] + i / 16;
  const int sh = code_shift((int)(i & 15u));
  const uint32_t code = ternary_code(wp[j], st.tau_cur[l]);
  atomicAnd(word, ~(3u << sh));
  if (code) atomicOr(word, code << sh);
}

// ---------------------------------------------------------------------------
// Masked update: w_i <- round(fma(a, z_i, w_i)), a = -(lr g); exact delta of
// the clean fixed-point sum.
// ---------------------------------------------------------------------------
__global__ void k_set_coeff(float* scal, float a) {
  scal[0] = a;
  scal[1] = 0.0f;
}

// g = (F+ - F-) / (2 eps) and a = -(lr g), in fp32 (eq. spsa).
__global__ void k_coeff_from_losses(const float* fp, const float* fm, float eps, float lr,
                                    float* scal, int32_t* err) {
  const float g = __fdiv_rn(*fp - *fm, 2.0f * eps);
  const float a = -(lr * g);
  scal[0] = a;
  scal[1] = g;
  if (!isfinite(a)) atomicOr(err, 2);
}

template <typename T>
__global__ void __launch_bounds__(256) k_update(DevState st, const uint32_t* act,
                                                const int64_t* act_off, uint64_t seed,
                                                const float* scal) {
  const float a = scal[0];
  if (!isfinite(a)) return;   // reported by the coefficient kernel; latents untouched
  const int64_t k = act_off[st.L];
  const int64_t j0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * kRun;
  int l = j0 < k ? layer_of(act_off, st.L, j0) : 0;
  long long acc = 0;
  bool bad = false, any = false;
  for (int r = 0; r < kRun; ++r) {
    const int64_t j = j0 + r;
    if (j >= k) break;
    if (act_off[l + 1] <= j) {
      if (any) atomicAdd((unsigned long long*)&st.S_clean[l], (unsigned long long)acc);
      acc = 0;
      while (act_off[l + 1] <= j) ++l;
    }
    const uint32_t i = act[j];
    T* w = reinterpret_cast<T*>(const_cast<void*>(st.w[l]));
    const float wv = load1(w, i);
    const float nv = storage_round(w, fmaf(a, gauss_at(seed, (uint64_t)(st.gid0[l] + i)), wv));
    store1(w, i, nv);
    bad |= !in_fix_range(nv);
    acc += (long long)fix_abs(nv) - (long long)fix_abs(wv);
    any = true;
  }
  flush_delta((long long*)st.S_clean, l, acc, any);
  if (bad) atomicOr(st.err, 1);
}

// ---------------------------------------------------------------------------
// Shrink-only set update: keep the actives with ||w| - tau| <= xi0.
// Block b handles entries [b * kShrinkBlk, (b+1) * kShrinkBlk).
// ---------------------------------------------------------------------------
constexpr int kShrinkPer = 16;
constexpr int kShrinkBlk = 256 * kShrinkPer;

template <typename T>
__device__ __forceinline__ uint32_t shrink_flags(const DevState& st, const uint32_t* act,
                                                 const int64_t* act_off, int64_t k, int64_t j0,
                                                 float xi0) {
  uint32_t m = 0;
  if (j0 >= k) return 0;
  int l = layer_of(act_off, st.L, j0);
  for (int r = 0; r < kShrinkPer; ++r) {
    const int64_t j = j0 + r;
    if (j >= k) break;
    while (act_off[l + 1] <= j) ++l;
    const uint32_t i = act[j];
    const float wv = load1(reinterpret_cast<const T*>(st.w[l]), i);
    if (fabsf(fabsf(wv) - st.tau[l]) <= xi0) m |= 1u << r;
  }
  return m;
}

template <typename T>
__global__ void __launch_bounds__(256) k_shrink_count(DevState st, const uint32_t* act,
                                                      const int64_t* act_off, float xi0,
                                                      int64_t* blk_cnt) {
  __shared__ unsigned long long red[4];
  const int64_t k = act_off[st.L];
  const int64_t j0 = (int64_t)blockIdx.x * kShrinkBlk + (int64_t)threadIdx.x * kShrinkPer;
  const uint32_t m = shrink_flags<T>(st, act, act_off, k, j0, xi0);
  const unsigned long long s = block_sum_u64(__popc(m), red);
  if (threadIdx.x == 0) blk_cnt[blockIdx.x] = (int64_t)s;
}

__global__ void __launch_bounds__(256) k_blocks_scan(int64_t* blk_cnt, int64_t nb, int64_t* total) {
  __shared__ long long lds[256];
  const int64_t per = (nb + 255) / 256;
  const int64_t a = min(nb, (int64_t)threadIdx.x * per), b = min(nb, a + per);
  long long s = 0;
  for (int64_t i = a; i < b; ++i) s += blk_cnt[i];
  long long tot;
  long long off = block_excl_scan_i64(s, lds, &tot);
  for (int64_t i = a; i < b; ++i) {
    const long long c = blk_cnt[i];
    blk_cnt[i] = off;
    off += c;
  }
  if (threadIdx.x == 0) *total = tot;
}

template <typename T>
__global__ void __launch_bounds__(256) k_shrink_write(DevState st, const uint32_t* act,
                                                      const int64_t* act_off, float xi0,
                                                      const int64_t* blk_off, uint32_t* act_new,
                                                      int64_t* act_off_new) {
  __shared__ long long lds[256];
  const int64_t k = act_off[st.L];
  const int64_t j0 = (int64_t)blockIdx.x * kShrinkBlk + (int64_t)threadIdx.x * kShrinkPer;
  const uint32_t m = shrink_flags<T>(st, act, act_off, k, j0, xi0);
  long long tot;
  long long pos = blk_off[blockIdx.x] + block_excl_scan_i64(__popc(m), lds, &tot);
  if (j0 >= k) return;
  int l = layer_of(act_off, st.L, j0);
  for (int r = 0; r < kShrinkPer; ++r) {
    const int64_t j = j0 + r;
    if (j >= k) break;
    while (act_off[l + 1] <= j) ++l;
    if (j == act_off[l]) act_off_new[l] = pos;   // first entry of layer l
    if (m & (1u << r)) act_new[pos++] = act[j];
  }
}

// Layers that were empty before the shrink take the next layer's offset.
__global__ void k_shrink_offsets(const int64_t* act_off, int64_t* act_off_new, int L,
                                 const int64_t* total) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  act_off_new[L] = *total;
  for (int l = L - 1; l >= 0; --l)
    if (act_off[l] == act_off[l + 1]) act_off_new[l] = act_off_new[l + 1];
}

// ---------------------------------------------------------------------------
// Inspection: unpack one layer's codes to int8.
// ---------------------------------------------------------------------------
__global__ void k_unpack(const uint32_t* codes, int64_t n, int8_t* out) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t word = codes[i / 16];
    const uint32_t c = (word >> code_shift((int)(i & 15))) & 3u;
    out[i] = c == 1u ? 1 : (c == 3u ? -1 : 0);
  }
}

__global__ void k_gauss(uint64_t seed, const uint64_t* gids, int64_t n, float* z) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    z[i] = gauss_at(seed, gids[i]);
}

hipError_t launch_gauss(uint64_t seed, const uint64_t* gids, int64_t n, float* z, hipStream_t s) {
  const int64_t g = max((int64_t)1, min((int64_t)4096, (n + 255) / 256));
  hipLaunchKernelGGL(k_gauss, dim3(g), dim3(256), 0, s, seed, gids, n, z);
  return hipGetLastError();
}

// Config-1 loss: one block, fixed reduction order (deterministic).
__global__ void __launch_bounds__(256) k_mse(const float* y, const float* t, int64_t n,
                                             double* out) {
  __shared__ double lds[256];
  double acc = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += 256) {
    const float e = y[i] - t[i];
    const float e2 = e * e;
    acc += (double)e2;
  }
  lds[threadIdx.x] = acc;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off) lds[threadIdx.x] += lds[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = lds[0];
}

// ===========================================================================
// Launchers
// ===========================================================================
static inline int64_t grid_for(int64_t T, int64_t target, int64_t* tpb) {
  const int64_t g = max((int64_t)1, min(T, target));
  *tpb = (T + g - 1) / g;
  return (T + *tpb - 1) / *tpb;
}

hipError_t launch_abs_sum(termezo_ctx* c, int64_t* S_out) {
  int64_t tpb;
  const int64_t g = grid_for(c->T, 2048, &tpb);
  hipError_t e = launch_fill_u64((unsigned long long*)S_out, c->L, 0, c->stream);
  if (e != hipSuccess) return e;
  if (c->dtype == TERMEZO_F32)
    hipLaunchKernelGGL(k_abs_sum<float>, dim3(g), dim3(256), 0, c->stream, c->dev(), S_out, tpb);
  else
    hipLaunchKernelGGL(k_abs_sum<uint16_t>, dim3(g), dim3(256), 0, c->stream, c->dev(), S_out, tpb);
  return hipGetLastError();
}

hipError_t launch_thresholds(termezo_ctx* c, const int64_t* S, float* tau, float* beta) {
  hipLaunchKernelGGL(k_thresholds, dim3((c->L + 255) / 256), dim3(256), 0, c->stream, S, c->d_n,
                     c->delta, tau, beta, c->L);
  return hipGetLastError();
}

hipError_t launch_fill_u64(unsigned long long* p, int64_t n, unsigned long long v, hipStream_t s) {
  const int64_t g = max((int64_t)1, min((int64_t)1024, (n + 255) / 256));
  hipLaunchKernelGGL(k_fill_u64, dim3(g), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

hipError_t launch_copy_i64(int64_t* dst, const int64_t* src, int64_t n, hipStream_t s) {
  const int64_t g = max((int64_t)1, min((int64_t)1024, (n + 255) / 256));
  hipLaunchKernelGGL(k_copy_i64, dim3(g), dim3(256), 0, s, dst, src, n);
  return hipGetLastError();
}

hipError_t launch_select(termezo_ctx* c, int64_t k0) {
  hipLaunchKernelGGL(k_select_init, dim3(1), dim3(1), 0, c->stream, c->d_sel,
                     (unsigned long long)k0);
  hipError_t e = launch_fill_u64(c->d_hist, kHistBins, 0, c->stream);
  if (e != hipSuccess) return e;
  int64_t tpb;
  const int64_t g = grid_for(c->T, 2048, &tpb);
  for (int pass = 0; pass < 3; ++pass) {
    if (c->dtype == TERMEZO_F32)
      hipLaunchKernelGGL(k_hist<float>, dim3(g), dim3(256), 0, c->stream, c->dev(), pass, c->d_sel,
                         c->d_hist, tpb);
    else
      hipLaunchKernelGGL(k_hist<uint16_t>, dim3(g), dim3(256), 0, c->stream, c->dev(), pass,
                         c->d_sel, c->d_hist, tpb);
    hipLaunchKernelGGL(k_select_bucket, dim3(1), dim3(256), 0, c->stream, c->d_sel, c->d_hist, pass);
  }
  return hipGetLastError();
}

hipError_t launch_mask_compact_counts(termezo_ctx* c, int inclusive) {
  const int64_t g = max((int64_t)1, min(c->T, (int64_t)8192));
  if (c->dtype == TERMEZO_F32)
    hipLaunchKernelGGL(k_mask_count<float>, dim3(g), dim3(256), 0, c->stream, c->dev(), c->d_sel,
                       c->d_tile_cnt);
  else
    hipLaunchKernelGGL(k_mask_count<uint16_t>, dim3(g), dim3(256), 0, c->stream, c->dev(),
                       c->d_sel, c->d_tile_cnt);
  hipLaunchKernelGGL(k_mask_scan, dim3(1), dim3(256), 0, c->stream, c->d_sel, c->d_tile_cnt,
                     c->d_tile_layer, c->T, c->L, inclusive, c->d_tile_out, c->d_tile_eqb,
                     c->d_act_off);
  return hipGetLastError();
}

hipError_t launch_mask_compact_write(termezo_ctx* c, int inclusive) {
  const int64_t g = max((int64_t)1, min(c->T, (int64_t)8192));
  if (c->dtype == TERMEZO_F32)
    hipLaunchKernelGGL(k_mask_write<float>, dim3(g), dim3(256), 0, c->stream, c->dev(), c->d_sel,
                       c->d_tile_cnt, c->d_tile_out, c->d_tile_eqb, inclusive, c->d_act);
  else
    hipLaunchKernelGGL(k_mask_write<uint16_t>, dim3(g), dim3(256), 0, c->stream, c->dev(),
                       c->d_sel, c->d_tile_cnt, c->d_tile_out, c->d_tile_eqb, inclusive, c->d_act);
  return hipGetLastError();
}

hipError_t launch_requant_dense(termezo_ctx* c) {
  int64_t tpb;
  const int64_t g = grid_for(c->T, 8192, &tpb);
  if (c->dtype == TERMEZO_F32)
    hipLaunchKernelGGL(k_requant<float>, dim3(g), dim3(256), 0, c->stream, c->dev(), tpb);
  else
    hipLaunchKernelGGL(k_requant<uint16_t>, dim3(g), dim3(256), 0, c->stream, c->dev(), tpb);
  return hipGetLastError();
}

hipError_t launch_perturb_delta(termezo_ctx* c, int64_t k, uint64_t seed, float se) {
  if (k <= 0) return hipSuccess;
  const int64_t threads = (k + kRun - 1) / kRun;
  const int64_t g = (threads + 255) / 256;
  if (c->dtype == TERMEZO_F32)
    hipLaunchKernelGGL(k_perturb_delta<float>, dim3(g), dim3(256), 0, c->stream, c->dev(), c->d_act,
                       c->d_act_off, seed, se, c->d_wp);
  else
    hipLaunchKernelGGL(k_perturb_delta<uint16_t>, dim3(g), dim3(256), 0, c->stream, c->dev(),
                       c->d_act, c->d_act_off, seed, se, c->d_wp);
  return hipGetLastError();
}

hipError_t launch_patch_codes(termezo_ctx* c, int64_t k) {
  if (k <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_patch_codes, dim3((k + 255) / 256), dim3(256), 0, c->stream, c->dev(),
                     c->d_act, c->d_act_off, c->d_wp);
  return hipGetLastError();
}

hipError_t launch_set_coeff(termezo_ctx* c, float a) {
  hipLaunchKernelGGL(k_set_coeff, dim3(1), dim3(1), 0, c->stream, c->d_scal, a);
  return hipGetLastError();
}

hipError_t launch_coeff_from_losses(termezo_ctx* c, const float* fp, const float* fm, float eps,
                                    float lr) {
  hipLaunchKernelGGL(k_coeff_from_losses, dim3(1), dim3(1), 0, c->stream, fp, fm, eps, lr,
                     c->d_scal, c->d_err);
  return hipGetLastError();
}

hipError_t launch_update(termezo_ctx* c, int64_t k, uint64_t seed) {
  if (k <= 0) return hipSuccess;
  const int64_t threads = (k + kRun - 1) / kRun;
  const int64_t g = (threads + 255) / 256;
  if (c->dtype == TERMEZO_F32)
    hipLaunchKernelGGL(k_update<float>, dim3(g), dim3(256), 0, c->stream, c->dev(), c->d_act,
                       c->d_act_off, seed, (const float*)c->d_scal);
  else
    hipLaunchKernelGGL(k_update<uint16_t>, dim3(g), dim3(256), 0, c->stream, c->dev(), c->d_act,
                       c->d_act_off, seed, (const float*)c->d_scal);
  return hipGetLastError();
}

hipError_t launch_shrink(termezo_ctx* c, int64_t k) {
  const int64_t nb = max((int64_t)1, (k + kShrinkBlk - 1) / kShrinkBlk);
  int64_t* total = c->d_blk_cnt + nb;  // blk_cap >= nb + 1
  if (c->dtype == TERMEZO_F32)
    hipLaunchKernelGGL(k_shrink_count<float>, dim3(nb), dim3(256), 0, c->stream, c->dev(),
                       c->d_act, c->d_act_off, c->xi0, c->d_blk_cnt);
  else
    hipLaunchKernelGGL(k_shrink_count<uint16_t>, dim3(nb), dim3(256), 0, c->stream, c->dev(),
                       c->d_act, c->d_act_off, c->xi0, c->d_blk_cnt);
  hipLaunchKernelGGL(k_blocks_scan, dim3(1), dim3(256), 0, c->stream, c->d_blk_cnt, nb, total);
  // offsets of layers without any entry are fixed afterwards
  if (c->dtype == TERMEZO_F32)
    hipLaunchKernelGGL(k_shrink_write<float>, dim3(nb), dim3(256), 0, c->stream, c->dev(),
                       c->d_act, c->d_act_off, c->xi0, c->d_blk_cnt, c->d_act_tmp,
                       c->d_act_off_tmp);
  else
    hipLaunchKernelGGL(k_shrink_write<uint16_t>, dim3(nb), dim3(256), 0, c->stream, c->dev(),
                       c->d_act, c->d_act_off, c->xi0, c->d_blk_cnt, c->d_act_tmp,
                       c->d_act_off_tmp);
  hipLaunchKernelGGL(k_shrink_offsets, dim3(1), dim3(1), 0, c->stream, c->d_act_off,
                     c->d_act_off_tmp, c->L, total);
  return hipGetLastError();
}

hipError_t launch_unpack_layer(termezo_ctx* c, int layer, int8_t* out_dev) {
  const tmz::LayerHost& L = c->layers[layer];
  const int64_t g = max((int64_t)1, min((int64_t)4096, (L.n + 255) / 256));
  hipLaunchKernelGGL(k_unpack, dim3(g), dim3(256), 0, c->stream, c->d_codes + L.code_off, L.n,
                     out_dev);
  return hipGetLastError();
}

hipError_t launch_mse(const float* y, const float* t, int64_t n, double* acc, hipStream_t s) {
  hipLaunchKernelGGL(k_mse, dim3(1), dim3(256), 0, s, y, t, n, acc);
  return hipGetLastError();
}

}  // namespace tmz
