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

typedef uint32_t v4u __attribute__((ext_vector_type(4)));

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

// The L+1 active-list offsets in LDS (L <= kMaxLayers); all threads call.
__device__ __forceinline__ void load_offsets(int64_t* aoff, const int64_t* act_off, int L) {
  for (int i = threadIdx.x; i <= L; i += blockDim.x) aoff[i] = act_off[i];
  __syncthreads();
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
// Per-tile active ranges: tile_act[t] = first position of the active list
// whose element lies in tile t or a later tile; tile_act[T] = k.  One thread
// per tile, binary search in its layer's part of the list.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) k_tile_ranges(DevState st, const uint32_t* act,
                                                     const int64_t* act_off) {
  __shared__ int64_t aoff[kMaxLayers + 1];
  load_offsets(aoff, act_off, st.L);
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t <= st.T;
       t += (int64_t)gridDim.x * blockDim.x) {
    if (t == st.T) {
      st.tile_act[t] = aoff[st.L];
      continue;
    }
    const int l = st.tile_layer[t];
    const uint32_t key = (uint32_t)st.tile_start[t];
    int64_t lo = aoff[l], hi = aoff[l + 1];
    while (lo < hi) {
      const int64_t mid = lo + ((hi - lo) >> 1);
      if (act[mid] < key) lo = mid + 1; else hi = mid;
    }
    st.tile_act[t] = lo;
  }
}

// ---------------------------------------------------------------------------
// Dense requantisation of every layer with its current threshold; with
// PATCH the codes of the actives come from their perturbed values wp (the
// latents themselves are never written).  One block of 128 threads per tile;
// a thread streams 64 consecutive latents (non-temporal 16-byte loads: they
// are read once) and writes their 4 code words (one 16-byte non-temporal
// store where aligned).  A tile's actives are tile_act[t] .. tile_act[t+1]-1:
// with none, LDS is not touched; with some, the words meet in LDS and the
// actives are patched with LDS atomics; with every element active, the codes
// come from wp directly.
// ---------------------------------------------------------------------------
// Global-address-space views (the pointers are computed from device tables,
// so the compiler would otherwise emit FLAT accesses).
typedef const __attribute__((address_space(1))) v4u gv4u_c;
typedef __attribute__((address_space(1))) v4u gv4u;
typedef __attribute__((address_space(1))) uint32_t gu32;

__device__ __forceinline__ void vec_values(const v4u* b, int nvec, float* out, const float*) {
  for (int v = 0; v < nvec; ++v)
    for (int i = 0; i < 4; ++i) out[4 * v + i] = __uint_as_float(b[v][i]);
}
__device__ __forceinline__ void vec_values(const v4u* b, int nvec, float* out, const uint16_t*) {
  for (int v = 0; v < nvec; ++v)
    for (int i = 0; i < 4; ++i) {
      out[8 * v + 2 * i] = __uint_as_float(b[v][i] << 16);
      out[8 * v + 2 * i + 1] = __uint_as_float(b[v][i] & 0xFFFF0000u);
    }
}

__device__ __forceinline__ uint32_t code_word(const float* v, float tau) {
  uint32_t word = 0;
#pragma unroll
  for (int q = 0; q < 16; ++q) word |= ternary_code(v[q], tau) << code_shift(q);
  return word;
}

constexpr int kRqThreads = 128;
// Threads of the dense requantisation stream (one 8192-element tile per block: four
// 16-byte chunks per thread for bf16 latents); with non-temporal code stores this
// measured 6.1 TB/s against 5.2 TB/s for 128 threads and ordinary stores.
constexpr int kRqStream = 256;

// Code bits of the 16 / CPW consecutive elements v[] that start at element
// (part * 16 / CPW) of a code word.
template <int N>
__device__ __forceinline__ uint32_t partial_word(const float* v, int part, float tau) {
  uint32_t word = 0;
#pragma unroll
  for (int q = 0; q < N; ++q) word |= ternary_code(v[q], tau) << code_shift(part * N + q);
  return word;
}

// OR of a code word's parts held by CPW adjacent lanes (all of them get it).
template <int CPW>
__device__ __forceinline__ uint32_t join_word(uint32_t w) {
#pragma unroll
  for (int m = 1; m < CPW; m <<= 1) w |= (uint32_t)__shfl_xor((int)w, m, 64);
  return w;
}

// Loads are coalesced: 16-byte chunk c of the tile goes to lane c % 128, so
// one load instruction covers 1 KB of consecutive bytes; a code word's chunks
// (2 for bf16, 4 for fp32) sit in adjacent lanes and are joined by shuffles.
template <typename T, bool PATCH, int NT = kRqStream>
__device__ __forceinline__ void requant_tile(const DevState& st, const uint32_t* act,
                                             const float* wp, int64_t t) {
  constexpr int EPC = 16 / (int)sizeof(T);       // elements per 16-byte chunk
  constexpr int CPW = 16 / EPC;                  // chunks per code word
  constexpr int CPT = kTile / EPC / NT;  // chunks per thread
  __shared__ uint32_t words[kTile / 16];
  const int tid = threadIdx.x;
  const int l = st.tile_layer[t];
  const int64_t start = st.tile_start[t];
  const int cnt = (int)min((int64_t)kTile, st.n[l] - start);
  const float tau = st.tau_cur[l];
  const T* w = reinterpret_cast<const T*>(st.w[l]) + start;
  gu32* out = (gu32*)(st.codes + st.code_off[l] + start / 16);
  const bool owner = (tid % CPW) == 0;            // stores the word of its lane group
  int64_t a0 = 0, a1 = 0;
  uint32_t aw = 0;
  float pw = 0.0f;
  if (PATCH) {
    a0 = st.tile_act[t];
    a1 = st.tile_act[t + 1];
    const int64_t jj = a0 + tid;
    const int64_t jc = jj < a1 ? jj : (a0 < a1 ? a0 : 0);   // the list holds at least one slot
    aw = act[jc];
    pw = wp[jc];
  }
  const int64_t na = a1 - a0;
  if (PATCH && na == cnt) {
    // every element active: the codes come from wp (fp32, 4 per chunk)
    constexpr int FC = kTile / 4 / NT;   // 16 chunks per thread
    const float* src = wp + a0;
    const bool vec = (a0 & 3) == 0;
#pragma unroll
    for (int v = 0; v < FC; ++v) {
      const int c = v * NT + tid;
      const int e = c * 4;
      float x[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      if (e < cnt) {
        if (vec) {
          const v4u b = __builtin_nontemporal_load((gv4u_c*)(src + e));
#pragma unroll
          for (int r = 0; r < 4; ++r) x[r] = __uint_as_float(b[r]);
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) x[r] = src[e + r];
        }
      }
      const uint32_t wd = join_word<4>(partial_word<4>(x, c & 3, tau));
      if ((tid & 3) == 0 && e < cnt) out[c / 4] = wd;
    }
    return;
  }
  v4u buf[CPT];
#pragma unroll
  for (int v = 0; v < CPT; ++v) {
    const int e = (v * NT + tid) * EPC;
    buf[v] = __builtin_nontemporal_load((gv4u_c*)(w + (e < cnt ? e : 0)));   // clamped
  }
  uint32_t wd[CPT];
#pragma unroll
  for (int v = 0; v < CPT; ++v) {
    const int c = v * NT + tid;
    float x[EPC];
    vec_values(&buf[v], 1, x, (const T*)nullptr);
    wd[v] = join_word<CPW>(partial_word<EPC>(x, c % CPW, tau));
  }
  if (PATCH && na > 0) {
#pragma unroll
    for (int v = 0; v < CPT; ++v)
      if (owner) words[(v * NT + tid) / CPW] = wd[v];
    __syncthreads();
    auto patch_one = [&](uint32_t i, float x) __attribute__((always_inline)) {
      const uint32_t li = i - (uint32_t)start;
      const uint32_t code = ternary_code(x, tau);
      const int sh = code_shift((int)(li & 15u));
      atomicAnd(&words[li >> 4], ~(3u << sh));
      if (code) atomicOr(&words[li >> 4], code << sh);
    };
    if (tid < na) patch_one(aw, pw);
    for (int64_t jj = a0 + NT + tid; jj - tid < a1; jj += NT)
      if (jj < a1) patch_one(act[jj], wp[jj]);
    __syncthreads();
#pragma unroll
    for (int v = 0; v < CPT; ++v)
      if (owner) wd[v] = words[(v * NT + tid) / CPW];
  }
#pragma unroll
  for (int v = 0; v < CPT; ++v) {
    const int c = v * NT + tid;
    if (owner && c * EPC < cnt) __builtin_nontemporal_store(wd[v], &out[c / CPW]);
  }
}

// One tile per block: every tile of every layer (mask build, dense requantisation).
template <typename T, bool PATCH>
__global__ void __launch_bounds__(kRqStream) k_requant_tile(DevState st, const uint32_t* act,
                                                            const float* wp) {
  requant_tile<T, PATCH>(st, act, wp, blockIdx.x);
}

// The tiles of the layers the guard marked for the dense requantisation: dense_off[l]
// is the position of layer l's first tile in that list (dense_off[L] tiles in all);
// blocks stride over the list (none when every layer kept its frozen codes).
template <typename T>
__global__ void __launch_bounds__(kRqStream) k_requant_list(DevState st, const uint32_t* act,
                                                            const float* wp,
                                                            const int64_t* dense_off) {
  const int64_t total = dense_off[st.L];
  for (int64_t i = blockIdx.x; i < total; i += gridDim.x) {
    int lo = 0, hi = st.L - 1;                   // last layer with dense_off <= i
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (dense_off[mid] <= i) lo = mid; else hi = mid - 1;
    }
    __syncthreads();                             // the previous tile's LDS words are consumed
    requant_tile<T, true>(st, act, wp, st.tile0[lo] + (i - dense_off[lo]));
  }
}

// The four draws of Philox counter quad q on a stream: one Philox call and one
// Box-Muller pair per two ids -- the operations of gauss_at, so the values are the same.
__device__ __forceinline__ void gauss_quad(uint64_t seed, uint64_t q, uint32_t stream, float z[4]) {
  const U4 x = philox10((uint32_t)q, (uint32_t)(q >> 32), stream, 0u, (uint32_t)seed,
                        (uint32_t)(seed >> 32));
  box_muller(x.a, x.b, z[0], z[1]);     // ids 4q, 4q+1: cos, sin of the pair (x0, x1)
  box_muller(x.c, x.d, z[2], z[3]);     // ids 4q+2, 4q+3: cos, sin of the pair (x2, x3)
}

// ---------------------------------------------------------------------------
// Perturbation at the actives: w' = fma(se, z, w), stored compactly; the
// exact change of the fixed-point |w| sum goes to S_cur (initialised to
// S_clean by the caller).  Each thread walks kRun consecutive entries.
// ---------------------------------------------------------------------------
constexpr int kRun = 4;

// The kRun = 4 active-list entries j0 .. j0+3 of a run (j0 % 4 == 0): one
// 16-byte load when the run is whole; n = entries of the run below je.
__device__ __forceinline__ int run_entries(const uint32_t* act, int64_t j0, int64_t je,
                                           uint32_t i[4]) {
  if (j0 + 3 < je) {
    const v4u v = *reinterpret_cast<const v4u*>(act + j0);
    i[0] = v[0]; i[1] = v[1]; i[2] = v[2]; i[3] = v[3];
    return 4;
  }
  int n = 0;
  for (int r = 0; r < 4; ++r) {
    i[r] = j0 + r < je ? act[j0 + r] : 0u;
    n += j0 + r < je;
  }
  return n;
}

// Latents at four local indices: one load when they are the consecutive,
// 4-aligned i0 .. i0+3 (dense runs), four gathers otherwise.
__device__ __forceinline__ void gather4(const float* w, const uint32_t i[4], int n, float v[4]) {
  if (n == 4 && i[3] == i[0] + 3 && (i[0] & 3u) == 0) {
    const float4 a = *reinterpret_cast<const float4*>(w + i[0]);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  } else {
    for (int r = 0; r < 4; ++r) v[r] = r < n ? w[i[r]] : 0.0f;
  }
}
__device__ __forceinline__ void gather4(const uint16_t* w, const uint32_t i[4], int n, float v[4]) {
  if (n == 4 && i[3] == i[0] + 3 && (i[0] & 3u) == 0) {
    const uint2 a = *reinterpret_cast<const uint2*>(w + i[0]);
    v[0] = __uint_as_float(a.x << 16);
    v[1] = __uint_as_float(a.x & 0xFFFF0000u);
    v[2] = __uint_as_float(a.y << 16);
    v[3] = __uint_as_float(a.y & 0xFFFF0000u);
  } else {
    for (int r = 0; r < 4; ++r) v[r] = r < n ? bf16_to_f32(w[i[r]]) : 0.0f;
  }
}
__device__ __forceinline__ void scatter4(float* w, const uint32_t i[4], int n, const float v[4]) {
  if (n == 4 && i[3] == i[0] + 3 && (i[0] & 3u) == 0) {
    *reinterpret_cast<float4*>(w + i[0]) = make_float4(v[0], v[1], v[2], v[3]);
  } else {
    for (int r = 0; r < 4; ++r)
      if (r < n) w[i[r]] = v[r];
  }
}
__device__ __forceinline__ void scatter4(uint16_t* w, const uint32_t i[4], int n, const float v[4]) {
  if (n == 4 && i[3] == i[0] + 3 && (i[0] & 3u) == 0) {
    const uint32_t lo = (uint32_t)f32_to_bf16_rne(v[0]) | ((uint32_t)f32_to_bf16_rne(v[1]) << 16);
    const uint32_t hi = (uint32_t)f32_to_bf16_rne(v[2]) | ((uint32_t)f32_to_bf16_rne(v[3]) << 16);
    *reinterpret_cast<uint2*>(w + i[0]) = make_uint2(lo, hi);
  } else {
    for (int r = 0; r < 4; ++r)
      if (r < n) w[i[r]] = f32_to_bf16_rne(v[r]);
  }
}
// Four values to wp[j0 ..]: one 16-byte store for a whole run (8 bytes for bf16
// values, which the bf16 variant stores exactly).
__device__ __forceinline__ void put4(float* wp, int64_t j0, int n, const float v[4]) {
  if (n == 4) {
    *reinterpret_cast<float4*>(wp + j0) = make_float4(v[0], v[1], v[2], v[3]);
  } else {
    for (int r = 0; r < n; ++r) wp[j0 + r] = v[r];
  }
}
__device__ __forceinline__ void put4(uint16_t* wp, int64_t j0, int n, const float v[4]) {
  if (n == 4) {
    const uint32_t lo = (uint32_t)f32_to_bf16_rne(v[0]) | ((uint32_t)f32_to_bf16_rne(v[1]) << 16);
    const uint32_t hi = (uint32_t)f32_to_bf16_rne(v[2]) | ((uint32_t)f32_to_bf16_rne(v[3]) << 16);
    *reinterpret_cast<uint2*>(wp + j0) = make_uint2(lo, hi);
  } else {
    for (int r = 0; r < n; ++r) wp[j0 + r] = f32_to_bf16_rne(v[r]);
  }
}

// wc (compact mode): the active latents in list order, read instead of the layers.
// (j0 % 4 == 0: a whole run is one 8- or 16-byte load)
__device__ __forceinline__ void list4(const float* wc, int64_t j0, int n, float v[4]) {
  if (n == 4) {
    const float4 a = *reinterpret_cast<const float4*>(wc + j0);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  } else {
    for (int r = 0; r < 4; ++r) v[r] = r < n ? wc[j0 + r] : 0.0f;
  }
}
__device__ __forceinline__ void list4(const uint16_t* wc, int64_t j0, int n, float v[4]) {
  if (n == 4) {
    const uint2 a = *reinterpret_cast<const uint2*>(wc + j0);
    v[0] = __uint_as_float(a.x << 16);
    v[1] = __uint_as_float(a.x & 0xFFFF0000u);
    v[2] = __uint_as_float(a.y << 16);
    v[3] = __uint_as_float(a.y & 0xFFFF0000u);
  } else {
    for (int r = 0; r < 4; ++r) v[r] = r < n ? bf16_to_f32(wc[j0 + r]) : 0.0f;
  }
}

// PAIR: both signs of the perturbation from one pass -- w' at +se to wp with its
// delta in S_cur, w' at -se to wpm with its delta in S_alt (list order), so the other
// sign of the pair needs no generator pass; with zs the draws z themselves go to zs
// (list order), from which a single-direction update of the same seed reads them
// instead of drawing again.
template <typename T, bool PAIR>
__global__ void __launch_bounds__(256) k_perturb_delta(DevState st,
                                                       const uint32_t* __restrict__ act,
                                                       const int64_t* act_off, uint64_t seed,
                                                       float se, float* __restrict__ wp,
                                                       const T* __restrict__ wc,
                                                       float* __restrict__ wpm,
                                                       int64_t* S_alt, float* __restrict__ zs) {
  __shared__ int64_t aoff[kMaxLayers + 1];
  load_offsets(aoff, act_off, st.L);
  const int64_t k = aoff[st.L];
  // Block b owns the contiguous entries [jb, je): a thread's layer changes
  // rarely, so its partial sum goes out with one atomic per layer change and
  // one wave-level atomic at the end.
  const int64_t per = (k + gridDim.x - 1) / gridDim.x;
  const int64_t chunk = (per + 256 * kRun - 1) / (256 * kRun) * (256 * kRun);
  const int64_t jb = (int64_t)blockIdx.x * chunk, je = min(k, jb + chunk);
  bool bad = false, any = false;
  int l = -1;
  long long acc = 0, acc2 = 0;
  GaussCache zc;
  auto flush_layer = [&]() __attribute__((always_inline)) {
    if (any) {
      atomicAdd((unsigned long long*)&st.S_cur[l], (unsigned long long)acc);
      if (PAIR) atomicAdd((unsigned long long*)&S_alt[l], (unsigned long long)acc2);
    }
    acc = 0;
    acc2 = 0;
  };
  // the next run's indices are loaded one iteration ahead
  uint32_t inx[4] = {0u, 0u, 0u, 0u};
  int nnx = jb + (int64_t)threadIdx.x * kRun < je
                ? run_entries(act, jb + (int64_t)threadIdx.x * kRun, je, inx) : 0;
  for (int64_t j0 = jb + (int64_t)threadIdx.x * kRun; j0 < je; j0 += 256 * kRun) {
    uint32_t i[4] = {inx[0], inx[1], inx[2], inx[3]};
    const int n = nnx;
    nnx = j0 + 256 * kRun < je ? run_entries(act, j0 + 256 * kRun, je, inx) : 0;
    // the run lies in one layer, or it is handled entry by entry
    const int lr = layer_of(aoff, st.L, j0);
    const bool one = aoff[lr + 1] >= j0 + n;
    float wv[4], v[4], vm[4], z[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    if (wc)
      list4(wc, j0, n, wv);
    else if (one)
      gather4(reinterpret_cast<const T*>(st.w[lr]), i, n, wv);
    const uint64_t g0 = one ? (uint64_t)(st.gid0[lr] + i[0]) : 0ull;
    if (one && n == 4 && i[3] == i[0] + 3 && (g0 & 3u) == 0) {
      // a whole Philox quad (dense runs): one draw, no per-entry layer walk
      if (l != lr) {
        flush_layer();
        l = lr;
      }
      if (se != 0.0f) gauss_quad(seed, g0 >> 2, 0u, z);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        v[r] = se != 0.0f ? fmaf(se, z[r], wv[r]) : wv[r];
        bad |= !in_fix_range(v[r]);
        const long long f0 = (long long)fix_abs(wv[r]);
        acc += (long long)fix_abs(v[r]) - f0;
        if (PAIR) {
          vm[r] = fmaf(-se, z[r], wv[r]);
          bad |= !in_fix_range(vm[r]);
          acc2 += (long long)fix_abs(vm[r]) - f0;
        }
      }
      any = true;
      put4(wp, j0, 4, v);
      if (PAIR) put4(wpm, j0, 4, vm);
      if (PAIR && zs) put4(zs, j0, 4, z);
      continue;
    }
    for (int r = 0; r < n; ++r) {
      const int64_t j = j0 + r;
      if (l < 0) {
        l = layer_of(aoff, st.L, j);
      } else if (aoff[l + 1] <= j) {        // into a later layer
        flush_layer();
        any = false;
        while (aoff[l + 1] <= j) ++l;
      }
      if (!wc && !one) wv[r] = load1(reinterpret_cast<const T*>(st.w[l]), i[r]);
      if (se != 0.0f) z[r] = zc.get(seed, (uint64_t)(st.gid0[l] + i[r]));
      v[r] = se != 0.0f ? fmaf(se, z[r], wv[r]) : wv[r];
      bad |= !in_fix_range(v[r]);
      const long long f0 = (long long)fix_abs(wv[r]);
      acc += (long long)fix_abs(v[r]) - f0;
      if (PAIR) {
        vm[r] = fmaf(-se, z[r], wv[r]);
        bad |= !in_fix_range(vm[r]);
        acc2 += (long long)fix_abs(vm[r]) - f0;
      }
      any = true;
    }
    put4(wp, j0, n, v);
    if (PAIR) put4(wpm, j0, n, vm);
    if (PAIR && zs) put4(zs, j0, n, z);
  }
  flush_delta((long long*)st.S_cur, l, acc, any);
  if (PAIR) flush_delta((long long*)S_alt, l, acc2, any);
  if (bad) atomicOr(st.err, 1);
}

// ---------------------------------------------------------------------------
// Full-precision parameters theta (Algorithm 1 perturbs and updates them
// densely, together with the masked latents): z at theta id t is the draw of
// the step's seed on Philox stream 1.  One Philox call per id quad and one
// Box-Muller pair per two ids -- the operations of gauss_at, so the values are
// the same.  Both perturbed copies theta +- eps z (rounded to the storage
// type) come from one pass; the update is in place.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float th_load(const float* p) { return *p; }
__device__ __forceinline__ float th_load(const uint16_t* p) { return bf16_to_f32(*p); }
__device__ __forceinline__ void th_store(float* p, float v) { *p = v; }
__device__ __forceinline__ void th_store(uint16_t* p, float v) { *p = f32_to_bf16_rne(v); }

// Quads q of the theta id space covering [tid0, tid0 + n); the four elements of a
// quad are local indices 4q - tid0 .. + 3.  With tid0 % 4 == 0 (and 16-byte
// aligned tensors) inner quads are one 16-byte (fp32) or 8-byte (bf16) access.
template <typename F>
__device__ __forceinline__ void theta_quads(int64_t n, int64_t tid0, F&& f) {
  const int64_t q0 = tid0 >> 2, q1 = (tid0 + n + 3) >> 2;
  for (int64_t q = q0 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < q1;
       q += (int64_t)gridDim.x * blockDim.x)
    f(q, 4 * q - tid0);
}

__device__ __forceinline__ void gather_quad(const float* p, float v[4]) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
}
__device__ __forceinline__ void gather_quad(const uint16_t* p, float v[4]) {
  const uint2 a = *reinterpret_cast<const uint2*>(p);
  v[0] = __uint_as_float(a.x << 16);
  v[1] = __uint_as_float(a.x & 0xFFFF0000u);
  v[2] = __uint_as_float(a.y << 16);
  v[3] = __uint_as_float(a.y & 0xFFFF0000u);
}
__device__ __forceinline__ void scatter_quad(float* p, const float v[4]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void scatter_quad(uint16_t* p, const float v[4]) {
  const uint32_t lo = (uint32_t)f32_to_bf16_rne(v[0]) | ((uint32_t)f32_to_bf16_rne(v[1]) << 16);
  const uint32_t hi = (uint32_t)f32_to_bf16_rne(v[2]) | ((uint32_t)f32_to_bf16_rne(v[3]) << 16);
  *reinterpret_cast<uint2*>(p) = make_uint2(lo, hi);
}
template <typename T>
__device__ __forceinline__ void load_quad(const T* p, int64_t e0, int64_t n, bool vec, float v[4]) {
  if (vec && e0 >= 0 && e0 + 3 < n) {
    gather_quad(p + e0, v);
  } else {
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] = (e0 + r >= 0 && e0 + r < n) ? th_load(p + e0 + r) : 0.0f;
  }
}
template <typename T>
__device__ __forceinline__ void store_quad(T* p, int64_t e0, int64_t n, bool vec, const float v[4]) {
  if (vec && e0 >= 0 && e0 + 3 < n) {
    scatter_quad(p + e0, v);
  } else {
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (e0 + r >= 0 && e0 + r < n) th_store(p + e0 + r, v[r]);
  }
}

template <typename T>
__global__ void __launch_bounds__(256) k_theta_pair(const T* __restrict__ th, int64_t n,
                                                    int64_t tid0, uint64_t seed, float eps,
                                                    T* __restrict__ plus, T* __restrict__ minus) {
  const bool vec = (tid0 & 3) == 0;
  const float me = -eps;
  theta_quads(n, tid0, [&](int64_t q, int64_t e0) {
    float z[4], w[4], vp[4], vm[4];
    gauss_quad(seed, (uint64_t)q, 1u, z);
    load_quad(th, e0, n, vec, w);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      vp[r] = fmaf(eps, z[r], w[r]);
      vm[r] = fmaf(me, z[r], w[r]);
    }
    store_quad(plus, e0, n, vec, vp);
    store_quad(minus, e0, n, vec, vm);
  });
}

// True when every coefficient of the update is finite (a non-finite one, reported
// by the coefficient kernel, leaves latents and theta untouched).
__device__ __forceinline__ bool coeffs_ok(const float* scal, int K) {
  bool ok = true;
  for (int q = 0; q < K; ++q) ok = ok && isfinite(scal[q]);
  return ok;
}

// theta <- rnd(v), v = fma(a_K, z_K, ... fma(a_1, z_1, theta)) in fp32, a_k = scal[k].
template <typename T>
__global__ void __launch_bounds__(256) k_theta_update(T* __restrict__ th, int64_t n, int64_t tid0,
                                                      SeedList seeds, const float* scal) {
  if (!coeffs_ok(scal, seeds.K)) return;
  const bool vec = (tid0 & 3) == 0;
  theta_quads(n, tid0, [&](int64_t q, int64_t e0) {
    float z[4], w[4];
    load_quad(th, e0, n, vec, w);
    for (int k = 0; k < seeds.K; ++k) {
      const float a = scal[k];
      gauss_quad(seeds.s[k], (uint64_t)q, 1u, z);
#pragma unroll
      for (int r = 0; r < 4; ++r) w[r] = fmaf(a, z[r], w[r]);
    }
    store_quad(th, e0, n, vec, w);
  });
}

// ---------------------------------------------------------------------------
// Masked update: w_i <- round(fma(a, z_i, w_i)), a = -(lr g); exact delta of
// the clean fixed-point sum.
// ---------------------------------------------------------------------------
__global__ void k_set_coeff(float* scal, float a) {
  scal[0] = a;
  scal[kScalG] = 0.0f;
}

struct CoefList {
  float a[kMaxK];
};
__global__ void k_set_coeffs(float* scal, CoefList c, int K) {
  if ((int)threadIdx.x < K) scal[threadIdx.x] = c.a[threadIdx.x];
}

// K directions: g_k = (F+_k - F-_k) / (2 eps), a_k = -((lr / K) g_k), all fp32.
__global__ void k_coeffs_multi_from_losses(const float* losses, int K, float eps, float lr,
                                           float* scal, int32_t* err) {
  const int k = threadIdx.x;
  if (k >= K) return;
  const float g = __fdiv_rn(losses[2 * k] - losses[2 * k + 1], 2.0f * eps);
  const float c = __fdiv_rn(lr, (float)K);
  const float a = -(c * g);
  scal[k] = a;
  if (!isfinite(a)) atomicOr(err, 2);
}

// Evolution strategies on the mask (appendix on RL-based fine-tuning): a_n =
// (lr / N) Rt_n in fp32, Rt the population z-score of the rewards in fp64 (index
// order; zero when the deviation is zero) or the raw rewards.  One thread: the
// sums run in a fixed order.  A non-finite coefficient skips the update (the
// update kernels test every coefficient) and raises the deferred error bit 2.
__global__ void k_es_coeffs(const float* rewards, int N, float lr, int standardize, float* scal,
                            int32_t* err) {
  if (threadIdx.x != 0) return;
  float rt[kMaxK];
  for (int n = 0; n < N; ++n) rt[n] = rewards[n];
  if (standardize) {
    double mu = 0.0, var = 0.0;
    for (int n = 0; n < N; ++n) mu += (double)rewards[n];
    mu /= (double)N;
    for (int n = 0; n < N; ++n) {
      const double d = (double)rewards[n] - mu;
      var += d * d;
    }
    var /= (double)N;
    const double sd = sqrt(var);
    for (int n = 0; n < N; ++n)
      rt[n] = sd > 0.0 ? (float)(((double)rewards[n] - mu) / sd) : (isfinite(sd) ? 0.0f : NAN);
  }
  const float c = __fdiv_rn(lr, (float)N);
  bool ok = true;
  for (int n = 0; n < N; ++n) {
    const float a = c * rt[n];
    scal[n] = a;
    ok &= isfinite(a) != 0;
  }
  if (!ok) atomicOr(err, 2);
}

// g = (F+ - F-) / (2 eps) and a = -(lr g), in fp32 (eq. spsa).
__global__ void k_coeff_from_losses(const float* fp, const float* fm, float eps, float lr,
                                    float* scal, int32_t* err) {
  const float g = __fdiv_rn(*fp - *fm, 2.0f * eps);
  const float a = -(lr * g);
  scal[0] = a;
  scal[kScalG] = g;
  if (!isfinite(a)) atomicOr(err, 2);
}

// The new values also go, in list order and the latent dtype, to wn (read by the
// shrink).  With a non-finite coefficient (reported by the coefficient kernel) the
// latents are left untouched and wn holds their current values.
template <typename T>
__global__ void __launch_bounds__(256) k_update(DevState st, const uint32_t* __restrict__ act,
                                                const int64_t* act_off, SeedList seeds,
                                                const float* scal, T* __restrict__ wn,
                                                T* __restrict__ wc,
                                                int write_latents,
                                                const float* __restrict__ zs) {
  __shared__ int64_t aoff[kMaxLayers + 1];
  load_offsets(aoff, act_off, st.L);
  const float a = scal[0];
  const uint64_t seed = seeds.s[0];
  const int K = seeds.K;
  const bool a_ok = coeffs_ok(scal, K);
  const int64_t k = aoff[st.L];
  const int64_t per = (k + gridDim.x - 1) / gridDim.x;
  const int64_t chunk = (per + 256 * kRun - 1) / (256 * kRun) * (256 * kRun);
  const int64_t jb = (int64_t)blockIdx.x * chunk, je = min(k, jb + chunk);
  bool bad = false, any = false;
  int l = -1;
  long long acc = 0;
  GaussCache zc;
  // the next run's indices are loaded one iteration ahead
  uint32_t inx[4] = {0u, 0u, 0u, 0u};
  int nnx = jb + (int64_t)threadIdx.x * kRun < je
                ? run_entries(act, jb + (int64_t)threadIdx.x * kRun, je, inx) : 0;
  for (int64_t j0 = jb + (int64_t)threadIdx.x * kRun; j0 < je; j0 += 256 * kRun) {
    uint32_t i[4] = {inx[0], inx[1], inx[2], inx[3]};
    const int n = nnx;
    nnx = j0 + 256 * kRun < je ? run_entries(act, j0 + 256 * kRun, je, inx) : 0;
    const int lr = layer_of(aoff, st.L, j0);
    const bool one = aoff[lr + 1] >= j0 + n;
    float wv[4], nv[4];
    if (wc)
      list4((const T*)wc, j0, n, wv);
    else if (one)
      gather4(reinterpret_cast<const T*>(st.w[lr]), i, n, wv);
    const uint64_t g0 = one ? (uint64_t)(st.gid0[lr] + i[0]) : 0ull;
    if (one && n == 4 && i[3] == i[0] + 3 && (g0 & 3u) == 0) {
      // a whole Philox quad (dense runs): one draw per direction, same fma chain
      if (l != lr) {
        if (any) atomicAdd((unsigned long long*)&st.S_clean[l], (unsigned long long)acc);
        acc = 0;
        l = lr;
      }
      T* w = reinterpret_cast<T*>(const_cast<void*>(st.w[lr]));
#pragma unroll
      for (int r = 0; r < 4; ++r) nv[r] = wv[r];
      if (a_ok) {
        float z[4], v[4];
        if (zs) {                               // the pair pass's draws (K = 1)
          const float4 zz = *reinterpret_cast<const float4*>(zs + j0);
          z[0] = zz.x; z[1] = zz.y; z[2] = zz.z; z[3] = zz.w;
        } else {
          gauss_quad(seed, g0 >> 2, 0u, z);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = fmaf(a, z[r], wv[r]);
        for (int q = 1; q < K; ++q) {
          gauss_quad(seeds.s[q], g0 >> 2, 0u, z);
#pragma unroll
          for (int r = 0; r < 4; ++r) v[r] = fmaf(scal[q], z[r], v[r]);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) nv[r] = storage_round(w, v[r]);
        if (wc) put4(wc, j0, 4, nv);
        if (write_latents) scatter4(w, i, 4, nv);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        bad |= !in_fix_range(nv[r]);
        acc += (long long)fix_abs(nv[r]) - (long long)fix_abs(wv[r]);
      }
      any = true;
      put4(wn, j0, 4, nv);
      continue;
    }
    for (int r = 0; r < n; ++r) {
      const int64_t j = j0 + r;
      if (l < 0) {
        l = layer_of(aoff, st.L, j);
      } else if (aoff[l + 1] <= j) {
        if (any) atomicAdd((unsigned long long*)&st.S_clean[l], (unsigned long long)acc);
        acc = 0;
        any = false;
        while (aoff[l + 1] <= j) ++l;
      }
      T* w = reinterpret_cast<T*>(const_cast<void*>(st.w[l]));
      if (!wc && !one) wv[r] = load1(w, i[r]);
      nv[r] = wv[r];
      if (a_ok) {
        const uint64_t gid = (uint64_t)(st.gid0[l] + i[r]);
        float v = fmaf(a, zs ? zs[j] : zc.get(seed, gid), wv[r]);
        for (int q = 1; q < K; ++q) v = fmaf(scal[q], gauss_at(seeds.s[q], gid), v);
        nv[r] = storage_round(w, v);
        if (wc) store1(wc, j, nv[r]);
        if (write_latents && !one) store1(w, i[r], nv[r]);
      }
      bad |= !in_fix_range(nv[r]);
      acc += (long long)fix_abs(nv[r]) - (long long)fix_abs(wv[r]);
      any = true;
    }
    if (write_latents && one && a_ok) scatter4(reinterpret_cast<T*>(const_cast<void*>(st.w[lr])), i, n, nv);
    put4(wn, j0, n, nv);
  }
  flush_delta((long long*)st.S_clean, l, acc, any);
  if (bad) atomicOr(st.err, 1);
}

// ---------------------------------------------------------------------------
// Guarded requantisation.  The codes of frozen (inactive) weights of layer l are
// Q(w; tau_ref[l]); every frozen weight lies at least mref[l] (exactly, in fp64)
// from tau_ref[l].  A perturbed threshold tau' with |tau' - tau_ref| < mref
// cannot change a frozen code (the sign of |w| - tau is the same at tau_ref and
// tau'), so the codes equal the dense requantisation at tau' once the actives'
// codes are rewritten.  Otherwise the layer is requantised densely, its frozen
// codes then refer to tau' and no bound is kept for it (mref < 0: dense until the
// next mask build).
// ---------------------------------------------------------------------------
// One block: need[l] for every layer, then dense_off (the layers needing the dense
// pass, their tiles listed in layer order).  A layer whose weights are all active has
// no frozen code and always passes.  force: every layer takes the dense pass.
// Compact mode (no frozen latents kept): a layer that fails the guard cannot be
// re-quantised; its frozen codes stay and the deferred error bit 4 is raised.
__global__ void __launch_bounds__(256) k_guard(DevState st, int force, int64_t* dense_off,
                                               int compact, const int64_t* act_off) {
  __shared__ int64_t cnt[kMaxLayers + 1];
  for (int l = threadIdx.x; l < st.L; l += blockDim.x) {
    const float tc = st.tau_cur[l], tr = st.tau_ref[l];
    const bool none_frozen = act_off[l + 1] - act_off[l] == st.n[l];
    const bool pass = tc == tr || none_frozen || fabs((double)tc - (double)tr) < st.mref[l];
    if (compact && !pass) atomicOr(st.err, 4);
    // forced dense pass: a layer that passes rewrites its frozen codes unchanged, so
    // its reference and bound stay valid
    const bool keep = compact || (!force && pass);
    st.need[l] = keep ? 0 : 1;
    if (!pass && !compact) {
      st.tau_ref[l] = tc;
      st.mref[l] = -1.0;
    }
    cnt[l] = keep ? 0 : (l + 1 < st.L ? st.tile0[l + 1] : st.T) - st.tile0[l];
  }
  __syncthreads();
  if (threadIdx.x == 0) {                        // exclusive scan in LDS
    int64_t run = 0;
    for (int l = 0; l < st.L; ++l) {
      const int64_t c = cnt[l];
      cnt[l] = run;
      run += c;
    }
    cnt[st.L] = run;
  }
  __syncthreads();
  for (int l = threadIdx.x; l <= st.L; l += blockDim.x) dense_off[l] = cnt[l];
}

// After a dense requantisation of every layer at tau_cur (the mask build): every
// inactive weight's fp32 distance is at least xi0, so its exact distance is at
// least xi_lo = xi0 - ulp(xi0)/2.
__global__ void k_ref_init(DevState st, double xi_lo) {
  const int l = blockIdx.x * blockDim.x + threadIdx.x;
  if (l >= st.L) return;
  st.tau_ref[l] = st.tau_cur[l];
  st.mref[l] = xi_lo;
}

// After an update: a weight leaving the set has fp32 distance above xi0 to the new
// clean threshold tau, so it lies at least xi_lo - |tau - tau_ref| from tau_ref
// (its code is written at tau_ref by the shrink).
__global__ void k_ref_after_update(DevState st, double xi_lo) {
  const int l = blockIdx.x * blockDim.x + threadIdx.x;
  if (l >= st.L || st.mref[l] < 0.0) return;
  const double m = xi_lo - fabs((double)st.tau[l] - (double)st.tau_ref[l]);
  st.mref[l] = fmin(st.mref[l], m);
}

// Rewrite the 2-bit code of local index i of layer l (other fields of the word may
// be written concurrently by other threads: only the changed bits are flipped, with
// one atomic; the word is read past the L1 cache).
__device__ __forceinline__ void set_code(uint32_t* codes, int64_t code_off, uint32_t i,
                                         uint32_t code) {
  uint32_t* wp = codes + code_off + (i >> 4);
  const int sh = code_shift((int)(i & 15u));
  const uint32_t cur = __hip_atomic_load(wp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint32_t diff = (((cur >> sh) & 3u) ^ code) << sh;
  if (diff) atomicXor(wp, diff);
}

// The actives' codes at their perturbed values, for the layers that kept their frozen
// codes.  Each thread walks kRun consecutive list entries.  An entry whose code word
// holds no other active (its list neighbours lie in other words) is the word's only
// writer and updates it with a plain read-modify-write; shared words take the atomic.
__global__ void __launch_bounds__(256) k_patch_codes(DevState st, const uint32_t* __restrict__ act,
                                                     const int64_t* act_off,
                                                     const float* __restrict__ wp) {
  __shared__ int64_t aoff[kMaxLayers + 1];
  load_offsets(aoff, act_off, st.L);
  const int64_t k = aoff[st.L];
  for (int64_t j0 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * kRun; j0 < k;
       j0 += (int64_t)gridDim.x * 256 * kRun) {
    uint32_t i[kRun + 2];                        // i[0], i[kRun+1]: the run's list neighbours
    const int n = run_entries(act, j0, k, i + 1);
    i[0] = j0 > 0 ? act[j0 - 1] : 0xFFFFFFFFu;
    i[n + 1] = j0 + n < k ? act[j0 + n] : 0xFFFFFFFFu;
    int l = layer_of(aoff, st.L, j0);
    for (int r = 1; r <= n; ++r) {
      const int64_t j = j0 + r - 1;
      while (aoff[l + 1] <= j) ++l;
      if (st.need[l]) continue;
      const uint32_t idx = i[r], code = ternary_code(wp[j], st.tau_cur[l]);
      const bool sole = (i[r - 1] >> 4) != (idx >> 4) && (i[r + 1] >> 4) != (idx >> 4);
      if (sole) {
        uint32_t* wptr = st.codes + st.code_off[l] + (idx >> 4);
        const int sh = code_shift((int)(idx & 15u));
        const uint32_t cur = *wptr, nw = (cur & ~(3u << sh)) | (code << sh);
        if (nw != cur) *wptr = nw;
      } else {
        set_code(st.codes, st.code_off[l], idx, code);
      }
    }
  }
}

// The same codes tile by tile, for denser sets (one block per tile): a tile with
// actives reads its code words back into LDS (one 16-byte load per thread), rewrites
// the actives' codes there and stores the words (the frozen codes are reused, so the
// latents are not read); a fully active tile takes every code from w'; tiles without
// actives, and the tiles of layers that take the dense pass, are not touched.
__global__ void __launch_bounds__(kRqThreads) k_patch_tiles(DevState st,
                                                            const uint32_t* __restrict__ act,
                                                            const float* __restrict__ wp) {
  __shared__ uint32_t words[kTile / 16];
  const int tid = threadIdx.x;
  const int64_t t = blockIdx.x;
  const int l = st.tile_layer[t];
  const int64_t a0 = st.tile_act[t], a1 = st.tile_act[t + 1];
  if (st.need[l] || a1 == a0) return;            // block-uniform
  const int64_t start = st.tile_start[t];
  const int cnt = (int)min((int64_t)kTile, st.n[l] - start);   // a multiple of 16
  const int nw = cnt / 16;
  const float tau = st.tau_cur[l];
  const int64_t woff = st.code_off[l] + start / 16;
  gu32* out = (gu32*)(st.codes + woff);
  if (a1 - a0 == cnt) {                          // every element active: codes from w'
    constexpr int FC = kTile / 4 / kRqThreads;
    const float* src = wp + a0;
    const bool vec = (a0 & 3) == 0;
#pragma unroll
    for (int v = 0; v < FC; ++v) {
      const int c = v * kRqThreads + tid;
      const int e = c * 4;
      float x[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      if (e < cnt) {
        if (vec) {
          const v4u b = __builtin_nontemporal_load((gv4u_c*)(src + e));
#pragma unroll
          for (int r = 0; r < 4; ++r) x[r] = __uint_as_float(b[r]);
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) x[r] = src[e + r];
        }
      }
      const uint32_t wd = join_word<4>(partial_word<4>(x, c & 3, tau));
      if ((tid & 3) == 0 && e < cnt) out[c / 4] = wd;
    }
    return;
  }
  static_assert(kTile / 16 == 4 * kRqThreads, "one 16-byte chunk of words per thread");
  const bool vec = (woff & 3) == 0;
  const int i0 = 4 * tid;
  // the first active entry of this thread is loaded together with the words
  const int64_t jf = a0 + tid;
  const uint32_t af = jf < a1 ? act[jf] : 0u;
  const float wf = jf < a1 ? wp[jf] : 0.0f;
  if (vec && i0 + 3 < nw) {
    const v4u v = *(gv4u_c*)(out + i0);
    words[i0] = v[0]; words[i0 + 1] = v[1]; words[i0 + 2] = v[2]; words[i0 + 3] = v[3];
  } else {
    for (int r = 0; r < 4; ++r)
      if (i0 + r < nw) words[i0 + r] = out[i0 + r];
  }
  __syncthreads();
  auto patch = [&](uint32_t idx, float x) __attribute__((always_inline)) {
    const uint32_t li = idx - (uint32_t)start;
    const uint32_t code = ternary_code(x, tau);
    const int sh = code_shift((int)(li & 15u));
    atomicAnd(&words[li >> 4], ~(3u << sh));
    if (code) atomicOr(&words[li >> 4], code << sh);
  };
  if (jf < a1) patch(af, wf);
  for (int64_t jj = jf + kRqThreads; jj < a1; jj += kRqThreads) patch(act[jj], wp[jj]);
  __syncthreads();
  if (vec && i0 + 3 < nw) {
    *(gv4u*)(out + i0) = v4u{words[i0], words[i0 + 1], words[i0 + 2], words[i0 + 3]};
  } else {
    for (int r = 0; r < 4; ++r)
      if (i0 + r < nw) out[i0 + r] = words[i0 + r];
  }
}

// ---------------------------------------------------------------------------
// Shrink-only set update: keep the actives with ||w| - tau| <= xi0.
// Block b handles entries [b * 256 per, (b+1) * 256 per); thread t takes the
// four consecutive entries b * 256 per + 4 (256 r + t) + e (r < per / 4, e < 4,
// per <= kShrinkPer), so a lane's values and indices are one 8- or 16-byte load
// and a wave's are contiguous; per grows with the list so that small lists still
// spread over many blocks.  Kept entries keep the list order (r, wave, lane, e).
// The updated values come from wn (list order, in the latent dtype: the rounded
// new values are exact there).
// ---------------------------------------------------------------------------
constexpr int kShrinkPer = 64;                // entries per thread at most (block: 256 * per)

// Offsets and clean thresholds of every layer in LDS; all threads call.
__device__ __forceinline__ void load_layer_lds(int64_t* aoff, float* tau, const int64_t* act_off,
                                               const float* tau_g, int L) {
  for (int i = threadIdx.x; i <= L; i += blockDim.x) {
    aoff[i] = act_off[i];
    if (i < L) tau[i] = tau_g[i];
  }
  __syncthreads();
}

// Four consecutive list entries j .. j+3 (j % 4 == 0) below k: one vector load
// when all four exist.
__device__ __forceinline__ void load_quad4(const float* p, int64_t j, int64_t k, float v[4]) {
  if (j + 3 < k) {
    const float4 a = *reinterpret_cast<const float4*>(p + j);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  } else {
    for (int e = 0; e < 4; ++e) v[e] = j + e < k ? p[j + e] : 0.0f;
  }
}
__device__ __forceinline__ void load_quad4(const uint16_t* p, int64_t j, int64_t k, float v[4]) {
  if (j + 3 < k) {
    const uint2 a = *reinterpret_cast<const uint2*>(p + j);
    v[0] = __uint_as_float(a.x << 16);
    v[1] = __uint_as_float(a.x & 0xFFFF0000u);
    v[2] = __uint_as_float(a.y << 16);
    v[3] = __uint_as_float(a.y & 0xFFFF0000u);
  } else {
    for (int e = 0; e < 4; ++e) v[e] = j + e < k ? bf16_to_f32(p[j + e]) : 0.0f;
  }
}

// Keep flags of a thread's entries (bit 4 r + e); four quads in flight at a time.
template <typename T>
__device__ __forceinline__ uint64_t shrink_flags(const int64_t* aoff, const float* tau, int L,
                                                 const T* __restrict__ wn, int64_t k,
                                                 int64_t base, int per, float xi0) {
  uint64_t m = 0;
  const int64_t j0 = base + 4 * (int64_t)threadIdx.x;
  if (j0 >= k) return 0;
  int l = layer_of(aoff, L, j0);
  int64_t nxt = aoff[l + 1];
  const int R = per / 4;
  for (int r0 = 0; r0 < R; r0 += 4) {
    float v[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t j = j0 + 1024 * (int64_t)(r0 + u);
      if (r0 + u < R && j < k)
        load_quad4(wn, j, k, v[u]);
      else
        v[u][0] = v[u][1] = v[u][2] = v[u][3] = 0.0f;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t jq = j0 + 1024 * (int64_t)(r0 + u);
      if (r0 + u >= R || jq >= k) break;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t j = jq + e;
        if (j >= k) break;
        while (nxt <= j) nxt = aoff[++l + 1];
        if (fabsf(fabsf(v[u][e]) - tau[l]) <= xi0) m |= 1ull << (4 * (r0 + u) + e);
      }
    }
  }
  return m;
}

// Pass 1: the flags of every thread (kept for pass 2) and the block's kept count.
template <typename T>
__global__ void __launch_bounds__(256) k_shrink_count(DevState st, const int64_t* act_off,
                                                      const T* __restrict__ wn, float xi0,
                                                      int per, int64_t* blk_cnt,
                                                      uint64_t* __restrict__ flags) {
  __shared__ int64_t aoff[kMaxLayers + 1];
  __shared__ float tau[kMaxLayers];
  __shared__ unsigned long long red[4];
  load_layer_lds(aoff, tau, act_off, st.tau, st.L);
  const int64_t k = aoff[st.L];
  const uint64_t m = shrink_flags(aoff, tau, st.L, wn, k, (int64_t)blockIdx.x * 256 * per, per, xi0);
  flags[(int64_t)blockIdx.x * 256 + threadIdx.x] = m;
  const unsigned long long s = block_sum_u64(__popcll(m), red);
  if (threadIdx.x == 0) blk_cnt[blockIdx.x] = (int64_t)s;
}

// Exclusive scan of the per-block counts in place (one block of 1024 threads,
// 1024 counts per round, the next round's counts loaded ahead); *total = sum.
__device__ __forceinline__ long long wave_incl_scan_i64(long long v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t lo = __shfl_up((uint32_t)v, off, 64);
    const uint32_t hi = __shfl_up((uint32_t)((unsigned long long)v >> 32), off, 64);
    const long long u = (long long)(((unsigned long long)hi << 32) | lo);
    if (lane >= off) v += u;
  }
  return v;
}

__global__ void __launch_bounds__(1024) k_blocks_scan(int64_t* blk_cnt, int64_t nb, int64_t* total) {
  __shared__ long long wsum[16];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  long long carry = 0;
  long long v = tid < nb ? blk_cnt[tid] : 0;
  for (int64_t base = 0; base < nb; base += 1024) {
    const int64_t i = base + tid;
    const int64_t in = i + 1024;
    const long long vn = in < nb ? blk_cnt[in] : 0;       // next round, in flight
    const long long inc = wave_incl_scan_i64(v);
    if (lane == 63) wsum[wid] = inc;
    __syncthreads();
    long long before = 0, round = 0;
#pragma unroll
    for (int w = 0; w < 16; ++w) {
      const long long t = wsum[w];
      before += w < wid ? t : 0;
      round += t;
    }
    if (i < nb) blk_cnt[i] = carry + before + inc - v;
    carry += round;
    v = vn;
    __syncthreads();
  }
  if (tid == 0) *total = carry;
}

// Pass 2: kept entries to their new positions (ordered r, then wave, then lane,
// then e within a block), dropped ones get their code at tau_ref.
template <typename T>
__global__ void __launch_bounds__(256) k_shrink_write(DevState st, const uint32_t* __restrict__ act,
                                                      const int64_t* act_off,
                                                      const T* __restrict__ wn, int per,
                                                      const int64_t* blk_off,
                                                      const uint64_t* __restrict__ flags,
                                                      uint32_t* __restrict__ act_new,
                                                      int64_t* act_off_new, T* wc_new) {
  __shared__ int64_t aoff[kMaxLayers + 1];
  __shared__ int32_t cnt[kShrinkPer];       // kept entries per (r, wave), then their offsets
  for (int i = threadIdx.x; i <= st.L; i += blockDim.x) aoff[i] = act_off[i];
  const int64_t k = act_off[st.L];
  const int64_t base = (int64_t)blockIdx.x * 256 * per;
  const int R = per / 4;
  const uint64_t m = flags[(int64_t)blockIdx.x * 256 + threadIdx.x];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const unsigned long long below = (1ull << lane) - 1ull;
  for (int r = 0; r < R; ++r) {
    const int c = __popcll(m >> (4 * r) & 0xFull);
    // wave total of the lanes' counts: one ballot per bit of the count
    int tot = 0;
#pragma unroll
    for (int b = 0; b < 3; ++b) tot += __popcll(__ballot((c >> b) & 1)) << b;
    if (lane == 0) cnt[4 * r + wid] = tot;
  }
  __syncthreads();
  if (threadIdx.x == 0) {                    // entries are ordered r, then wave, then lane
    int32_t run = 0;
    for (int i = 0; i < R * 4; ++i) {
      const int32_t c = cnt[i];
      cnt[i] = run;
      run += c;
    }
  }
  __syncthreads();
  const int64_t j0 = base + 4 * (int64_t)threadIdx.x;
  if (j0 >= k) return;
  const int64_t boff = blk_off[blockIdx.x];
  int l = layer_of(aoff, st.L, j0);
  int64_t cur = aoff[l], nxt = aoff[l + 1];
  for (int r = 0; r < R; ++r) {
    const int64_t jq = j0 + 1024 * (int64_t)r;
    const uint32_t q = (uint32_t)(m >> (4 * r)) & 0xFu;
    const int c = __popc(q);
    // kept entries of the lower lanes of the wave for this r
    int before = 0;
#pragma unroll
    for (int b = 0; b < 3; ++b) before += __popcll(__ballot((c >> b) & 1) & below) << b;
    if (jq >= k) break;
    uint32_t a[4];
    if (jq + 3 < k) {
      const uint4 v = *reinterpret_cast<const uint4*>(act + jq);
      a[0] = v.x; a[1] = v.y; a[2] = v.z; a[3] = v.w;
    } else {
      for (int e = 0; e < 4; ++e) a[e] = jq + e < k ? act[jq + e] : 0u;
    }
    int64_t pos = boff + cnt[4 * r + wid] + before;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t j = jq + e;
      if (j >= k) break;
      while (nxt <= j) {
        cur = nxt;
        nxt = aoff[++l + 1];
      }
      if (j == cur) act_off_new[l] = pos;     // first entry of layer l
      if ((q >> e) & 1u) {
        act_new[pos] = a[e];
        if (wc_new) wc_new[pos] = wn[j];      // compact mode: the kept latent, list order
        ++pos;
      } else {                                // frozen from now on: its code at tau_ref
        set_code(st.codes, st.code_off[l], a[e], ternary_code(load1(wn, j), st.tau_ref[l]));
      }
    }
  }
}

// Layers that were empty before the shrink take the next layer's offset (one block:
// both offset arrays in LDS, the backward pass over the layers there).
__global__ void __launch_bounds__(256) k_shrink_offsets(const int64_t* act_off,
                                                        int64_t* act_off_new, int L,
                                                        const int64_t* total) {
  __shared__ int64_t o[kMaxLayers + 1], n[kMaxLayers + 1];
  for (int l = threadIdx.x; l <= L; l += blockDim.x) {
    o[l] = act_off[l];
    n[l] = l == L ? *total : act_off_new[l];
  }
  __syncthreads();
  if (threadIdx.x == 0)
    for (int l = L - 1; l >= 0; --l)
      if (o[l] == o[l + 1]) n[l] = n[l + 1];
  __syncthreads();
  for (int l = threadIdx.x; l <= L; l += blockDim.x) act_off_new[l] = n[l];
}

// ---------------------------------------------------------------------------
// Active latents in list order: from the layers (compaction) or, in compact mode,
// from the compact array; out in the latent dtype (to_f32 = 0) or as fp32.
// Entries [j0, j1) of the list.
// ---------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) k_active_values(DevState st, const uint32_t* act,
                                                       const int64_t* act_off, const T* wc,
                                                       int64_t j0, int64_t j1, void* out,
                                                       int to_f32) {
  __shared__ int64_t aoff[kMaxLayers + 1];
  load_offsets(aoff, act_off, st.L);
  for (int64_t j = j0 + (int64_t)blockIdx.x * 256 + threadIdx.x; j < j1;
       j += (int64_t)gridDim.x * 256) {
    float v;
    if (wc) {
      v = load1(wc, j);
    } else {
      const int l = layer_of(aoff, st.L, j);
      v = load1(reinterpret_cast<const T*>(st.w[l]), act[j]);
    }
    if (to_f32)
      reinterpret_cast<float*>(out)[j - j0] = v;
    else
      store1(reinterpret_cast<T*>(out), j - j0, v);   // exact: v is a T value
  }
}

// ---------------------------------------------------------------------------
// Inspection: unpack one layer's codes to int8.
// ---------------------------------------------------------------------------
__global__ void k_unpack(const uint32_t* codes, int64_t n, int8_t* out) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t word = codes[i / 16];
    const uint32_t c = (word >> code_shift((int)(i & 15))) & 3u;
    out[i] = c == 1u ? 1 : (c == 2u ? -1 : 0);
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

// MSE loss of the single-layer workload: one block, fixed reduction order (deterministic).
// Sum of squared errors in fp64 (e = y - t and e * e in fp32), into *out; with
// out32 non-null also the mean rounded to fp32.
__global__ void __launch_bounds__(256) k_mse(const float* y, const float* t, int64_t n,
                                             double* out, float* out32) {
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
  if (threadIdx.x == 0) {
    *out = lds[0];
    if (out32) *out32 = (float)(lds[0] / (double)n);
  }
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

static inline int64_t sparse_grid(int64_t k) {
  return max((int64_t)1, min((int64_t)8192, (k + 256 * kRun - 1) / (256 * kRun)));
}

hipError_t launch_requant(termezo_ctx* c, int patch) {
  const dim3 g((unsigned)c->T), b(kRqStream);
  if (c->dtype == TERMEZO_F32) {
    if (patch)
      hipLaunchKernelGGL((k_requant_tile<float, true>), g, b, 0, c->stream, c->dev(), c->d_act,
                         c->d_wp);
    else
      hipLaunchKernelGGL((k_requant_tile<float, false>), g, b, 0, c->stream, c->dev(), c->d_act,
                         c->d_wp);
  } else {
    if (patch)
      hipLaunchKernelGGL((k_requant_tile<uint16_t, true>), g, b, 0, c->stream, c->dev(), c->d_act,
                         c->d_wp);
    else
      hipLaunchKernelGGL((k_requant_tile<uint16_t, false>), g, b, 0, c->stream, c->dev(), c->d_act,
                         c->d_wp);
  }
  return hipGetLastError();
}

hipError_t launch_requant_guarded(termezo_ctx* c, int force) {
  hipLaunchKernelGGL(k_guard, dim3(1), dim3(256), 0, c->stream, c->dev(), force, c->d_dense_off,
                     c->compact ? 1 : 0, (const int64_t*)c->d_act_off);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (force) return launch_requant(c, 1);      // every layer: one block per tile
  const unsigned g = (unsigned)min(c->T, (int64_t)(c->n_cu > 0 ? 8 * c->n_cu : 2048));
  if (c->dtype == TERMEZO_F32)
    hipLaunchKernelGGL((k_requant_list<float>), dim3(g), dim3(kRqStream), 0, c->stream, c->dev(),
                       c->d_act, c->d_wp, (const int64_t*)c->d_dense_off);
  else
    hipLaunchKernelGGL((k_requant_list<uint16_t>), dim3(g), dim3(kRqStream), 0, c->stream,
                       c->dev(), c->d_act, c->d_wp, (const int64_t*)c->d_dense_off);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (c->k_bound <= 0) return hipSuccess;
  // sparse sets: one scattered code-word update per active; above 1/256 active the
  // code words of the tiles with actives are rewritten whole (0.5 byte per weight)
  if (c->k_bound * 256 <= c->D)
    hipLaunchKernelGGL(k_patch_codes, dim3((unsigned)sparse_grid(c->k_bound)), dim3(256), 0,
                       c->stream, c->dev(), c->d_act, c->d_act_off, c->d_wp);
  else
    hipLaunchKernelGGL(k_patch_tiles, dim3((unsigned)c->T), dim3(kRqThreads), 0, c->stream,
                       c->dev(), c->d_act, c->d_wp);
  return hipGetLastError();
}

hipError_t launch_ref_init(termezo_ctx* c, double xi_lo) {
  hipLaunchKernelGGL(k_ref_init, dim3((unsigned)((c->L + 255) / 256)), dim3(256), 0, c->stream,
                     c->dev(), xi_lo);
  return hipGetLastError();
}

hipError_t launch_ref_after_update(termezo_ctx* c, double xi_lo) {
  hipLaunchKernelGGL(k_ref_after_update, dim3((unsigned)((c->L + 255) / 256)), dim3(256), 0,
                     c->stream, c->dev(), xi_lo);
  return hipGetLastError();
}

hipError_t launch_tile_ranges(termezo_ctx* c) {
  const int64_t g = max((int64_t)1, min((int64_t)2048, (c->T + 1 + 255) / 256));
  hipLaunchKernelGGL(k_tile_ranges, dim3(g), dim3(256), 0, c->stream, c->dev(), c->d_act,
                     c->d_act_off);
  return hipGetLastError();
}


hipError_t launch_perturb_delta(termezo_ctx* c, int64_t k, uint64_t seed, float se, bool pair) {
  if (k <= 0) return hipSuccess;
  const int64_t g = sparse_grid(k);
  const void* wcp = c->mirror ? c->d_wc : nullptr;
  float* wpm = pair ? c->d_wpm : nullptr;
  int64_t* sa = pair ? c->d_S_alt : nullptr;
  float* zs = pair ? c->d_zs : nullptr;
  if (c->dtype == TERMEZO_F32) {
    if (pair)
      hipLaunchKernelGGL((k_perturb_delta<float, true>), dim3(g), dim3(256), 0, c->stream,
                         c->dev(), c->d_act, c->d_act_off, seed, se, c->d_wp,
                         (const float*)wcp, wpm, sa, zs);
    else
      hipLaunchKernelGGL((k_perturb_delta<float, false>), dim3(g), dim3(256), 0, c->stream,
                         c->dev(), c->d_act, c->d_act_off, seed, se, c->d_wp,
                         (const float*)wcp, wpm, sa, zs);
  } else {
    if (pair)
      hipLaunchKernelGGL((k_perturb_delta<uint16_t, true>), dim3(g), dim3(256), 0, c->stream,
                         c->dev(), c->d_act, c->d_act_off, seed, se, c->d_wp,
                         (const uint16_t*)wcp, wpm, sa, zs);
    else
      hipLaunchKernelGGL((k_perturb_delta<uint16_t, false>), dim3(g), dim3(256), 0, c->stream,
                         c->dev(), c->d_act, c->d_act_off, seed, se, c->d_wp,
                         (const uint16_t*)wcp, wpm, sa, zs);
  }
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

hipError_t launch_update(termezo_ctx* c, int64_t k, const SeedList& seeds) {
  if (k <= 0) return hipSuccess;
  const int64_t g = sparse_grid(k);
  void* wcp = c->mirror ? c->d_wc : nullptr;
  const int wl = c->compact ? 0 : 1;           // the caller's latents, unless dropped
  // one direction whose draws the pair pass kept for the same active list: read them
  const float* zs =
      (seeds.K == 1 && c->z_valid && c->z_seed == seeds.s[0]) ? c->d_zs : nullptr;
  if (c->dtype == TERMEZO_F32)
    hipLaunchKernelGGL(k_update<float>, dim3(g), dim3(256), 0, c->stream, c->dev(), c->d_act,
                       c->d_act_off, seeds, (const float*)c->d_scal, c->d_wp, (float*)wcp,
                       wl, zs);
  else
    hipLaunchKernelGGL(k_update<uint16_t>, dim3(g), dim3(256), 0, c->stream, c->dev(), c->d_act,
                       c->d_act_off, seeds, (const float*)c->d_scal, (uint16_t*)c->d_wp,
                       (uint16_t*)wcp, wl, zs);
  return hipGetLastError();
}

hipError_t launch_set_coeffs(termezo_ctx* c, const float* a, int K) {
  CoefList cl = {};
  for (int q = 0; q < K && q < kMaxK; ++q) cl.a[q] = a[q];
  hipLaunchKernelGGL(k_set_coeffs, dim3(1), dim3(kMaxK), 0, c->stream, c->d_scal, cl, K);
  return hipGetLastError();
}

hipError_t launch_es_coeffs(termezo_ctx* c, const float* rewards, int N, float lr,
                            int standardize) {
  hipLaunchKernelGGL(k_es_coeffs, dim3(1), dim3(64), 0, c->stream, rewards, N, lr, standardize,
                     c->d_scal, c->d_err);
  return hipGetLastError();
}

hipError_t launch_coeffs_multi_from_losses(termezo_ctx* c, const float* losses, int K, float eps,
                                           float lr) {
  hipLaunchKernelGGL(k_coeffs_multi_from_losses, dim3(1), dim3(kMaxK), 0, c->stream, losses, K,
                     eps, lr, c->d_scal, c->d_err);
  return hipGetLastError();
}

hipError_t launch_shrink(termezo_ctx* c, int64_t k) {
  // entries per thread: 4 .. kShrinkPer, about 2048 blocks for large lists
  int per = 4;
  while (per < kShrinkPer && k > (int64_t)2048 * 256 * per) per *= 2;
  const int64_t nb = max((int64_t)1, (k + 256 * per - 1) / (256 * per));
  int64_t* total = c->d_blk_cnt + nb;  // blk_cap >= nb + 1
  if (nb > c->blk_cap - 1 || nb * 256 > c->flag_cap) return hipErrorInvalidValue;
  const bool bf = c->dtype == TERMEZO_BF16;
  if (bf)
    hipLaunchKernelGGL(k_shrink_count<uint16_t>, dim3(nb), dim3(256), 0, c->stream, c->dev(),
                       c->d_act_off, (const uint16_t*)c->d_wp, c->xi0, per, c->d_blk_cnt,
                       c->d_shrink_flags);
  else
    hipLaunchKernelGGL(k_shrink_count<float>, dim3(nb), dim3(256), 0, c->stream, c->dev(),
                       c->d_act_off, (const float*)c->d_wp, c->xi0, per, c->d_blk_cnt,
                       c->d_shrink_flags);
  hipLaunchKernelGGL(k_blocks_scan, dim3(1), dim3(1024), 0, c->stream, c->d_blk_cnt, nb, total);
  // offsets of layers without any entry are fixed afterwards
  if (bf)
    hipLaunchKernelGGL(k_shrink_write<uint16_t>, dim3(nb), dim3(256), 0, c->stream, c->dev(),
                       c->d_act, c->d_act_off, (const uint16_t*)c->d_wp, per, c->d_blk_cnt,
                       (const uint64_t*)c->d_shrink_flags, c->d_act_tmp, c->d_act_off_tmp,
                       (uint16_t*)(c->mirror ? c->d_wc_tmp : nullptr));
  else
    hipLaunchKernelGGL(k_shrink_write<float>, dim3(nb), dim3(256), 0, c->stream, c->dev(),
                       c->d_act, c->d_act_off, (const float*)c->d_wp, per, c->d_blk_cnt,
                       (const uint64_t*)c->d_shrink_flags, c->d_act_tmp, c->d_act_off_tmp,
                       (float*)(c->mirror ? c->d_wc_tmp : nullptr));
  hipLaunchKernelGGL(k_shrink_offsets, dim3(1), dim3(256), 0, c->stream, c->d_act_off,
                     c->d_act_off_tmp, c->L, total);
  return hipGetLastError();
}

static unsigned theta_grid(const termezo_ctx* c, int64_t n, int64_t tid0) {
  const int64_t quads = ((tid0 + n + 3) >> 2) - (tid0 >> 2);
  const int64_t cap = (int64_t)(c->n_cu > 0 ? c->n_cu : 256) * 16;
  return (unsigned)max((int64_t)1, min(cap, (quads + 255) / 256));
}

hipError_t launch_theta_pair(termezo_ctx* c, const ThetaHost& t, uint64_t seed, float eps) {
  if (t.n <= 0) return hipSuccess;
  const unsigned g = theta_grid(c, t.n, t.tid0);
  if (t.dtype == TERMEZO_F32)
    hipLaunchKernelGGL(k_theta_pair<float>, dim3(g), dim3(256), 0, c->stream, (const float*)t.data,
                       t.n, t.tid0, seed, eps, (float*)t.plus, (float*)t.minus);
  else
    hipLaunchKernelGGL(k_theta_pair<uint16_t>, dim3(g), dim3(256), 0, c->stream,
                       (const uint16_t*)t.data, t.n, t.tid0, seed, eps, (uint16_t*)t.plus,
                       (uint16_t*)t.minus);
  return hipGetLastError();
}

hipError_t launch_theta_update(termezo_ctx* c, const ThetaHost& t, const SeedList& seeds) {
  if (t.n <= 0) return hipSuccess;
  const unsigned g = theta_grid(c, t.n, t.tid0);
  if (t.dtype == TERMEZO_F32)
    hipLaunchKernelGGL(k_theta_update<float>, dim3(g), dim3(256), 0, c->stream, (float*)t.data, t.n,
                       t.tid0, seeds, (const float*)c->d_scal);
  else
    hipLaunchKernelGGL(k_theta_update<uint16_t>, dim3(g), dim3(256), 0, c->stream,
                       (uint16_t*)t.data, t.n, t.tid0, seeds, (const float*)c->d_scal);
  return hipGetLastError();
}

hipError_t launch_active_values(termezo_ctx* c, int64_t j0, int64_t j1, void* out, int to_f32,
                                int from_compact) {
  if (j1 <= j0) return hipSuccess;
  const unsigned g = (unsigned)max((int64_t)1, min((int64_t)4096, (j1 - j0 + 255) / 256));
  if (c->dtype == TERMEZO_F32)
    hipLaunchKernelGGL(k_active_values<float>, dim3(g), dim3(256), 0, c->stream, c->dev(), c->d_act,
                       c->d_act_off, from_compact ? (const float*)c->d_wc : (const float*)nullptr,
                       j0, j1, out, to_f32);
  else
    hipLaunchKernelGGL(k_active_values<uint16_t>, dim3(g), dim3(256), 0, c->stream, c->dev(),
                       c->d_act, c->d_act_off,
                       from_compact ? (const uint16_t*)c->d_wc : (const uint16_t*)nullptr, j0, j1,
                       out, to_f32);
  return hipGetLastError();
}

hipError_t launch_unpack_layer(termezo_ctx* c, int layer, int8_t* out_dev) {
  const tmz::LayerHost& L = c->layers[layer];
  const int64_t g = max((int64_t)1, min((int64_t)4096, (L.n + 255) / 256));
  hipLaunchKernelGGL(k_unpack, dim3(g), dim3(256), 0, c->stream, c->d_codes + L.code_off, L.n,
                     out_dev);
  return hipGetLastError();
}

hipError_t launch_mse(const float* y, const float* t, int64_t n, double* acc, float* mean32,
                      hipStream_t s) {
  hipLaunchKernelGGL(k_mse, dim3(1), dim3(256), 0, s, y, t, n, acc, mean32);
  return hipGetLastError();
}

}  // namespace tmz
