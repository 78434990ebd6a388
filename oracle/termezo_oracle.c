/*
 * TerMeZO CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously-correct CPU statement of what the TerMeZO sparse
 * zeroth-order step computes (Algorithm 1 of the paper, K = 1; the
 * full-precision parameters theta either frozen or perturbed and updated with
 * the latents).  Only the test-suite, the smoke check and the bench's
 * CPU baseline may load this library; the product path never does.  It shares
 * no code, header, table or helper with the HIP library.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -shared -fPIC
 * (no contraction: every floating-point operation below is one IEEE-754
 * correctly rounded operation, and fmaf is used only where written).  A second
 * build of the same source with -fopenmp runs the loops marked "omp parallel
 * for" over several host threads; each iteration of those loops writes only its
 * own outputs (the one reduction is an exact integer sum), so both builds give
 * identical results.  The plain build ignores the pragmas.
 *
 * Arithmetic conventions fixed here (the paper leaves them open; each reading
 * is listed in the design notes):
 *   - global id (gid): layers enumerated in registration order, each layer
 *     row-major [d_out][d_in]; gid = layer offset + row * d_in + col.
 *   - Gaussian directions z: Philox4x32-10 (Salmon et al., SC'11) keyed by the
 *     64-bit seed, counter (q_lo, q_hi, stream, 0) with q = gid >> 2, followed
 *     by the Box-Muller transform (Box & Muller, 1958) evaluated with the
 *     project's own fp32 logarithm and sin/cos-of-pi routines, whose
 *     coefficients are the Taylor coefficients of atanh, sin and cos rounded
 *     to fp32.
 *   - absmean threshold (Sec. 3, eq. quant): the layer sum of |w| is the exact
 *     integer sum of floor(|w| * 2^36); gamma = S * 2^-36 / n in fp64;
 *     beta = fp32(gamma + delta), tau = fp32(0.5 * (gamma + delta)).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_OK 0
#define ORC_ERR_INVALID 1
#define ORC_ERR_STATE 2
#define ORC_ERR_NUMERIC 5

/* Host threads the parallel loops use: n > 0 sets it (OpenMP build only);
 * returns the count in effect (1 for the plain build). */
int orc_set_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
  return omp_get_max_threads();
#else
  (void)n;
  return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw: "Parallel random numbers: as   */
/* easy as 1, 2, 3", SC'11).  Ten rounds of the 4x32 S-box with two 32-bit   */
/* multipliers; the key is bumped by the Weyl constants between rounds.     */
/* ------------------------------------------------------------------------ */
static const uint32_t PHILOX_M0 = 0xD2511F53u;
static const uint32_t PHILOX_M1 = 0xCD9E8D57u;
static const uint32_t PHILOX_W0 = 0x9E3779B9u; /* golden ratio */
static const uint32_t PHILOX_W1 = 0xBB67AE85u; /* sqrt(3) - 1   */

void orc_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2],
                       uint32_t out[4]) {
  uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
  uint32_t k0 = key_in[0], k1 = key_in[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {
      k0 += PHILOX_W0;
      k1 += PHILOX_W1;
    }
    uint64_t p0 = (uint64_t)PHILOX_M0 * (uint64_t)c0;
    uint64_t p1 = (uint64_t)PHILOX_M1 * (uint64_t)c2;
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t n0 = hi1 ^ c1 ^ k0;
    uint32_t n1 = lo1;
    uint32_t n2 = hi0 ^ c3 ^ k1;
    uint32_t n3 = lo0;
    c0 = n0;
    c1 = n1;
    c2 = n2;
    c3 = n3;
  }
  out[0] = c0;
  out[1] = c1;
  out[2] = c2;
  out[3] = c3;
}

/* ------------------------------------------------------------------------ */
/* Natural logarithm on positive normal fp32 inputs.                         */
/* x = m * 2^e with m in [sqrt(1/2), sqrt(2)); ln m = 2 atanh(f),            */
/* f = (m - 1) / (m + 1), atanh(f) = f + f^3/3 + f^5/5 + ... (|f| < 0.172,   */
/* terms through f^11 leave a truncation error below 1e-10 relative).        */
/* ln x = e * ln2 + ln m with ln2 split so e * LN2_HI is exact.              */
/* ------------------------------------------------------------------------ */
static const float LN2_HI = 0x1.62e000p-1f;
static const float LN2_LO = 0x1.0bfbe8p-15f;
static const float ATANH_C3 = 0x1.555556p-2f;  /* 1/3  */
static const float ATANH_C5 = 0x1.99999ap-3f;  /* 1/5  */
static const float ATANH_C7 = 0x1.24924ap-3f;  /* 1/7  */
static const float ATANH_C9 = 0x1.c71c72p-4f;  /* 1/9  */
static const float ATANH_C11 = 0x1.745d18p-4f; /* 1/11 */

float orc_ln(float x) {
  uint32_t bits;
  memcpy(&bits, &x, 4);
  int e = (int)(bits >> 23) - 127;
  uint32_t frac = bits & 0x7FFFFFu;
  uint32_t mbits = frac | 0x3F800000u; /* m in [1, 2) */
  if (frac > 0x3504F3u) {              /* m > sqrt(2): use m/2, e+1 */
    mbits -= 0x00800000u;
    e += 1;
  }
  float m;
  memcpy(&m, &mbits, 4);
  float f = (m - 1.0f) / (m + 1.0f);
  float two_f = 2.0f * f;
  float t = f * f;
  float p = fmaf(ATANH_C11, t, ATANH_C9);
  p = fmaf(p, t, ATANH_C7);
  p = fmaf(p, t, ATANH_C5);
  p = fmaf(p, t, ATANH_C3);
  float ln_m = fmaf(two_f * t, p, two_f);
  float ef = (float)e;
  return fmaf(ef, LN2_HI, fmaf(ef, LN2_LO, ln_m));
}

/* ------------------------------------------------------------------------ */
/* sin and cos of the angle 2*pi*j/2^24 for an integer j in [0, 2^24).       */
/* With x = 2j/2^24 (so the angle is pi*x, x in [0,2)), the quarter-turn     */
/* index q = round(2x) and remainder r = x - q/2 in [-1/4, 1/4] are exact    */
/* integer operations; sin(pi r), cos(pi r) use their Taylor series          */
/* (through r^11 and r^12), then the quadrant is applied.                    */
/* ------------------------------------------------------------------------ */
static const float PI_HI = 0x1.921fb6p+1f;
static const float PI_LO = -0x1.777a5cp-24f;
static const float SINPI_C3 = -0x1.4abbcep+2f;  /* -pi^3/3!   */
static const float SINPI_C5 = 0x1.466bc6p+1f;   /*  pi^5/5!   */
static const float SINPI_C7 = -0x1.32d2ccp-1f;  /* -pi^7/7!   */
static const float SINPI_C9 = 0x1.507834p-4f;   /*  pi^9/9!   */
static const float SINPI_C11 = -0x1.e30750p-8f; /* -pi^11/11! */
static const float COSPI_C2 = -0x1.3bd3ccp+2f;  /* -pi^2/2!   */
static const float COSPI_C4 = 0x1.03c1f0p+2f;   /*  pi^4/4!   */
static const float COSPI_C6 = -0x1.55d3c8p+0f;  /* -pi^6/6!   */
static const float COSPI_C8 = 0x1.e1f506p-3f;   /*  pi^8/8!   */
static const float COSPI_C10 = -0x1.a6d1f2p-6f; /* -pi^10/10! */
static const float COSPI_C12 = 0x1.f9d38ap-10f; /*  pi^12/12! */

void orc_sincos_turn24(uint32_t j, float* s_out, float* c_out) {
  uint32_t q = (j + (1u << 21)) >> 22; /* 0..4 */
  int32_t rem = (int32_t)j - (int32_t)(q << 22);
  float r = (float)rem * 0x1p-23f;
  float t = r * r;
  float ps = fmaf(SINPI_C11, t, SINPI_C9);
  ps = fmaf(ps, t, SINPI_C7);
  ps = fmaf(ps, t, SINPI_C5);
  ps = fmaf(ps, t, SINPI_C3);
  float sin_r = fmaf(r * t, ps, fmaf(r, PI_HI, r * PI_LO));
  float pc = fmaf(COSPI_C12, t, COSPI_C10);
  pc = fmaf(pc, t, COSPI_C8);
  pc = fmaf(pc, t, COSPI_C6);
  pc = fmaf(pc, t, COSPI_C4);
  pc = fmaf(pc, t, COSPI_C2);
  float cos_r = fmaf(t, pc, 1.0f);
  float s, c;
  switch (q & 3u) {
    case 0: s = sin_r; c = cos_r; break;
    case 1: s = cos_r; c = -sin_r; break;
    case 2: s = -sin_r; c = -cos_r; break;
    default: s = -cos_r; c = sin_r; break;
  }
  *s_out = s;
  *c_out = c;
}

/* ------------------------------------------------------------------------ */
/* Standard-normal direction z for one global id (Algorithm 1 draws          */
/* z ~ N(0, I) from the seed s_{t,k}; the draw is a pure function of         */
/* (seed, stream, gid), so it can be regenerated for the update).            */
/* One Philox call at q = gid >> 2 feeds two Box-Muller pairs:               */
/*   gid&3 = 0 -> R(x0) cos(x1), 1 -> R(x0) sin(x1),                         */
/*           2 -> R(x2) cos(x3), 3 -> R(x2) sin(x3),                         */
/* u1 = ((x >> 8) + 1) 2^-24 in (0,1],  angle = 2 pi (x' >> 8) 2^-24.        */
/* ------------------------------------------------------------------------ */
float orc_gauss_one(uint64_t seed, uint32_t stream, uint64_t gid) {
  uint64_t q = gid >> 2;
  uint32_t ctr[4] = {(uint32_t)q, (uint32_t)(q >> 32), stream, 0u};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t x[4];
  orc_philox4x32_10(ctr, key, x);
  unsigned lane = (unsigned)(gid & 3u);
  uint32_t xr = (lane < 2) ? x[0] : x[2];
  uint32_t xa = (lane < 2) ? x[1] : x[3];
  float u1 = (float)((xr >> 8) + 1u) * 0x1p-24f;
  float radius = sqrtf(-2.0f * orc_ln(u1));
  float s, c;
  orc_sincos_turn24(xa >> 8, &s, &c);
  return (lane & 1u) ? radius * s : radius * c;
}

void orc_gauss(uint64_t seed, uint32_t stream, const int64_t* gids, int64_t n,
               float* z) {
#pragma omp parallel for
  for (int64_t i = 0; i < n; ++i) z[i] = orc_gauss_one(seed, stream, (uint64_t)gids[i]);
}

void orc_gauss_range(uint64_t seed, uint32_t stream, int64_t gid0, int64_t n,
                     float* z) {
#pragma omp parallel for
  for (int64_t i = 0; i < n; ++i) z[i] = orc_gauss_one(seed, stream, (uint64_t)(gid0 + i));
}

void orc_ln_array(const float* x, int64_t n, float* y) {
  for (int64_t i = 0; i < n; ++i) y[i] = orc_ln(x[i]);
}

void orc_sincos_turn24_array(const uint32_t* j, int64_t n, float* s, float* c) {
  for (int64_t i = 0; i < n; ++i) orc_sincos_turn24(j[i], &s[i], &c[i]);
}

/* ------------------------------------------------------------------------ */
/* Absmean threshold (Sec. 3, eq. quant and the definition of tau^l).        */
/* ------------------------------------------------------------------------ */
/* floor(|w| * 2^36): exact in fp64 (a power-of-two scaling of an fp32). */
int64_t orc_fix_abs(float w) {
  double a = fabs((double)w) * 68719476736.0;
  return (int64_t)floor(a);
}

/* Exact integer sum S = sum_i floor(|w_i| 2^36).  Every |w_i| must be finite
 * and below 4 so that S stays inside int64 for layers of up to 2^25 weights. */
int orc_layer_abs_sum(const float* w, int64_t n, int64_t* S_out) {
  int64_t S = 0, bad = 0;
#pragma omp parallel for reduction(+ : S, bad)
  for (int64_t i = 0; i < n; ++i) {
    if (!isfinite(w[i]) || fabsf(w[i]) >= 4.0f)
      bad += 1;
    else
      S += orc_fix_abs(w[i]);
  }
  if (bad) return ORC_ERR_NUMERIC;
  *S_out = S;
  return ORC_OK;
}

/* gamma = mean |w| = S 2^-36 / n;  beta = gamma + delta;  tau = beta / 2. */
void orc_threshold(int64_t S, int64_t n, float delta, float* tau, float* beta) {
  double gamma = ((double)S * 0x1p-36) / (double)n;
  double b = gamma + (double)delta;
  *beta = (float)b;
  *tau = (float)(0.5 * b);
}

/* Ternary quantiser Q (eq. quant): +1 above tau, -1 below -tau, 0 otherwise. */
void orc_quantize(const float* w, int64_t n, float tau, int8_t* codes) {
#pragma omp parallel for
  for (int64_t i = 0; i < n; ++i) {
    if (w[i] > tau)
      codes[i] = 1;
    else if (w[i] < -tau)
      codes[i] = -1;
    else
      codes[i] = 0;
  }
}

/* Boundary distance (eq. distance): min(|w - tau|, |w + tau|) = ||w| - tau|. */
void orc_distance(const float* w, int64_t n, float tau, float* d) {
#pragma omp parallel for
  for (int64_t i = 0; i < n; ++i) d[i] = fabsf(fabsf(w[i]) - tau);
}

/* ------------------------------------------------------------------------ */
/* Initial selection (eq. selection_init): the k smallest distances over all */
/* layers, ordered by (distance, gid).  xi0 is the distance of the k-th.     */
/* With inclusive != 0 every gid whose distance equals xi0 is also kept      */
/* (the literal "d <= xi0" set).                                             */
/* ------------------------------------------------------------------------ */
typedef struct {
  float d;
  int64_t gid;
} orc_key;

static int orc_key_cmp(const void* a, const void* b) {
  const orc_key* x = (const orc_key*)a;
  const orc_key* y = (const orc_key*)b;
  if (x->d < y->d) return -1;
  if (x->d > y->d) return 1;
  if (x->gid < y->gid) return -1;
  if (x->gid > y->gid) return 1;
  return 0;
}

static int orc_i64_cmp(const void* a, const void* b) {
  int64_t x = *(const int64_t*)a, y = *(const int64_t*)b;
  return (x > y) - (x < y);
}

/* d: all distances in gid order (length D).  out: capacity cap, receives the
 * selected gids in ascending gid order.  Returns ORC_ERR_INVALID if cap is
 * too small, ORC_ERR_STATE if k == 0. */
int orc_select(const float* d, int64_t D, int64_t k, int inclusive, int64_t* out,
               int64_t cap, int64_t* n_out, float* xi0) {
  if (k <= 0 || k > D) return ORC_ERR_STATE;
  orc_key* keys = (orc_key*)malloc((size_t)D * sizeof(orc_key));
  if (!keys) return ORC_ERR_INVALID;
  for (int64_t i = 0; i < D; ++i) {
    keys[i].d = d[i];
    keys[i].gid = i;
  }
  qsort(keys, (size_t)D, sizeof(orc_key), orc_key_cmp);
  float xi = keys[k - 1].d;
  int64_t n = k;
  if (inclusive)
    while (n < D && keys[n].d == xi) ++n;
  if (n > cap) {
    free(keys);
    return ORC_ERR_INVALID;
  }
  for (int64_t i = 0; i < n; ++i) out[i] = keys[i].gid;
  free(keys);
  qsort(out, (size_t)n, sizeof(int64_t), orc_i64_cmp);
  *n_out = n;
  *xi0 = xi;
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Perturbed latents (Algorithm 1, the +eps / -eps evaluations), written     */
/* functionally: w'_i = fma(sign*eps, z_i, w_i) on the active set, w'_i = w_i */
/* elsewhere.  act: ascending local indices of the layer's active set;       */
/* gid0: global id of the layer's first element.                             */
/* ------------------------------------------------------------------------ */
void orc_perturbed_layer(const float* w, int64_t n, const int64_t* act, int64_t k,
                         int64_t gid0, uint64_t seed, float eps, int sign, float* w_out) {
  float se = (float)sign * eps;
  memcpy(w_out, w, (size_t)n * sizeof(float));
#pragma omp parallel for
  for (int64_t j = 0; j < k; ++j) {
    int64_t i = act[j];
    float z = orc_gauss_one(seed, 0u, (uint64_t)(gid0 + i));
    w_out[i] = fmaf(se, z, w[i]);
  }
}

/* ------------------------------------------------------------------------ */
/* BitLinear forward with 8-bit activations.                                 */
/* Per token row m: a_m = max_k |x|, s_m = 127 / max(a_m, 1e-5),             */
/* x_q = clamp(rne(x * s_m), -128, 127).                                     */
/* acc[m][n] = sum_k x_q[m][k] * c[n][k]  (exact, int32);                    */
/* y[m][n] = float(acc) * (beta / s_m).                                      */
/* ------------------------------------------------------------------------ */
void orc_act_quant(const float* x, int64_t M, int64_t K, int8_t* xq, float* s) {
#pragma omp parallel for
  for (int64_t m = 0; m < M; ++m) {
    const float* row = x + m * K;
    float a = 0.0f;
    for (int64_t k = 0; k < K; ++k) a = fmaxf(a, fabsf(row[k]));
    float sm = 127.0f / fmaxf(a, 1e-5f);
    s[m] = sm;
    for (int64_t k = 0; k < K; ++k) {
      float v = rintf(row[k] * sm);
      if (v > 127.0f) v = 127.0f;
      if (v < -128.0f) v = -128.0f;
      xq[m * K + k] = (int8_t)v;
    }
  }
}

void orc_bitlinear(const int8_t* xq, const float* s, const int8_t* codes, float beta,
                   int64_t M, int64_t K, int64_t N, int32_t* acc, float* y) {
#pragma omp parallel for
  for (int64_t m = 0; m < M; ++m) {
    float r = beta / s[m];
    for (int64_t n = 0; n < N; ++n) {
      int32_t a = 0;
      const int8_t* xr = xq + m * K;
      const int8_t* cr = codes + n * K;
      for (int64_t k = 0; k < K; ++k) a += (int32_t)xr[k] * (int32_t)cr[k];
      if (acc) acc[m * N + n] = a;
      if (y) y[m * N + n] = (float)a * r;
    }
  }
}

/* ------------------------------------------------------------------------ */
/* Masked update (Algorithm 1, weight update with eta/K, K = 1):             */
/* w_i <- round(fma(a, z_i, w_i)) with a = -(lr * g), for i in the active    */
/* set only; round is RNE to bfloat16 for bf16 storage, identity for fp32.   */
/* ------------------------------------------------------------------------ */
static float orc_round_bf16(float v) {
  uint32_t b;
  memcpy(&b, &v, 4);
  if ((b & 0x7F800000u) == 0x7F800000u) { /* inf / nan: keep (nan stays nan) */
    if (b & 0x7FFFFFu) b |= 0x00400000u;
    b &= 0xFFFF0000u;
  } else {
    uint32_t lsb = (b >> 16) & 1u;
    b += 0x7FFFu + lsb;
    b &= 0xFFFF0000u;
  }
  float r;
  memcpy(&r, &b, 4);
  return r;
}

void orc_bf16_round_array(const float* x, int64_t n, float* y) {
#pragma omp parallel for
  for (int64_t i = 0; i < n; ++i) y[i] = orc_round_bf16(x[i]);
}

void orc_update_layer(float* w, const int64_t* act, int64_t k, int64_t gid0,
                      uint64_t seed, float lr, float g, int bf16_storage) {
  float a = -(lr * g);
#pragma omp parallel for
  for (int64_t j = 0; j < k; ++j) {
    int64_t i = act[j];
    float z = orc_gauss_one(seed, 0u, (uint64_t)(gid0 + i));
    float v = fmaf(a, z, w[i]);
    w[i] = bf16_storage ? orc_round_bf16(v) : v;
  }
}

/* Shrink-only set update (eq. selection_): keep the active indices whose
 * distance to the current threshold is still within xi0.  In-place, order
 * preserving; returns the new count. */
int64_t orc_shrink_layer(const float* w, int64_t* act, int64_t k, float tau, float xi0) {
  int64_t n = 0;
  for (int64_t j = 0; j < k; ++j) {
    int64_t i = act[j];
    float d = fabsf(fabsf(w[i]) - tau);
    if (d <= xi0) act[n++] = i;
  }
  return n;
}

/* ------------------------------------------------------------------------ */
/* Full-precision parameters theta (Sec. 3: embeddings, norms, LM head),     */
/* perturbed and updated densely with the latents (Algorithm 1): from the    */
/* same seed, z_theta is drawn on Philox stream 1 at theta ids tid0 + i      */
/* (tensors enumerated in registration order).  The perturbed values are     */
/* materialised in the storage type for the forward pass:                    */
/*   theta'_i = rnd(fma(sign * eps, z_i, theta_i));                          */
/* the update is theta_i <- rnd(fma(-(lr g), z_i, theta_i)), with rnd the    */
/* round-to-nearest-even bf16 conversion for bf16 storage, else identity.    */
/* ------------------------------------------------------------------------ */
void orc_theta_perturbed(const float* theta, int64_t n, int64_t tid0, uint64_t seed,
                         float eps, int sign, int bf16_storage, float* out) {
  float se = (float)sign * eps;
#pragma omp parallel for
  for (int64_t i = 0; i < n; ++i) {
    float z = orc_gauss_one(seed, 1u, (uint64_t)(tid0 + i));
    float v = fmaf(se, z, theta[i]);
    out[i] = bf16_storage ? orc_round_bf16(v) : v;
  }
}

void orc_theta_update(float* theta, int64_t n, int64_t tid0, uint64_t seed, float lr, float g,
                      int bf16_storage) {
  float a = -(lr * g);
#pragma omp parallel for
  for (int64_t i = 0; i < n; ++i) {
    float z = orc_gauss_one(seed, 1u, (uint64_t)(tid0 + i));
    float v = fmaf(a, z, theta[i]);
    theta[i] = bf16_storage ? orc_round_bf16(v) : v;
  }
}

/* ------------------------------------------------------------------------ */
/* K perturbation directions per step (Algorithm 1): the K estimates are     */
/* taken at w_t, then the K updates w <- w - (eta/K) g_k m (.) z_k are       */
/* applied in order.  Here the chain runs in fp32 and is rounded to the      */
/* storage type once:  v = w;  v = fma(a_k, z_k, v) for k = 1..K;            */
/* w = rnd(v),  with a_k = -((lr / K) g_k) (lr / K one fp32 division).       */
/* For fp32 storage this equals K single updates applied one after another.  */
/* ------------------------------------------------------------------------ */
float orc_multi_coeff(float lr, int K, float g) {
  float c = lr / (float)K;
  return -(c * g);
}

void orc_update_layer_multi(float* w, const int64_t* act, int64_t k, int64_t gid0,
                            const uint64_t* seeds, const float* g, int K, float lr,
                            int bf16_storage) {
#pragma omp parallel for
  for (int64_t j = 0; j < k; ++j) {
    int64_t i = act[j];
    float v = w[i];
    for (int q = 0; q < K; ++q) {
      float z = orc_gauss_one(seeds[q], 0u, (uint64_t)(gid0 + i));
      v = fmaf(orc_multi_coeff(lr, K, g[q]), z, v);
    }
    w[i] = bf16_storage ? orc_round_bf16(v) : v;
  }
}

void orc_theta_update_multi(float* theta, int64_t n, int64_t tid0, const uint64_t* seeds,
                            const float* g, int K, float lr, int bf16_storage) {
#pragma omp parallel for
  for (int64_t i = 0; i < n; ++i) {
    float v = theta[i];
    for (int q = 0; q < K; ++q) {
      float z = orc_gauss_one(seeds[q], 1u, (uint64_t)(tid0 + i));
      v = fmaf(orc_multi_coeff(lr, K, g[q]), z, v);
    }
    theta[i] = bf16_storage ? orc_round_bf16(v) : v;
  }
}

/* ------------------------------------------------------------------------ */
/* Evolution strategies restricted to the mask (appendix on RL-based        */
/* fine-tuning): N one-sided perturbations w + sigma m (.) z_n, a reward R_n */
/* for each, then the reward-weighted sum of the directions,                 */
/*   w <- w + (eta / N) sum_n Rt_n m (.) z_n,                                */
/* where Rt are the rewards standardised over the population (z-score, the   */
/* population standard deviation; all zero when that deviation is zero, so   */
/* N = 1 or equal rewards leave w unchanged), or the raw rewards.            */
/* Standardisation in fp64, in index order:                                  */
/*   mu = (sum R) / N;  var = (sum (R - mu)^2) / N;  sd = sqrt(var);         */
/*   Rt_n = fp32((R_n - mu) / sd).                                           */
/* Coefficients a_n = (eta / N) * Rt_n in fp32 (eta / N one fp32 division); */
/* the fp32 chain v = fma(a_n, z_n, v) over n, rounded to storage once.     */
/* ------------------------------------------------------------------------ */
void orc_es_standardize(const float* r, int N, float* out) {
  double mu = 0.0, var = 0.0;
  for (int n = 0; n < N; ++n) mu += (double)r[n];
  mu /= (double)N;
  for (int n = 0; n < N; ++n) {
    double d = (double)r[n] - mu;
    var += d * d;
  }
  var /= (double)N;
  double sd = sqrt(var);
  for (int n = 0; n < N; ++n) out[n] = sd > 0.0 ? (float)(((double)r[n] - mu) / sd) : 0.0f;
}

void orc_es_coeffs(const float* r, int N, float lr, int standardize, float* a) {
  float c = lr / (float)N;
  for (int n = 0; n < N; ++n) a[n] = r[n];
  if (standardize) orc_es_standardize(r, N, a);
  for (int n = 0; n < N; ++n) a[n] = c * a[n];
}

void orc_update_layer_coeffs(float* w, const int64_t* act, int64_t k, int64_t gid0,
                             const uint64_t* seeds, const float* a, int N, int bf16_storage) {
#pragma omp parallel for
  for (int64_t j = 0; j < k; ++j) {
    int64_t i = act[j];
    float v = w[i];
    for (int n = 0; n < N; ++n) v = fmaf(a[n], orc_gauss_one(seeds[n], 0u, (uint64_t)(gid0 + i)), v);
    w[i] = bf16_storage ? orc_round_bf16(v) : v;
  }
}

void orc_theta_update_coeffs(float* theta, int64_t n, int64_t tid0, const uint64_t* seeds,
                             const float* a, int N, int bf16_storage) {
#pragma omp parallel for
  for (int64_t i = 0; i < n; ++i) {
    float v = theta[i];
    for (int q = 0; q < N; ++q) v = fmaf(a[q], orc_gauss_one(seeds[q], 1u, (uint64_t)(tid0 + i)), v);
    theta[i] = bf16_storage ? orc_round_bf16(v) : v;
  }
}
