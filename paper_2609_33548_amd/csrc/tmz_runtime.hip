// C ABI of the TerMeZO library: validation, buffer ownership, launch order.
#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <string>

#include "tmz_internal.h"

using namespace tmz;

// Scratch of termezo_bitlinear_forward_noalloc: the int8 activations [M][d_in] of one
// call, then (at the next 256-byte boundary) its per-token scales [M].  Each device
// holds its own copy until the process ends.  In host code the name is only a
// host-side stand-in: the device address comes from hipGetSymbolAddress, taken once
// per device at context creation.
constexpr int64_t kNoAllocScratchBytes = int64_t(16) << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices] = {};

// Device address of `scratch` on `device`, which must be the current device.
hipError_t noalloc_scratch_address(int device, void** out) {
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_addr[device] = p;
  }
  *out = g_scratch_addr[device];
  return hipSuccess;
}

termezo_status fail(termezo_ctx* c, termezo_status st, const std::string& msg) {
  if (c) c->last_error = msg;
  return st;
}

termezo_status hip_fail(termezo_ctx* c, hipError_t e, const char* what) {
  const termezo_status st = e == hipErrorOutOfMemory ? TERMEZO_ERR_OOM : TERMEZO_ERR_DEVICE;
  return fail(c, st, std::string(what) + ": " + hipGetErrorString(e));
}

#define TMZ_HIP(c, expr)                                 \
  do {                                                   \
    hipError_t _e = (expr);                              \
    if (_e != hipSuccess) return hip_fail((c), _e, #expr); \
  } while (0)

template <typename P>
hipError_t dalloc(P** p, size_t count) {
  void* v = nullptr;
  hipError_t e = hipMalloc(&v, count * sizeof(P) > 0 ? count * sizeof(P) : 1);
  *p = static_cast<P*>(v);
  return e;
}

template <typename P>
void dfree(P*& p) {
  if (p) (void)hipFree((void*)p);
  p = nullptr;
}

size_t dtype_size(termezo_dtype t) {
  switch (t) {
    case TERMEZO_F32: return 4;
    case TERMEZO_BF16: return 2;
    case TERMEZO_I8: return 1;
    case TERMEZO_I32: return 4;
  }
  return 0;
}

// Wait for the stream and surface a deferred numeric error.
termezo_status sync_and_check(termezo_ctx* c) {
  TMZ_HIP(c, hipStreamSynchronize(c->stream));
  int32_t err = 0;
  TMZ_HIP(c, hipMemcpy(&err, c->d_err, sizeof(err), hipMemcpyDeviceToHost));
  if (err) {
    const int32_t zero = 0;
    TMZ_HIP(c, hipMemcpy(c->d_err, &zero, sizeof(zero), hipMemcpyHostToDevice));
    std::string msg;
    if (err & 1) msg += "a latent (or perturbed latent) is non-finite or has |w| >= 4; ";
    if (err & 2) msg += "a projected gradient or update coefficient is not finite; ";
    if (err & 4)
      msg += "compact mode: a layer's threshold moved by more than its frozen latents' margin "
             "(their codes were kept; rebuild the mask from full latents); ";
    if (err & 8) msg += "model_loss: a token id lies outside [0, vocab) (read as id 0); ";
    return fail(c, (err & ~8) ? TERMEZO_ERR_NUMERIC : TERMEZO_ERR_INVALID_ARG, msg);
  }
  return TERMEZO_OK;
}

termezo_status ensure_active_capacity(termezo_ctx* c, int64_t k) {
  if (k <= c->act_cap && c->d_act) return TERMEZO_OK;
  dfree(c->d_act);
  dfree(c->d_act_tmp);
  dfree(c->d_wp);
  dfree(c->d_wpm);
  dfree(c->d_zs);
  dfree(c->d_blk_cnt);
  dfree(c->d_shrink_flags);
  c->act_cap = 0;
  c->pair_valid = false;
  c->z_valid = false;
  const int64_t cap = k > 0 ? k : 1;
  TMZ_HIP(c, dalloc(&c->d_act, (size_t)cap));
  TMZ_HIP(c, dalloc(&c->d_act_tmp, (size_t)cap));
  TMZ_HIP(c, dalloc(&c->d_wp, (size_t)cap));
  TMZ_HIP(c, dalloc(&c->d_wpm, (size_t)cap));
  TMZ_HIP(c, dalloc(&c->d_zs, (size_t)cap));
  c->blk_cap = cap / 1024 + 2;   // shrink blocks hold at least 1024 entries (4 per thread)
  TMZ_HIP(c, dalloc(&c->d_blk_cnt, (size_t)c->blk_cap));
  // shrink flags, one word per thread: at most 2048 blocks below 64 entries per thread
  c->flag_cap = std::max((int64_t)2048 * 256, cap / 64) + 256;
  TMZ_HIP(c, dalloc(&c->d_shrink_flags, (size_t)c->flag_cap));
  c->act_cap = cap;
  return TERMEZO_OK;
}

// The list-order copy of the active latents (and the buffer the shrink compacts it into).
termezo_status ensure_wc_capacity(termezo_ctx* c, int64_t k) {
  if (k <= c->wc_cap && c->d_wc) return TERMEZO_OK;
  if (c->d_wc) (void)hipFree(c->d_wc);
  if (c->d_wc_tmp) (void)hipFree(c->d_wc_tmp);
  c->d_wc = c->d_wc_tmp = nullptr;
  c->wc_cap = 0;
  const size_t bytes = (size_t)(k > 0 ? k : 1) * dtype_size(c->dtype);
  TMZ_HIP(c, hipMalloc(&c->d_wc, bytes));
  TMZ_HIP(c, hipMalloc(&c->d_wc_tmp, bytes));
  c->wc_cap = k > 0 ? k : 1;
  return TERMEZO_OK;
}

termezo_status ensure_xq_capacity(termezo_ctx* c, int64_t M, int64_t K) {
  const int64_t need = M * K;
  if (need > c->xq_cap) {
    dfree(c->d_xq);
    c->xq_cap = 0;
    TMZ_HIP(c, dalloc(&c->d_xq, (size_t)need));
    c->xq_cap = need;
  }
  return TERMEZO_OK;
}

termezo_status ensure_xs_capacity(termezo_ctx* c, int64_t M) {
  if (M > c->xs_cap) {
    dfree(c->d_xs);
    dfree(c->d_xrs);
    c->xs_cap = 0;
    TMZ_HIP(c, dalloc(&c->d_xs, (size_t)M));
    TMZ_HIP(c, dalloc(&c->d_xrs, (size_t)M));
    c->xs_cap = M;
  }
  return TERMEZO_OK;
}

void free_all(termezo_ctx* c) {
  dfree(c->d_wptr);
  dfree(c->d_n);
  dfree(c->d_gid0);
  dfree(c->d_code_off);
  dfree(c->d_tile_layer);
  dfree(c->d_tile_start);
  dfree(c->d_tile0);
  dfree(c->d_tile_act);
  dfree(c->d_codes);
  dfree(c->d_codes_snap);
  dfree(c->d_beta_snap);
  dfree(c->d_S_clean);
  dfree(c->d_S_cur);
  dfree(c->d_S_alt);
  dfree(c->d_tau);
  dfree(c->d_beta);
  dfree(c->d_tau_cur);
  dfree(c->d_beta_cur);
  dfree(c->d_tau_ref);
  dfree(c->d_mref);
  dfree(c->d_need);
  dfree(c->d_dense_off);
  dfree(c->d_err);
  dfree(c->d_act);
  dfree(c->d_act_tmp);
  dfree(c->d_act_off);
  dfree(c->d_act_off_tmp);
  dfree(c->d_wp);
  dfree(c->d_wpm);
  dfree(c->d_zs);
  dfree(c->d_hist);
  dfree(c->d_sel);
  dfree(c->d_tile_cnt);
  dfree(c->d_tile_out);
  dfree(c->d_tile_eqb);
  dfree(c->d_blk_cnt);
  dfree(c->d_shrink_flags);
  dfree(c->d_loss);
  dfree(c->d_scal);
  dfree(c->d_xq);
  dfree(c->d_xs);
  dfree(c->d_xrs);
  if (c->d_wc) (void)hipFree(c->d_wc);
  if (c->d_wc_tmp) (void)hipFree(c->d_wc_tmp);
  c->d_wc = c->d_wc_tmp = nullptr;
  for (ThetaHost& t : c->theta) {
    if (t.plus) (void)hipFree(t.plus);
    if (t.minus) (void)hipFree(t.minus);
  }
  c->theta.clear();
}

bool finite(float v) { return std::isfinite(v); }

}  // namespace

extern "C" {

termezo_status termezo_create(const termezo_layer* layers, int32_t n_layers,
                              termezo_dtype latent_dtype, void* hip_stream, termezo_ctx** out) {
  if (!out) return TERMEZO_ERR_INVALID_ARG;
  *out = nullptr;
  if (!layers || n_layers <= 0 || n_layers > kMaxLayers) return TERMEZO_ERR_INVALID_ARG;
  if (latent_dtype != TERMEZO_F32 && latent_dtype != TERMEZO_BF16) return TERMEZO_ERR_INVALID_ARG;
  for (int32_t l = 0; l < n_layers; ++l) {
    const termezo_layer& L = layers[l];
    if (!L.latent || L.d_out <= 0 || L.d_in <= 0 || L.d_in % 16 != 0) return TERMEZO_ERR_INVALID_ARG;
    if ((reinterpret_cast<uintptr_t>(L.latent) & 15u) != 0) return TERMEZO_ERR_INVALID_ARG;
    if (L.d_out > (int64_t(1) << 25) / L.d_in) return TERMEZO_ERR_INVALID_ARG;  // n <= 2^25
  }
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || ndev <= 0) return TERMEZO_ERR_DEVICE;

  termezo_ctx* c = new (std::nothrow) termezo_ctx();
  if (!c) return TERMEZO_ERR_OOM;
  if (hipGetDevice(&c->device) != hipSuccess) {
    delete c;
    return TERMEZO_ERR_DEVICE;
  }
  c->stream = static_cast<hipStream_t>(hip_stream);
  c->dtype = latent_dtype;
  c->L = n_layers;

  std::vector<void*> wptr(n_layers);
  std::vector<int64_t> n(n_layers), gid0(n_layers), code_off(n_layers), tile0(n_layers);
  std::vector<int32_t> tile_layer;
  int64_t D = 0, words = 0;
  for (int32_t l = 0; l < n_layers; ++l) {
    LayerHost h;
    h.w = layers[l].latent;
    h.d_out = layers[l].d_out;
    h.d_in = layers[l].d_in;
    h.n = h.d_out * h.d_in;
    h.gid0 = D;
    h.code_off = words;
    h.tile0 = (int64_t)tile_layer.size();
    h.ntiles = (h.n + kTile - 1) / kTile;
    for (int64_t t = 0; t < h.ntiles; ++t) {
      tile_layer.push_back(l);
      c->tile_start_host.push_back(t * kTile);
    }
    c->layers.push_back(h);
    wptr[l] = h.w;
    n[l] = h.n;
    gid0[l] = h.gid0;
    code_off[l] = h.code_off;
    tile0[l] = h.tile0;
    D += h.n;
    words += h.n / 16;
  }
  c->D = D;
  c->T = (int64_t)tile_layer.size();
  c->code_words = words;

  termezo_status st = TERMEZO_OK;
  auto chk = [&](hipError_t e, const char* what) {
    if (e != hipSuccess && st == TERMEZO_OK) st = hip_fail(c, e, what);
  };
  chk(dalloc(&c->d_wptr, n_layers), "alloc");
  chk(dalloc(&c->d_n, n_layers), "alloc");
  chk(dalloc(&c->d_gid0, n_layers), "alloc");
  chk(dalloc(&c->d_code_off, n_layers), "alloc");
  chk(dalloc(&c->d_tile_layer, (size_t)c->T), "alloc");
  chk(dalloc(&c->d_tile_start, (size_t)c->T), "alloc");
  chk(dalloc(&c->d_tile0, n_layers), "alloc");
  chk(dalloc(&c->d_tile_act, (size_t)c->T + 1), "alloc");
  chk(dalloc(&c->d_codes, (size_t)words), "alloc codes");
  chk(dalloc(&c->d_S_clean, n_layers), "alloc");
  chk(dalloc(&c->d_S_cur, n_layers), "alloc");
  chk(dalloc(&c->d_S_alt, n_layers), "alloc");
  chk(dalloc(&c->d_tau, n_layers), "alloc");
  chk(dalloc(&c->d_beta, n_layers), "alloc");
  chk(dalloc(&c->d_tau_cur, n_layers), "alloc");
  chk(dalloc(&c->d_beta_cur, n_layers), "alloc");
  chk(dalloc(&c->d_tau_ref, n_layers), "alloc");
  chk(dalloc(&c->d_mref, n_layers), "alloc");
  chk(dalloc(&c->d_need, n_layers), "alloc");
  chk(dalloc(&c->d_dense_off, (size_t)n_layers + 1), "alloc");
  chk(dalloc(&c->d_err, 1), "alloc");
  chk(noalloc_scratch_address(c->device, &c->noalloc_scratch), "hipGetSymbolAddress(scratch)");
  chk(dalloc(&c->d_act_off, (size_t)n_layers + 1), "alloc");
  chk(dalloc(&c->d_act_off_tmp, (size_t)n_layers + 1), "alloc");
  chk(dalloc(&c->d_hist, kHistBins), "alloc");
  chk(dalloc(&c->d_sel, 1), "alloc");
  chk(dalloc(&c->d_tile_cnt, (size_t)(2 * c->T)), "alloc");
  chk(dalloc(&c->d_tile_out, (size_t)c->T), "alloc");
  chk(dalloc(&c->d_tile_eqb, (size_t)c->T), "alloc");
  chk(dalloc(&c->d_loss, 4), "alloc");
  chk(dalloc(&c->d_scal, kScalLen), "alloc");
  chk(hipDeviceGetAttribute(&c->n_cu, hipDeviceAttributeMultiprocessorCount, c->device),
      "device attribute");
  if (st == TERMEZO_OK) {
    chk(hipMemcpy(c->d_wptr, wptr.data(), n_layers * sizeof(void*), hipMemcpyHostToDevice), "copy");
    chk(hipMemcpy(c->d_n, n.data(), n_layers * sizeof(int64_t), hipMemcpyHostToDevice), "copy");
    chk(hipMemcpy(c->d_gid0, gid0.data(), n_layers * sizeof(int64_t), hipMemcpyHostToDevice), "copy");
    chk(hipMemcpy(c->d_code_off, code_off.data(), n_layers * sizeof(int64_t), hipMemcpyHostToDevice),
        "copy");
    chk(hipMemcpy(c->d_tile0, tile0.data(), n_layers * sizeof(int64_t), hipMemcpyHostToDevice),
        "copy");
    chk(hipMemcpy(c->d_tile_layer, tile_layer.data(), c->T * sizeof(int32_t), hipMemcpyHostToDevice),
        "copy");
    chk(hipMemcpy(c->d_tile_start, c->tile_start_host.data(), c->T * sizeof(int64_t),
                  hipMemcpyHostToDevice),
        "copy");
    const int32_t zero = 0;
    chk(hipMemcpy(c->d_err, &zero, sizeof(zero), hipMemcpyHostToDevice), "copy");
  }
  if (st != TERMEZO_OK) {
    free_all(c);
    delete c;
    return st;
  }
  *out = c;
  return TERMEZO_OK;
}

void termezo_destroy(termezo_ctx* ctx) {
  if (!ctx) return;
  (void)hipStreamSynchronize(ctx->stream);
  free_all(ctx);
  delete ctx;
}

const char* termezo_last_error(const termezo_ctx* ctx) {
  return ctx ? ctx->last_error.c_str() : "null context";
}

termezo_status termezo_sync(termezo_ctx* c) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  return sync_and_check(c);
}

termezo_status termezo_build_mask(termezo_ctx* c, float rho0, float delta, int32_t tie_inclusive,
                                  int64_t* k0_out, float* xi0_out) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  if (c->compact)
    return fail(c, TERMEZO_ERR_STATE, "build_mask needs the full latents (compact mode)");
  if (!finite(rho0) || !(rho0 > 0.0f) || rho0 > 1.0f)
    return fail(c, TERMEZO_ERR_INVALID_ARG, "rho0 must lie in (0, 1]");
  if (!finite(delta) || !(delta > 0.0f))
    return fail(c, TERMEZO_ERR_INVALID_ARG, "delta must be positive and finite");
  const int64_t k0 = (int64_t)std::floor((double)rho0 * (double)c->D);
  if (k0 <= 0) return fail(c, TERMEZO_ERR_STATE, "rho0 * D rounds down to an empty mask");

  c->has_mask = false;
  c->pair_valid = false;
  c->z_valid = false;
  c->codes_valid = false;
  c->pending_perturb = false;
  c->delta = delta;
  TMZ_HIP(c, launch_abs_sum(c, c->d_S_clean));
  TMZ_HIP(c, launch_thresholds(c, c->d_S_clean, c->d_tau, c->d_beta));
  termezo_status st = sync_and_check(c);
  if (st != TERMEZO_OK) return st;

  TMZ_HIP(c, launch_select(c, k0));
  // counts and offsets first: the inclusive reading may admit more than k0
  const int inclusive = tie_inclusive ? 1 : 0;
  TMZ_HIP(c, launch_mask_compact_counts(c, inclusive));
  int64_t total = 0;
  TMZ_HIP(c, hipMemcpyAsync(&total, c->d_act_off + c->L, sizeof(int64_t), hipMemcpyDeviceToHost,
                            c->stream));
  TMZ_HIP(c, hipStreamSynchronize(c->stream));
  st = ensure_active_capacity(c, total);
  if (st != TERMEZO_OK) return st;
  TMZ_HIP(c, launch_mask_compact_write(c, inclusive));
  TMZ_HIP(c, launch_tile_ranges(c));
  // sparse sets: keep the active latents in list order as well (contiguous reads in the
  // perturbation and the update instead of gathers; the update writes both copies)
  c->mirror = false;
  if (total > 0 && total * 8 <= c->D) {
    st = ensure_wc_capacity(c, total);
    if (st != TERMEZO_OK) return st;
    TMZ_HIP(c, launch_active_values(c, 0, total, c->d_wc, 0, 0));
    c->mirror = true;
  }

  // clean codes: current = clean
  TMZ_HIP(c, launch_copy_i64(c->d_S_cur, c->d_S_clean, c->L, c->stream));
  TMZ_HIP(c, launch_thresholds(c, c->d_S_cur, c->d_tau_cur, c->d_beta_cur));
  TMZ_HIP(c, launch_requant(c, 0));

  SelectState sel;
  TMZ_HIP(c, hipMemcpyAsync(&sel, c->d_sel, sizeof(sel), hipMemcpyDeviceToHost, c->stream));
  st = sync_and_check(c);
  if (st != TERMEZO_OK) return st;
  float xi0;
  std::memcpy(&xi0, &sel.prefix, sizeof(float));
  c->xi0 = xi0;
  // every inactive weight has fp32 distance >= xi0 to the clean threshold the codes were
  // just computed with, so an exact distance >= xi0 - ulp(xi0) / 2
  c->xi_lo = (double)xi0 - 0.5 * ((double)std::nextafter(xi0, INFINITY) - (double)xi0);
  TMZ_HIP(c, launch_ref_init(c, c->xi_lo));
  c->k0 = total;
  c->k_bound = total;
  c->tie_inclusive = inclusive;
  c->has_mask = true;
  c->codes_valid = true;
  if (k0_out) *k0_out = total;
  if (xi0_out) *xi0_out = xi0;
  return TERMEZO_OK;
}

termezo_status termezo_perturb(termezo_ctx* c, uint64_t seed, float eps, int32_t sign) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  if (sign < -1 || sign > 1) return fail(c, TERMEZO_ERR_INVALID_ARG, "sign must be -1, 0 or 1");
  if (!finite(eps) || !(eps > 0.0f)) return fail(c, TERMEZO_ERR_INVALID_ARG, "eps must be > 0");
  if (!c->has_mask) return fail(c, TERMEZO_ERR_STATE, "perturb before build_mask");
  const float se = (float)sign * eps;
  if (sign != 0 && c->pair_valid && c->pair_seed == seed && c->pair_eps == eps) {
    // the other sign of a pair: its values and sums came with the first call
    if (sign != c->pair_sign) {
      std::swap(c->d_wp, c->d_wpm);
      std::swap(c->d_S_cur, c->d_S_alt);
      c->pair_sign = sign;
    }
  } else {
    c->pair_valid = false;
    if (sign != 0) c->z_valid = false;          // the pair pass below rewrites the draws
    TMZ_HIP(c, launch_copy_i64(c->d_S_cur, c->d_S_clean, c->L, c->stream));
    if (sign != 0) TMZ_HIP(c, launch_copy_i64(c->d_S_alt, c->d_S_clean, c->L, c->stream));
    TMZ_HIP(c, launch_perturb_delta(c, c->k_bound, seed, se, sign != 0));
    if (sign != 0) {
      c->pair_valid = true;
      c->z_valid = true;
      c->z_seed = seed;
      c->pair_seed = seed;
      c->pair_eps = eps;
      c->pair_sign = sign;
    }
  }
  TMZ_HIP(c, launch_thresholds(c, c->d_S_cur, c->d_tau_cur, c->d_beta_cur));
  // guarded requantisation: the actives' codes only, while no frozen code can change
  // (every latent re-quantised on request)
  const int force = !c->compact && c->dense_requant;
  TMZ_HIP(c, launch_requant_guarded(c, force));
  // theta: both signs of the pair come from one pass, so the second evaluation
  // of a pair (same seed and eps) only switches to the other copy
  if (!c->theta.empty() && sign != 0 &&
      !(c->theta_pair_valid && c->theta_pair_seed == seed && c->theta_pair_eps == eps)) {
    c->theta_pair_valid = false;
    for (const ThetaHost& t : c->theta) TMZ_HIP(c, launch_theta_pair(c, t, seed, eps));
    c->theta_pair_valid = true;
    c->theta_pair_seed = seed;
    c->theta_pair_eps = eps;
  }
  c->theta_sign = sign;
  c->codes_valid = true;
  c->pending_perturb = true;
  c->last_seed = seed;
  c->last_eps = eps;
  return TERMEZO_OK;
}

namespace {
termezo_status check_forward_args(termezo_ctx* c, int32_t layer, const void* x,
                                  termezo_dtype x_dtype, int64_t M, const void* y,
                                  termezo_dtype y_dtype) {
  if (layer < 0 || layer >= c->L) return fail(c, TERMEZO_ERR_INVALID_ARG, "layer out of range");
  if (M <= 0 || !x || !y) return fail(c, TERMEZO_ERR_INVALID_ARG, "M <= 0 or null x / y");
  if ((x_dtype != TERMEZO_F32 && x_dtype != TERMEZO_BF16) ||
      (y_dtype != TERMEZO_F32 && y_dtype != TERMEZO_BF16))
    return fail(c, TERMEZO_ERR_INVALID_ARG, "x and y must be F32 or BF16");
  if ((reinterpret_cast<uintptr_t>(x) & 15u) != 0)
    return fail(c, TERMEZO_ERR_INVALID_ARG, "x must be 16-byte aligned");
  if (!c->codes_valid) return fail(c, TERMEZO_ERR_STATE, "no current codes (perturb first)");
  return TERMEZO_OK;
}
}  // namespace

termezo_status termezo_bitlinear_forward(termezo_ctx* c, int32_t layer, const void* x,
                                         termezo_dtype x_dtype, int64_t M, void* y,
                                         termezo_dtype y_dtype, int8_t* xq_out, float* xscale_out,
                                         int32_t* acc_out) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  if (xq_out && (reinterpret_cast<uintptr_t>(xq_out) & 15u) != 0)
    return fail(c, TERMEZO_ERR_INVALID_ARG, "xq_out must be 16-byte aligned");
  const termezo_status ck = check_forward_args(c, layer, x, x_dtype, M, y, y_dtype);
  if (ck != TERMEZO_OK) return ck;
  const LayerHost& L = c->layers[layer];
  if (!xq_out && !xscale_out && !acc_out && gemv1_fused_ok(M, L.d_in)) {
    TMZ_HIP(c, launch_gemv1_fused(x, x_dtype, c->d_codes + L.code_off, c->d_beta_cur + layer,
                                  L.d_in, L.d_out, y, y_dtype, c->stream));
    return TERMEZO_OK;
  }
  if (!xq_out && !xscale_out && !acc_out && gemv_fused_ok(M, L.d_in, x_dtype)) {
    TMZ_HIP(c, launch_gemv_fused(x, x_dtype, c->d_codes + L.code_off, c->d_beta_cur + layer, M,
                                 L.d_in, L.d_out, y, y_dtype, c->n_cu, c->stream));
    return TERMEZO_OK;
  }
  int8_t* xq = xq_out;
  float* xs = xscale_out;
  termezo_status st = ensure_xs_capacity(c, M);       // the row sums live here in any case
  if (st != TERMEZO_OK) return st;
  if (!xq) {
    st = ensure_xq_capacity(c, M, L.d_in);
    if (st != TERMEZO_OK) return st;
    xq = c->d_xq;
  }
  if (!xs) xs = c->d_xs;
  TMZ_HIP(c, launch_act_quant(x, x_dtype, M, L.d_in, xq, xs, c->d_xrs, c->stream));
  TMZ_HIP(c, launch_bitlinear_gemm(xq, xs, c->d_xrs, c->d_codes + L.code_off,
                                   c->d_beta_cur + layer, M, L.d_in, L.d_out, y, y_dtype, acc_out,
                                   c->n_cu, c->stream));
  return TERMEZO_OK;
}

termezo_status termezo_bitlinear_forward_noalloc(termezo_ctx* c, int32_t layer, const void* x,
                                                 termezo_dtype x_dtype, int64_t M, void* y,
                                                 termezo_dtype y_dtype) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  const termezo_status ck = check_forward_args(c, layer, x, x_dtype, M, y, y_dtype);
  if (ck != TERMEZO_OK) return ck;
  const LayerHost& L = c->layers[layer];
  if (gemv1_fused_ok(M, L.d_in)) {                    // one token: no scratch at all
    TMZ_HIP(c, launch_gemv1_fused(x, x_dtype, c->d_codes + L.code_off, c->d_beta_cur + layer,
                                  L.d_in, L.d_out, y, y_dtype, c->stream));
    return TERMEZO_OK;
  }
  if (gemv_fused_ok(M, L.d_in, x_dtype)) {             // up to 16 tokens: none either
    TMZ_HIP(c, launch_gemv_fused(x, x_dtype, c->d_codes + L.code_off, c->d_beta_cur + layer, M,
                                 L.d_in, L.d_out, y, y_dtype, c->n_cu, c->stream));
    return TERMEZO_OK;
  }
  // int8 activations, then the scales and the row sums, each at a 256-byte boundary
  const int64_t xq_bytes = M <= kNoAllocScratchBytes ? ((M * L.d_in + 255) / 256) * 256 : -1;
  const int64_t xs_bytes = ((4 * M + 255) / 256) * 256;
  if (xq_bytes < 0 || xq_bytes + xs_bytes + 4 * M > kNoAllocScratchBytes)
    return fail(c, TERMEZO_ERR_INVALID_ARG,
                "bitlinear_forward_noalloc: M * d_in + 8 M bytes (256-aligned parts) exceed the "
                "16 MiB scratch");
  if (!c->noalloc_scratch) return fail(c, TERMEZO_ERR_DEVICE, "no scratch address");
  char* base = static_cast<char*>(c->noalloc_scratch);
  int8_t* xq = reinterpret_cast<int8_t*>(base);
  float* xs = reinterpret_cast<float*>(base + xq_bytes);
  int32_t* xrs = reinterpret_cast<int32_t*>(base + xq_bytes + xs_bytes);
  TMZ_HIP(c, launch_act_quant(x, x_dtype, M, L.d_in, xq, xs, xrs, c->stream));
  TMZ_HIP(c, launch_bitlinear_gemm(xq, xs, xrs, c->d_codes + L.code_off, c->d_beta_cur + layer,
                                   M, L.d_in, L.d_out, y, y_dtype, nullptr, c->n_cu, c->stream));
  return TERMEZO_OK;
}

namespace {
SeedList one_seed(uint64_t s) {
  SeedList l = {};
  l.s[0] = s;
  l.K = 1;
  return l;
}
SeedList seed_list(const uint64_t* s, int32_t K) {
  SeedList l = {};
  for (int32_t q = 0; q < K; ++q) l.s[q] = s[q];
  l.K = K;
  return l;
}

// Update at the actives with the coefficients already in d_scal, then the new
// thresholds and the shrink; the compacted list replaces the old one.
termezo_status finish_update(termezo_ctx* c, const SeedList& seeds, int64_t* k_out) {
  TMZ_HIP(c, launch_update(c, c->k_bound, seeds));
  c->pair_valid = false;
  c->z_valid = false;                          // the shrink below changes the list
  c->theta_pair_valid = false;
  c->theta_sign = 0;
  for (const ThetaHost& t : c->theta) TMZ_HIP(c, launch_theta_update(c, t, seeds));
  TMZ_HIP(c, launch_thresholds(c, c->d_S_clean, c->d_tau, c->d_beta));
  TMZ_HIP(c, launch_shrink(c, c->k_bound));
  std::swap(c->d_act, c->d_act_tmp);
  std::swap(c->d_act_off, c->d_act_off_tmp);
  if (c->mirror) std::swap(c->d_wc, c->d_wc_tmp);
  TMZ_HIP(c, launch_tile_ranges(c));
  TMZ_HIP(c, launch_ref_after_update(c, c->xi_lo));
  c->codes_valid = false;
  c->pending_perturb = false;
  if (k_out) {
    int64_t k = 0;
    TMZ_HIP(c, hipMemcpyAsync(&k, c->d_act_off + c->L, sizeof(int64_t), hipMemcpyDeviceToHost,
                              c->stream));
    termezo_status st = sync_and_check(c);
    if (st != TERMEZO_OK) return st;
    c->k_bound = k;
    *k_out = k;
  }
  return TERMEZO_OK;
}
}  // namespace

termezo_status termezo_update(termezo_ctx* c, float proj_grad, float lr, int64_t* k_out) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  if (!finite(proj_grad) || !finite(lr))
    return fail(c, TERMEZO_ERR_INVALID_ARG, "projected gradient and lr must be finite");
  if (!c->pending_perturb) return fail(c, TERMEZO_ERR_STATE, "update without a perturbation");
  const float a = -(lr * proj_grad);
  TMZ_HIP(c, launch_set_coeff(c, a));
  return finish_update(c, one_seed(c->last_seed), k_out);
}

termezo_status termezo_update_from_losses(termezo_ctx* c, const float* loss_plus,
                                          const float* loss_minus, float eps, float lr) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  if (!loss_plus || !loss_minus) return fail(c, TERMEZO_ERR_INVALID_ARG, "null loss pointer");
  if (!finite(eps) || !(eps > 0.0f) || !finite(lr))
    return fail(c, TERMEZO_ERR_INVALID_ARG, "eps must be > 0 and lr finite");
  if (!c->pending_perturb) return fail(c, TERMEZO_ERR_STATE, "update without a perturbation");
  TMZ_HIP(c, launch_coeff_from_losses(c, loss_plus, loss_minus, eps, lr));
  return finish_update(c, one_seed(c->last_seed), nullptr);
}

termezo_status termezo_update_multi(termezo_ctx* c, const uint64_t* seeds, const float* proj_grads,
                                    int32_t K, float lr, int64_t* k_out) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  if (!seeds || !proj_grads || K < 1 || K > kMaxK)
    return fail(c, TERMEZO_ERR_INVALID_ARG, "null seeds / gradients or K outside [1, 32]");
  if (!finite(lr)) return fail(c, TERMEZO_ERR_INVALID_ARG, "lr must be finite");
  for (int32_t q = 0; q < K; ++q)
    if (!finite(proj_grads[q]))
      return fail(c, TERMEZO_ERR_INVALID_ARG, "projected gradients must be finite");
  if (!c->pending_perturb) return fail(c, TERMEZO_ERR_STATE, "update without a perturbation");
  float a[kMaxK];
  const float cK = lr / (float)K;
  for (int32_t q = 0; q < K; ++q) a[q] = -(cK * proj_grads[q]);
  TMZ_HIP(c, launch_set_coeffs(c, a, K));
  return finish_update(c, seed_list(seeds, K), k_out);
}

termezo_status termezo_update_multi_from_losses(termezo_ctx* c, const uint64_t* seeds,
                                                const float* losses, int32_t K, float eps,
                                                float lr) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  if (!seeds || !losses || K < 1 || K > kMaxK)
    return fail(c, TERMEZO_ERR_INVALID_ARG, "null seeds / losses or K outside [1, 32]");
  if (!finite(eps) || !(eps > 0.0f) || !finite(lr))
    return fail(c, TERMEZO_ERR_INVALID_ARG, "eps must be > 0 and lr finite");
  if (!c->pending_perturb) return fail(c, TERMEZO_ERR_STATE, "update without a perturbation");
  TMZ_HIP(c, launch_coeffs_multi_from_losses(c, losses, K, eps, lr));
  return finish_update(c, seed_list(seeds, K), nullptr);
}

// Evolution strategies on the mask: the coefficients a_n = (lr / N) Rt_n (Rt: the
// population z-score of the rewards in fp64, index order, or the raw rewards),
// then the K-direction update with the N seeds.
termezo_status termezo_es_update(termezo_ctx* c, const uint64_t* seeds, const float* rewards,
                                 int32_t N, float lr, int32_t standardize, int64_t* k_out) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  if (!seeds || !rewards || N < 1 || N > kMaxK)
    return fail(c, TERMEZO_ERR_INVALID_ARG, "null seeds / rewards or N outside [1, 32]");
  if (!finite(lr)) return fail(c, TERMEZO_ERR_INVALID_ARG, "lr must be finite");
  for (int32_t n = 0; n < N; ++n)
    if (!finite(rewards[n])) return fail(c, TERMEZO_ERR_INVALID_ARG, "rewards must be finite");
  if (!c->pending_perturb) return fail(c, TERMEZO_ERR_STATE, "update without a perturbation");
  float rt[kMaxK];
  for (int32_t n = 0; n < N; ++n) rt[n] = rewards[n];
  if (standardize) {
    double mu = 0.0, var = 0.0;
    for (int32_t n = 0; n < N; ++n) mu += (double)rewards[n];
    mu /= (double)N;
    for (int32_t n = 0; n < N; ++n) {
      const double d = (double)rewards[n] - mu;
      var += d * d;
    }
    var /= (double)N;
    const double sd = std::sqrt(var);
    for (int32_t n = 0; n < N; ++n)
      rt[n] = sd > 0.0 ? (float)(((double)rewards[n] - mu) / sd) : 0.0f;
  }
  const float cN = lr / (float)N;
  float a[kMaxK];
  for (int32_t n = 0; n < N; ++n) {
    a[n] = cN * rt[n];
    if (!finite(a[n])) return fail(c, TERMEZO_ERR_INVALID_ARG, "ES coefficient is not finite");
  }
  TMZ_HIP(c, launch_set_coeffs(c, a, N));
  return finish_update(c, seed_list(seeds, N), k_out);
}

termezo_status termezo_es_update_from_rewards(termezo_ctx* c, const uint64_t* seeds,
                                              const float* rewards, int32_t N, float lr,
                                              int32_t standardize) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  if (!seeds || !rewards || N < 1 || N > kMaxK)
    return fail(c, TERMEZO_ERR_INVALID_ARG, "null seeds / rewards or N outside [1, 32]");
  if (!finite(lr)) return fail(c, TERMEZO_ERR_INVALID_ARG, "lr must be finite");
  if (!c->pending_perturb) return fail(c, TERMEZO_ERR_STATE, "update without a perturbation");
  TMZ_HIP(c, launch_es_coeffs(c, rewards, N, lr, standardize ? 1 : 0));
  return finish_update(c, seed_list(seeds, N), nullptr);
}

termezo_status termezo_compact(termezo_ctx* c) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  if (!c->has_mask) return fail(c, TERMEZO_ERR_STATE, "compact before build_mask");
  if (c->compact) return fail(c, TERMEZO_ERR_STATE, "already compact");
  if (c->pending_perturb) return fail(c, TERMEZO_ERR_STATE, "compact with a pending perturbation");
  int64_t k = 0;
  TMZ_HIP(c, hipMemcpyAsync(&k, c->d_act_off + c->L, sizeof(int64_t), hipMemcpyDeviceToHost,
                            c->stream));
  TMZ_HIP(c, hipStreamSynchronize(c->stream));
  if (!c->mirror) {                              // dense sets: the copy is made now
    termezo_status st = ensure_wc_capacity(c, k);
    if (st != TERMEZO_OK) return st;
    TMZ_HIP(c, launch_active_values(c, 0, k, c->d_wc, 0, 0));
  }
  termezo_status st = sync_and_check(c);
  if (st != TERMEZO_OK) return st;
  c->mirror = true;
  c->compact = true;
  c->pair_valid = false;
  c->z_valid = false;
  c->k_bound = k;
  return TERMEZO_OK;
}

termezo_status termezo_active_values(termezo_ctx* c, int32_t layer, float* values, int64_t cap,
                                     int64_t* n) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  if (layer < 0 || layer >= c->L || !n) return fail(c, TERMEZO_ERR_INVALID_ARG, "bad layer or n");
  if (!c->has_mask) return fail(c, TERMEZO_ERR_STATE, "no mask");
  int64_t off[2];
  TMZ_HIP(c, hipMemcpyAsync(off, c->d_act_off + layer, 2 * sizeof(int64_t), hipMemcpyDeviceToHost,
                            c->stream));
  TMZ_HIP(c, hipStreamSynchronize(c->stream));
  const int64_t cnt = off[1] - off[0];
  *n = cnt;
  if (cnt == 0) return TERMEZO_OK;
  if (!values || cap < cnt) return fail(c, TERMEZO_ERR_INVALID_ARG, "capacity below the count");
  float* tmp = nullptr;
  TMZ_HIP(c, hipMalloc(&tmp, (size_t)cnt * sizeof(float)));
  hipError_t e = launch_active_values(c, off[0], off[1], tmp, 1, c->compact ? 1 : 0);
  if (e == hipSuccess)
    e = hipMemcpyAsync(values, tmp, (size_t)cnt * sizeof(float), hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  (void)hipFree(tmp);
  if (e != hipSuccess) return hip_fail(c, e, "active values");
  return TERMEZO_OK;
}

termezo_status termezo_memory_footprint(termezo_ctx* c, int64_t* library_bytes,
                                        int64_t* latent_bytes) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  const int64_t L = c->L, T = c->T, cap = c->act_cap;
  const int64_t dsz = (int64_t)dtype_size(c->dtype);
  int64_t b = c->D / 4;                                          // 2-bit codes
  b += L * (8 * 8 + 4 * 4 + 4 + 8 + 4 + 8) + 3 * (L + 1) * 8;    // per-layer state, offsets
  b += T * (4 + 8 + 8 + 8 + 8 + 8) + 8;                          // tile tables and scratch
  b += cap * (4 + 4 + 4 + 4 + 4) + c->blk_cap * 8 + c->flag_cap * 8;  // lists, w' of both
                                                                    // signs, z, shrink
  b += L * 8;                                                    // |w| sums of the other sign
  if (c->mirror) b += 2 * c->wc_cap * dsz;                       // active latents (list order)
  b += (int64_t)kHistBins * 8 + (int64_t)sizeof(SelectState) + 4 * 8 + kScalLen * 4 + 4;
  b += c->xq_cap + c->xs_cap * 8;                                // activation-quant scratch
  for (const ThetaHost& t : c->theta) b += 2 * t.n * (int64_t)dtype_size(t.dtype);
  if (c->d_codes_snap) b += c->code_words * 4 + L * 4;               // codes snapshot
  if (library_bytes) *library_bytes = b;
  if (latent_bytes) *latent_bytes = c->compact ? 0 : c->D * dsz;
  return TERMEZO_OK;
}

termezo_status termezo_set_dense_requant(termezo_ctx* c, int32_t always_dense) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  c->dense_requant = always_dense ? 1 : 0;
  return TERMEZO_OK;
}

termezo_status termezo_theta_register(termezo_ctx* c, const termezo_theta* params, int32_t n) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  if (!params || n <= 0) return fail(c, TERMEZO_ERR_INVALID_ARG, "no theta tensors");
  if (!c->theta.empty()) return fail(c, TERMEZO_ERR_STATE, "theta is already registered");
  for (int32_t i = 0; i < n; ++i) {
    const termezo_theta& p = params[i];
    if (!p.data || p.n <= 0 || (p.dtype != TERMEZO_F32 && p.dtype != TERMEZO_BF16))
      return fail(c, TERMEZO_ERR_INVALID_ARG, "theta tensor: null data, n <= 0 or bad dtype");
    if ((reinterpret_cast<uintptr_t>(p.data) & 15u) != 0)
      return fail(c, TERMEZO_ERR_INVALID_ARG, "theta tensors must be 16-byte aligned");
  }
  std::vector<ThetaHost> th;
  int64_t tid = 0;
  for (int32_t i = 0; i < n; ++i) {
    ThetaHost t;
    t.data = params[i].data;
    t.n = params[i].n;
    t.dtype = params[i].dtype;
    t.tid0 = tid;
    t.plus = t.minus = nullptr;
    const size_t bytes = (size_t)t.n * dtype_size(t.dtype);
    hipError_t e = hipMalloc(&t.plus, bytes);
    if (e == hipSuccess) e = hipMalloc(&t.minus, bytes);
    if (e != hipSuccess) {
      if (t.plus) (void)hipFree(t.plus);
      for (ThetaHost& u : th) {
        (void)hipFree(u.plus);
        (void)hipFree(u.minus);
      }
      return hip_fail(c, e, "alloc theta copies");
    }
    th.push_back(t);
    tid += t.n;
  }
  c->theta = std::move(th);
  c->theta_P = tid;
  c->theta_sign = 0;
  c->theta_pair_valid = false;
  return TERMEZO_OK;
}

termezo_status termezo_theta_current(termezo_ctx* c, int32_t i, void** values) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  if (!values || i < 0 || i >= (int32_t)c->theta.size())
    return fail(c, TERMEZO_ERR_INVALID_ARG, "theta index out of range or null output");
  const ThetaHost& t = c->theta[i];
  *values = c->theta_sign == 0 ? t.data : (c->theta_sign > 0 ? t.plus : t.minus);
  return TERMEZO_OK;
}

termezo_status termezo_theta_copy(termezo_ctx* c, int32_t i, void* dst) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  void* src = nullptr;
  termezo_status st = termezo_theta_current(c, i, &src);
  if (st != TERMEZO_OK) return st;
  if (!dst) return fail(c, TERMEZO_ERR_INVALID_ARG, "null destination");
  const ThetaHost& t = c->theta[i];
  TMZ_HIP(c, hipMemcpyAsync(dst, src, (size_t)t.n * dtype_size(t.dtype), hipMemcpyDeviceToDevice,
                            c->stream));
  return TERMEZO_OK;
}

termezo_status termezo_gauss(void* hip_stream, uint64_t seed, const uint64_t* gids, int64_t n,
                             float* z) {
  if (n < 0 || (n > 0 && (!gids || !z))) return TERMEZO_ERR_INVALID_ARG;
  if (n == 0) return TERMEZO_OK;
  return launch_gauss(seed, gids, n, z, static_cast<hipStream_t>(hip_stream)) == hipSuccess
             ? TERMEZO_OK
             : TERMEZO_ERR_DEVICE;
}

termezo_status termezo_active_count(termezo_ctx* c, int64_t* k) {
  if (!c || !k) return TERMEZO_ERR_INVALID_ARG;
  if (!c->has_mask) return fail(c, TERMEZO_ERR_STATE, "no mask");
  int64_t v = 0;
  TMZ_HIP(c, hipMemcpyAsync(&v, c->d_act_off + c->L, sizeof(int64_t), hipMemcpyDeviceToHost,
                            c->stream));
  termezo_status st = sync_and_check(c);
  if (st != TERMEZO_OK) return st;
  c->k_bound = v;
  *k = v;
  return TERMEZO_OK;
}

termezo_status termezo_mask_export(termezo_ctx* c, int32_t layer, uint32_t* idx, int64_t cap,
                                   int64_t* n) {
  if (!c || !n) return TERMEZO_ERR_INVALID_ARG;
  if (layer < 0 || layer >= c->L) return fail(c, TERMEZO_ERR_INVALID_ARG, "layer out of range");
  if (!c->has_mask) return fail(c, TERMEZO_ERR_STATE, "no mask");
  std::vector<int64_t> off(c->L + 1);
  TMZ_HIP(c, hipMemcpyAsync(off.data(), c->d_act_off, (c->L + 1) * sizeof(int64_t),
                            hipMemcpyDeviceToHost, c->stream));
  termezo_status st = sync_and_check(c);
  if (st != TERMEZO_OK) return st;
  const int64_t cnt = off[layer + 1] - off[layer];
  *n = cnt;
  if (cnt > cap || (cnt > 0 && !idx))
    return fail(c, TERMEZO_ERR_INVALID_ARG, "index buffer too small");
  if (cnt > 0)
    TMZ_HIP(c, hipMemcpy(idx, c->d_act + off[layer], cnt * sizeof(uint32_t), hipMemcpyDeviceToHost));
  return TERMEZO_OK;
}

termezo_status termezo_codes_export(termezo_ctx* c, int32_t layer, int8_t* codes) {
  if (!c || !codes) return TERMEZO_ERR_INVALID_ARG;
  if (layer < 0 || layer >= c->L) return fail(c, TERMEZO_ERR_INVALID_ARG, "layer out of range");
  if (!c->codes_valid) return fail(c, TERMEZO_ERR_STATE, "no current codes");
  const LayerHost& L = c->layers[layer];
  int8_t* tmp = nullptr;
  TMZ_HIP(c, dalloc(&tmp, (size_t)L.n));
  hipError_t e = launch_unpack_layer(c, layer, tmp);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  if (e == hipSuccess) e = hipMemcpy(codes, tmp, (size_t)L.n, hipMemcpyDeviceToHost);
  (void)hipFree(tmp);
  if (e != hipSuccess) return hip_fail(c, e, "codes export");
  return sync_and_check(c);
}

termezo_status termezo_codes_snapshot(termezo_ctx* c) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  if (!c->codes_valid) return fail(c, TERMEZO_ERR_STATE, "codes_snapshot: no current codes");
  if (!c->d_codes_snap) {
    TMZ_HIP(c, dalloc(&c->d_codes_snap, (size_t)c->code_words));
    if (dalloc(&c->d_beta_snap, (size_t)c->L) != hipSuccess) {
      dfree(c->d_codes_snap);
      return fail(c, TERMEZO_ERR_OOM, "codes_snapshot: allocation");
    }
  }
  TMZ_HIP(c, hipMemcpyAsync(c->d_codes_snap, c->d_codes, (size_t)c->code_words * 4,
                            hipMemcpyDeviceToDevice, c->stream));
  TMZ_HIP(c, hipMemcpyAsync(c->d_beta_snap, c->d_beta_cur, (size_t)c->L * 4,
                            hipMemcpyDeviceToDevice, c->stream));
  c->snap_valid = true;
  return TERMEZO_OK;
}

termezo_status termezo_layer_stats(termezo_ctx* c, int32_t layer, float* tau, float* beta,
                                   int64_t* abs_sum_fix, float* tau_cur, float* beta_cur) {
  if (!c) return TERMEZO_ERR_INVALID_ARG;
  if (layer < 0 || layer >= c->L) return fail(c, TERMEZO_ERR_INVALID_ARG, "layer out of range");
  TMZ_HIP(c, hipStreamSynchronize(c->stream));
  if (tau) TMZ_HIP(c, hipMemcpy(tau, c->d_tau + layer, 4, hipMemcpyDeviceToHost));
  if (beta) TMZ_HIP(c, hipMemcpy(beta, c->d_beta + layer, 4, hipMemcpyDeviceToHost));
  if (abs_sum_fix) TMZ_HIP(c, hipMemcpy(abs_sum_fix, c->d_S_clean + layer, 8, hipMemcpyDeviceToHost));
  if (tau_cur) TMZ_HIP(c, hipMemcpy(tau_cur, c->d_tau_cur + layer, 4, hipMemcpyDeviceToHost));
  if (beta_cur) TMZ_HIP(c, hipMemcpy(beta_cur, c->d_beta_cur + layer, 4, hipMemcpyDeviceToHost));
  return TERMEZO_OK;
}

termezo_status termezo_mse_loss(termezo_ctx* c, const float* y, const float* target, int64_t n,
                                float* out) {
  if (!c || !y || !target || !out || n <= 0) return TERMEZO_ERR_INVALID_ARG;
  TMZ_HIP(c, launch_mse(y, target, n, c->d_loss, nullptr, c->stream));
  double sum = 0.0;
  TMZ_HIP(c, hipMemcpyAsync(&sum, c->d_loss, sizeof(double), hipMemcpyDeviceToHost, c->stream));
  termezo_status st = sync_and_check(c);
  if (st != TERMEZO_OK) return st;
  *out = (float)(sum / (double)n);
  return TERMEZO_OK;
}

termezo_status termezo_mse_loss_dev(termezo_ctx* c, const float* y, const float* target,
                                    int64_t n, float* loss_dev) {
  if (!c || !y || !target || !loss_dev || n <= 0) return TERMEZO_ERR_INVALID_ARG;
  TMZ_HIP(c, launch_mse(y, target, n, c->d_loss, loss_dev, c->stream));
  return TERMEZO_OK;
}

}  // extern "C"
