// Host-side internals shared by the TerMeZO library sources.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/termezo.h"

namespace tmz {

constexpr int kTile = 8192;          // elements per streaming tile (never straddles layers)
constexpr int kBlock = 256;          // threads per block for streaming kernels
constexpr int kHistBins = 2048;      // radix-select histogram width (11 bits)
constexpr int kMaxLayers = 2048;     // layers per context (active-list offsets fit in LDS)

struct LayerHost {
  void* w;
  int64_t d_out, d_in, n, gid0;
  int64_t code_off;                  // offset of the layer's packed codes, in 32-bit words
  int64_t tile0, ntiles;             // tile range of the layer
};

// Device-side view of the registered layers and the per-layer state.
struct DevState {
  const void* const* w;              // [L] latent pointers
  const int64_t* n;                  // [L]
  const int64_t* gid0;               // [L]
  const int64_t* code_off;           // [L]
  const int32_t* tile_layer;         // [T]
  const int64_t* tile_start;         // [T] layer-local start element
  const int64_t* tile0;              // [L] first tile of each layer
  int64_t* tile_act;                 // [T+1] first active-list position at or after tile t
  uint32_t* codes;                   // packed codes, all layers
  int64_t* S_clean;                  // [L] fixed-point sum of |w|
  int64_t* S_cur;                    // [L] fixed-point sum of |w'| of the current codes
  float* tau;                        // [L] clean threshold
  float* beta;                       // [L]
  float* tau_cur;                    // [L] threshold of the current codes
  float* beta_cur;                   // [L]
  float* tau_ref;                    // [L] threshold the frozen codes were computed with
  double* mref;                      // [L] lower bound of the frozen weights' distance to tau_ref
  int32_t* need;                     // [L] 1: the layer needs the dense requantisation now
  int32_t* err;                      // deferred numeric error flag
  int32_t L;
  int64_t T;                         // number of tiles
};

// Output description of a BitLinear GEMM whose N columns may be split in up
// to kMaxSeg segments (fused projections sharing one input), each with its
// own scale beta', destination and row stride.
constexpr int kMaxSeg = 3;
constexpr int kGemmStore = 0;      // y = round(acc * beta / s)
constexpr int kGemmResidual = 1;   // y <- round(y + round(acc * beta / s))
// SwiGLU of a gate|up pair: N = 2F code rows (gate rows 0..F-1, up rows F..2F-1), output
// y[m][f] = round(silu(g) u) with g, u the rounded gate and up projections (bf16 only)
constexpr int kGemmSwiGLU = 2;
struct GemmOut {
  void* y[kMaxSeg];
  int64_t ld[kMaxSeg];
  const float* beta[kMaxSeg];
  int64_t nstart[kMaxSeg + 1];
  int nseg;
};

// Perturbation directions applied by one update (Algorithm 1: K per step),
// passed to the update kernels by value; their coefficients a_k live on the
// device (d_scal[0 .. K-1]).
constexpr int kMaxK = 32;
struct SeedList {
  uint64_t s[kMaxK];
  int32_t K;
};
// d_scal layout: coefficients a_k at [0, kMaxK), the last single-direction g at kMaxK
constexpr int kScalG = kMaxK;
constexpr int kScalLen = kMaxK + 2;

// One registered full-precision parameter tensor (theta).
struct ThetaHost {
  void* data;                        // caller's tensor (clean values, updated in place)
  int64_t n;                         // elements
  int64_t tid0;                      // first theta id (Philox stream 1)
  termezo_dtype dtype;               // F32 or BF16
  void* plus;                        // library copies theta +- eps z (same dtype and size)
  void* minus;
};

struct SelectState {                 // radix-select bookkeeping (device)
  unsigned long long k0;             // budget
  unsigned long long less;           // keys strictly below the current prefix bucket
  uint32_t prefix;                   // key bits fixed so far
  uint32_t pad;
};

}  // namespace tmz

struct termezo_ctx {
  int device = 0;
  hipStream_t stream = nullptr;
  termezo_dtype dtype = TERMEZO_F32;
  int32_t L = 0;
  int64_t D = 0;
  std::vector<tmz::LayerHost> layers;
  std::vector<int64_t> tile_start_host;
  int64_t T = 0;

  // device buffers
  void** d_wptr = nullptr;
  int64_t* d_n = nullptr;
  int64_t* d_gid0 = nullptr;
  int64_t* d_code_off = nullptr;
  int32_t* d_tile_layer = nullptr;
  int64_t* d_tile_start = nullptr;
  int64_t* d_tile0 = nullptr;
  int64_t* d_tile_act = nullptr;             // T + 1
  uint32_t* d_codes = nullptr;
  int64_t code_words = 0;            // 32-bit code words of all layers
  // copy of the codes and output scales of one perturbation (termezo_codes_snapshot), for a
  // forward that runs while the next perturbation rewrites the current codes
  uint32_t* d_codes_snap = nullptr;
  float* d_beta_snap = nullptr;
  bool snap_valid = false;
  int64_t* d_S_clean = nullptr;
  int64_t* d_S_cur = nullptr;
  float* d_tau = nullptr;
  float* d_beta = nullptr;
  float* d_tau_cur = nullptr;
  float* d_beta_cur = nullptr;
  float* d_tau_ref = nullptr;
  double* d_mref = nullptr;
  int32_t* d_need = nullptr;
  int64_t* d_dense_off = nullptr;    // [L+1] tiles of the layers needing the dense pass
  int32_t* d_err = nullptr;
  int dense_requant = 0;             // 1: every perturbation re-quantises every latent
  double xi_lo = 0.0;                // lower bound of the frozen weights' exact distance at build

  // mask
  uint32_t* d_act = nullptr;         // active local indices, ascending, layer after layer
  uint32_t* d_act_tmp = nullptr;     // compaction target
  int64_t act_cap = 0;
  int64_t* d_act_off = nullptr;      // [L+1]
  int64_t* d_act_off_tmp = nullptr;  // [L+1]
  std::vector<int64_t> h_act_off;    // host copy, valid when act_off_host_valid
  bool act_off_host_valid = false;
  float* d_wp = nullptr;             // perturbed values at the actives (act_cap)
  // perturbation pair: the first call of a (seed, eps) pair also writes the other sign's
  // values (d_wpm, its |w| sums in d_S_alt), in list order
  float* d_wpm = nullptr;
  int64_t* d_S_alt = nullptr;        // [L]
  bool pair_valid = false;
  uint64_t pair_seed = 0;
  float pair_eps = 0.f;
  int pair_sign = 0;                 // sign whose values d_wp / d_S_cur hold
  // the draws z of the last pair pass, list order: valid for z_seed until the active list
  // changes; a single-direction update of that seed reads them instead of drawing again
  float* d_zs = nullptr;
  bool z_valid = false;
  uint64_t z_seed = 0;
  // compact mode: the active latents in list order (latent dtype), library-owned; the
  // caller's latent tensors are no longer read or written
  bool compact = false;
  // mirror: d_wc holds the active latents in list order and is kept current (always in
  // compact mode; otherwise for sparse sets, where it replaces the scattered reads of the
  // latents; the update then writes both)
  bool mirror = false;
  void* d_wc = nullptr;
  void* d_wc_tmp = nullptr;
  int64_t wc_cap = 0;

  // scratch
  unsigned long long* d_hist = nullptr;      // kHistBins
  tmz::SelectState* d_sel = nullptr;
  uint32_t* d_tile_cnt = nullptr;            // 2 * T  (less, equal) per tile
  int64_t* d_tile_out = nullptr;             // T      output offset per tile
  int64_t* d_tile_eqb = nullptr;             // T      equal keys before the tile
  int64_t* d_blk_cnt = nullptr;              // shrink block counts
  int64_t blk_cap = 0;
  uint64_t* d_shrink_flags = nullptr;        // shrink keep flags, one word per thread
  int64_t flag_cap = 0;
  double* d_loss = nullptr;                  // loss accumulators
  float* d_scal = nullptr;                   // [0] update coefficient a, [1] g
  int n_cu = 0;                              // compute units of the device
  void* noalloc_scratch = nullptr;           // this device's address of the file-scope scratch
  int8_t* d_xq = nullptr;                    // activation-quantisation scratch
  int64_t xq_cap = 0;
  float* d_xs = nullptr;                     // per-token scales
  int32_t* d_xrs = nullptr;                  // per-token sums of the int8 activations
  int64_t xs_cap = 0;                        // tokens d_xs and d_xrs hold

  // full-precision parameters theta (dense perturbation and update)
  std::vector<tmz::ThetaHost> theta;
  int64_t theta_P = 0;               // total theta elements
  int theta_sign = 0;                // which values the forward reads: 0 clean, +1 / -1 copies
  bool theta_pair_valid = false;     // copies hold theta +- eps z(seed) for the recorded pair
  uint64_t theta_pair_seed = 0;
  float theta_pair_eps = 0.f;

  // state
  bool has_mask = false;
  bool codes_valid = false;
  bool pending_perturb = false;
  uint64_t last_seed = 0;
  float last_eps = 0.f;
  float delta = 1e-5f;
  float xi0 = 0.f;
  int64_t k0 = 0;
  int64_t k_bound = 0;               // upper bound of the active count (exact after a sync)
  int tie_inclusive = 0;

  std::string last_error;

  tmz::DevState dev() const {
    tmz::DevState s;
    s.w = (const void* const*)d_wptr;
    s.n = d_n;
    s.gid0 = d_gid0;
    s.code_off = d_code_off;
    s.tile_layer = d_tile_layer;
    s.tile_start = d_tile_start;
    s.tile0 = d_tile0;
    s.tile_act = d_tile_act;
    s.codes = d_codes;
    s.S_clean = d_S_clean;
    s.S_cur = d_S_cur;
    s.tau = d_tau;
    s.beta = d_beta;
    s.tau_cur = d_tau_cur;
    s.beta_cur = d_beta_cur;
    s.tau_ref = d_tau_ref;
    s.mref = d_mref;
    s.need = d_need;
    s.err = d_err;
    s.L = L;
    s.T = T;
    return s;
  }
};

namespace tmz {

// Launchers (stream-ordered, no synchronisation).  Return hipSuccess or the
// launch error.
hipError_t launch_abs_sum(termezo_ctx* c, int64_t* S_out);
hipError_t launch_thresholds(termezo_ctx* c, const int64_t* S, float* tau, float* beta);
hipError_t launch_fill_u64(unsigned long long* p, int64_t n, unsigned long long v, hipStream_t s);
hipError_t launch_copy_i64(int64_t* dst, const int64_t* src, int64_t n, hipStream_t s);
hipError_t launch_select(termezo_ctx* c, int64_t k0);     // three radix passes -> d_sel
hipError_t launch_mask_compact_counts(termezo_ctx* c, int inclusive);  // -> act_off
hipError_t launch_mask_compact_write(termezo_ctx* c, int inclusive);   // -> act
hipError_t launch_tile_ranges(termezo_ctx* c);            // d_act, d_act_off -> d_tile_act
// codes of w with tau_cur; with patch, the actives' codes from their perturbed values d_wp
hipError_t launch_requant(termezo_ctx* c, int patch);
// Guarded requantisation of a perturbation: layers whose threshold moved less than
// the frozen weights' distance keep their frozen codes and get only the actives'
// codes (sparse); the others are re-quantised densely.
hipError_t launch_requant_guarded(termezo_ctx* c, int force);
// after a dense requantisation of every layer at tau_cur (mask build): frozen codes refer
// to tau_cur; every frozen weight is at least xi_lo from it
hipError_t launch_ref_init(termezo_ctx* c, double xi_lo);
// after an update: weights leaving the set are frozen at tau_ref (their distance to the new
// clean threshold exceeds xi0, so to tau_ref at least xi_lo - |tau - tau_ref|)
hipError_t launch_ref_after_update(termezo_ctx* c, double xi_lo);
hipError_t launch_perturb_delta(termezo_ctx* c, int64_t k, uint64_t seed, float se, bool pair);
hipError_t launch_set_coeff(termezo_ctx* c, float a);
// K host coefficients to d_scal[0 .. K-1]
hipError_t launch_set_coeffs(termezo_ctx* c, const float* a, int K);
hipError_t launch_coeff_from_losses(termezo_ctx* c, const float* fp, const float* fm, float eps,
                                    float lr);
// a_k = -((lr / K) g_k), g_k = (F+_k - F-_k) / (2 eps) from device losses [2K] (F+_k, F-_k pairs)
hipError_t launch_es_coeffs(termezo_ctx* c, const float* rewards, int N, float lr,
                            int standardize);
hipError_t launch_coeffs_multi_from_losses(termezo_ctx* c, const float* losses, int K, float eps,
                                           float lr);
// coefficients from d_scal[0 .. K-1]; the updated values of the actives go to d_wp (list order)
hipError_t launch_update(termezo_ctx* c, int64_t k, const SeedList& seeds);
// from d_wp (the updated values): d_act -> d_act_tmp, offsets -> tmp
hipError_t launch_shrink(termezo_ctx* c, int64_t k);
hipError_t launch_unpack_layer(termezo_ctx* c, int layer, int8_t* out_dev);
// list entries [j0, j1): latent values (compact array when from_compact, else the layers)
hipError_t launch_active_values(termezo_ctx* c, int64_t j0, int64_t j1, void* out, int to_f32,
                                int from_compact);
// theta: both perturbed copies in one pass; in-place update with the coefficient in d_scal[0]
hipError_t launch_theta_pair(termezo_ctx* c, const ThetaHost& t, uint64_t seed, float eps);
hipError_t launch_theta_update(termezo_ctx* c, const ThetaHost& t, const SeedList& seeds);
hipError_t launch_gauss(uint64_t seed, const uint64_t* gids, int64_t n, float* z, hipStream_t s);
hipError_t launch_mse(const float* y, const float* t, int64_t n, double* acc, float* mean32,
                      hipStream_t s);

// BitLinear.  The quantisers write per token the scale s and the sum of the int8
// activations rs; the GEMM reads both (rs, 16-byte aligned, for its offset weight
// encoding; the full-tile paths reject a null or misaligned rs).
hipError_t launch_act_quant(const void* x, termezo_dtype xdt, int64_t M, int64_t K, int8_t* xq,
                            float* s, int32_t* rs, hipStream_t st);
// Optional timing of one GEMM launch: non-null events take the start and the end of the
// kernel's own execution (hipExtLaunchKernel), not the time around the launch.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
hipError_t launch_gemm_i8(const int8_t* xq, const float* s, const int32_t* rs,
                          const uint32_t* codes, int64_t M, int64_t K, int64_t N,
                          const GemmOut& out, termezo_dtype ydt, int mode, int32_t* acc, int n_cu,
                          hipStream_t st, LaunchEvents ev = LaunchEvents());
// One token with the activation quantisation fused in (no x_q, scale or row-sum
// buffers): gemv1_fused_ok(M, K) tells whether it applies.
bool gemv1_fused_ok(int64_t M, int64_t K);
hipError_t launch_gemv1_fused(const void* x, termezo_dtype xdt, const uint32_t* codes,
                              const float* beta_dev, int64_t K, int64_t N, void* y,
                              termezo_dtype ydt, hipStream_t st);
// Two to sixteen tokens with the activation quantisation fused in (no inspection
// outputs): gemv_fused_ok(M, K, xdt) tells whether it applies.
bool gemv_fused_ok(int64_t M, int64_t K, termezo_dtype xdt);
hipError_t launch_gemv_fused(const void* x, termezo_dtype xdt, const uint32_t* codes,
                             const float* beta_dev, int64_t M, int64_t K, int64_t N, void* y,
                             termezo_dtype ydt, int n_cu, hipStream_t st);
// Whether kGemmSwiGLU (full-tile path only) supports an M x K x N gate|up pair.
bool gemm_swiglu_ok(int64_t M, int64_t K, int64_t N, termezo_dtype ydt);
hipError_t launch_bitlinear_gemm(const int8_t* xq, const float* s, const int32_t* rs,
                                 const uint32_t* codes, const float* beta_dev, int64_t M, int64_t K, int64_t N,
                                 void* y, termezo_dtype ydt, int32_t* acc, int n_cu,
                                 hipStream_t st);

}  // namespace tmz
