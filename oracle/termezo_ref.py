"""TerMeZO CPU oracle -- TEST INFRASTRUCTURE ONLY.

Plain, slow, obviously-correct statement of the TerMeZO sparse zeroth-order
step (Algorithm 1 with K = 1; the full-precision parameters theta frozen or,
when given, perturbed and updated densely with the masked latents),
composed from the C primitives in ``termezo_oracle.c``.  Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import
this module.  It shares no code with the HIP library.

Step by step (paper section in brackets):
  * thresholds tau^l = 0.5 (gamma^l + delta), gamma^l = mean |w^l|   [Sec. 3, eq. quant]
  * distances d_i = min(|w_i - tau|, |w_i + tau|)                    [eq. distance]
  * S_0 = the rho_0 fraction of all latents with the smallest d,
    xi_0 the largest selected distance                               [eq. selection_init]
  * perturbed evaluation at w +/- eps m (.) z, with z regenerated from
    the seed, requantised with the perturbed layer's own threshold    [Algorithm 1]
  * BitLinear: per-token absmax int8 activations x ternary codes     [Sec. 1, Sec. 3]
  * theta' = rnd(theta + sign eps z_theta), z_theta from the same seed
    (Philox stream 1, theta ids in registration order)               [Algorithm 1]
  * g = (F+ - F-) / (2 eps); w <- w - lr g m (.) z;
    theta <- rnd(theta - lr g z_theta)                                [eq. spsa, Algorithm 1]
  * S_{t+1} = {i in S_t : d_i(w_{t+1}) <= xi_0}                      [eq. selection_]
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_LIB_OMP_PATH = os.path.join(_HERE, "liboracle_omp.so")
_lib = None
_loaded = {}

OK, ERR_INVALID, ERR_STATE, ERR_NUMERIC = 0, 1, 2, 5


def _load(path):
    if path in _loaded:
        return _loaded[path]
    if not os.path.exists(path):
        from . import build_oracle  # type: ignore
        build_oracle.build()
    L = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i64, u64, u32, f32, i32 = (ctypes.c_int64, ctypes.c_uint64, ctypes.c_uint32,
                               ctypes.c_float, ctypes.c_int)
    sig = {
        "orc_set_threads": (i32, [i32]),
        "orc_philox4x32_10": (None, [P, P, P]),
        "orc_ln": (f32, [f32]),
        "orc_ln_array": (None, [P, i64, P]),
        "orc_sincos_turn24": (None, [u32, P, P]),
        "orc_sincos_turn24_array": (None, [P, i64, P, P]),
        "orc_gauss_one": (f32, [u64, u32, u64]),
        "orc_gauss": (None, [u64, u32, P, i64, P]),
        "orc_gauss_range": (None, [u64, u32, i64, i64, P]),
        "orc_fix_abs": (i64, [f32]),
        "orc_layer_abs_sum": (i32, [P, i64, P]),
        "orc_threshold": (None, [i64, i64, f32, P, P]),
        "orc_quantize": (None, [P, i64, f32, P]),
        "orc_distance": (None, [P, i64, f32, P]),
        "orc_select": (i32, [P, i64, i64, i32, P, i64, P, P]),
        "orc_perturbed_layer": (None, [P, i64, P, i64, i64, u64, f32, i32, P]),
        "orc_act_quant": (None, [P, i64, i64, P, P]),
        "orc_bitlinear": (None, [P, P, P, f32, i64, i64, i64, P, P]),
        "orc_bf16_round_array": (None, [P, i64, P]),
        "orc_update_layer": (None, [P, P, i64, i64, u64, f32, f32, i32]),
        "orc_shrink_layer": (i64, [P, P, i64, f32, f32]),
        "orc_theta_perturbed": (None, [P, i64, i64, u64, f32, i32, i32, P]),
        "orc_theta_update": (None, [P, i64, i64, u64, f32, f32, i32]),
        "orc_multi_coeff": (f32, [f32, i32, f32]),
        "orc_update_layer_multi": (None, [P, P, i64, i64, P, P, i32, f32, i32]),
        "orc_theta_update_multi": (None, [P, i64, i64, P, P, i32, f32, i32]),
        "orc_es_standardize": (None, [P, i32, P]),
        "orc_es_coeffs": (None, [P, i32, f32, i32, P]),
        "orc_update_layer_coeffs": (None, [P, P, i64, i64, P, P, i32, i32]),
        "orc_theta_update_coeffs": (None, [P, i64, i64, P, P, i32, i32]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _loaded[path] = L
    return L


def lib():
    """The C oracle library in use (built on first use if absent): the plain
    single-threaded build unless use_threads() chose the OpenMP one."""
    global _lib
    if _lib is None:
        _lib = _load(_LIB_PATH)
    return _lib


def use_threads(n: int) -> int:
    """Run the oracle's independent-iteration loops on n host threads (the OpenMP
    build of the same source; n = 1 selects the plain single-threaded build).
    Results do not depend on it.  Returns the thread count in effect."""
    global _lib
    if n <= 1:
        _lib = _load(_LIB_PATH)
        return 1
    _lib = _load(_LIB_OMP_PATH)
    return int(_lib.orc_set_threads(int(n)))


def _p(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


def _i64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int64)


# --------------------------------------------------------------------------
# Generator primitives
# --------------------------------------------------------------------------
def philox4x32_10(ctr: Sequence[int], key: Sequence[int]) -> Tuple[int, int, int, int]:
    c = (ctypes.c_uint32 * 4)(*[int(v) & 0xFFFFFFFF for v in ctr])
    k = (ctypes.c_uint32 * 2)(*[int(v) & 0xFFFFFFFF for v in key])
    o = (ctypes.c_uint32 * 4)()
    lib().orc_philox4x32_10(c, k, o)
    return tuple(int(v) for v in o)  # type: ignore


def ln(x: np.ndarray) -> np.ndarray:
    x = _f32(x)
    y = np.empty_like(x)
    lib().orc_ln_array(_p(x), x.size, _p(y))
    return y


def sincos_turn24(j: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    j = np.ascontiguousarray(j, dtype=np.uint32)
    s = np.empty(j.shape, np.float32)
    c = np.empty(j.shape, np.float32)
    lib().orc_sincos_turn24_array(_p(j), j.size, _p(s), _p(c))
    return s, c


def gauss(seed: int, gids, stream: int = 0) -> np.ndarray:
    """z_i for the given global ids (fp32), regenerated from (seed, stream)."""
    g = _i64(gids)
    z = np.empty(g.shape, np.float32)
    lib().orc_gauss(seed & (2**64 - 1), stream, _p(g), g.size, _p(z))
    return z


def gauss_range(seed: int, gid0: int, n: int, stream: int = 0) -> np.ndarray:
    z = np.empty(n, np.float32)
    lib().orc_gauss_range(seed & (2**64 - 1), stream, gid0, n, _p(z))
    return z


# --------------------------------------------------------------------------
# Quantiser primitives (Sec. 3)
# --------------------------------------------------------------------------
def layer_abs_sum(w: np.ndarray) -> int:
    """Exact S = sum floor(|w| 2^36); raises on |w| >= 4 or non-finite."""
    w = _f32(w).ravel()
    out = ctypes.c_int64()
    rc = lib().orc_layer_abs_sum(_p(w), w.size, ctypes.byref(out))
    if rc != OK:
        raise FloatingPointError("latent out of the fixed-point range (|w| >= 4 or non-finite)")
    return int(out.value)


def threshold(S: int, n: int, delta: float) -> Tuple[float, float]:
    """(tau, beta) as fp32 from the exact sum S of a layer with n weights."""
    tau = ctypes.c_float()
    beta = ctypes.c_float()
    lib().orc_threshold(int(S), int(n), float(delta), ctypes.byref(tau), ctypes.byref(beta))
    return float(np.float32(tau.value)), float(np.float32(beta.value))


def quantize(w: np.ndarray, tau: float) -> np.ndarray:
    w = _f32(w)
    c = np.empty(w.shape, np.int8)
    lib().orc_quantize(_p(w), w.size, float(tau), _p(c))
    return c


def distance(w: np.ndarray, tau: float) -> np.ndarray:
    w = _f32(w)
    d = np.empty(w.shape, np.float32)
    lib().orc_distance(_p(w), w.size, float(tau), _p(d))
    return d


def select(d_all: np.ndarray, k: int, inclusive: bool = False) -> Tuple[np.ndarray, float]:
    """Sorted gids of the k smallest (d, gid) pairs, and xi0 (the k-th d)."""
    d_all = _f32(d_all).ravel()
    cap = d_all.size
    out = np.empty(cap, np.int64)
    n = ctypes.c_int64()
    xi = ctypes.c_float()
    rc = lib().orc_select(_p(d_all), d_all.size, int(k), int(bool(inclusive)), _p(out), cap,
                          ctypes.byref(n), ctypes.byref(xi))
    if rc != OK:
        raise ValueError(f"selection failed (status {rc})")
    return out[: n.value].copy(), float(np.float32(xi.value))


def bf16_round(x: np.ndarray) -> np.ndarray:
    x = _f32(x)
    y = np.empty_like(x)
    lib().orc_bf16_round_array(_p(x), x.size, _p(y))
    return y


# --------------------------------------------------------------------------
# Layer-level steps of Algorithm 1 for callers that hold one layer at a time
# (global ids start at gid0); the same routines TerMeZOOracle applies.
# --------------------------------------------------------------------------
def perturbed_layer_values(w: np.ndarray, act, gid0: int, seed: int, eps: float,
                           sign: int) -> np.ndarray:
    """w + sign eps z(seed) at the active local indices act, w elsewhere."""
    w = _f32(w).ravel()
    act = _i64(act)
    out = np.empty_like(w)
    lib().orc_perturbed_layer(_p(w), w.size, _p(act), act.size, int(gid0),
                              seed & (2**64 - 1), float(eps), int(sign), _p(out))
    return out


def updated_layer_values(w: np.ndarray, act, gid0: int, seed: int, lr: float, g: float,
                         bf16: bool) -> np.ndarray:
    """A copy of w after w_i <- rnd(fma(-(lr g), z_i, w_i)) at the actives."""
    w = _f32(w).ravel().copy()
    act = _i64(act)
    lib().orc_update_layer(_p(w), _p(act), act.size, int(gid0), seed & (2**64 - 1), float(lr),
                           float(g), int(bool(bf16)))
    return w


def theta_perturbed(theta: np.ndarray, tid0: int, seed: int, eps: float, sign: int,
                    bf16: bool) -> np.ndarray:
    """theta'_i = rnd(fma(sign eps, z_i, theta_i)) with z on Philox stream 1 at ids tid0 + i."""
    theta = _f32(theta).ravel()
    out = np.empty_like(theta)
    lib().orc_theta_perturbed(_p(theta), theta.size, int(tid0), seed & (2**64 - 1), float(eps),
                              int(sign), int(bool(bf16)), _p(out))
    return out


def theta_updated(theta: np.ndarray, tid0: int, seed: int, lr: float, g: float,
                  bf16: bool) -> np.ndarray:
    """A copy of theta after theta_i <- rnd(fma(-(lr g), z_i, theta_i)) (stream 1)."""
    theta = _f32(theta).ravel().copy()
    lib().orc_theta_update(_p(theta), theta.size, int(tid0), seed & (2**64 - 1), float(lr),
                           float(g), int(bool(bf16)))
    return theta


def multi_coeff(lr: float, K: int, g: float) -> float:
    """a_k = -((lr / K) g_k) in fp32 (the coefficient of direction k)."""
    return float(np.float32(lib().orc_multi_coeff(float(lr), int(K), float(g))))


def es_standardize(rewards) -> np.ndarray:
    """Population z-score of the rewards (fp64, index order), rounded to fp32;
    all zero when the standard deviation is zero (RL appendix, ES reading)."""
    r = _f32(np.asarray(rewards)).ravel()
    out = np.empty(r.size, np.float32)
    lib().orc_es_standardize(_p(r), r.size, _p(out))
    return out


def es_coeffs(rewards, lr: float, standardize: bool = True) -> np.ndarray:
    """a_n = (lr / N) * Rt_n in fp32 (Rt: standardised or raw rewards)."""
    r = _f32(np.asarray(rewards)).ravel()
    out = np.empty(r.size, np.float32)
    lib().orc_es_coeffs(_p(r), r.size, float(lr), int(bool(standardize)), _p(out))
    return out


def shrink_layer(w: np.ndarray, act, tau: float, xi0: float) -> np.ndarray:
    """The actives kept by eq. selection_ (distance to tau at most xi0), in order."""
    w = _f32(w).ravel()
    act = _i64(act).copy()
    n = lib().orc_shrink_layer(_p(w), _p(act), act.size, float(tau), float(xi0))
    return act[:n].copy()


# --------------------------------------------------------------------------
# BitLinear (8-bit activations x ternary weights)
# --------------------------------------------------------------------------
def act_quant(x: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    x = _f32(x)
    M, K = x.shape
    xq = np.empty((M, K), np.int8)
    s = np.empty(M, np.float32)
    lib().orc_act_quant(_p(x), M, K, _p(xq), _p(s))
    return xq, s


def bitlinear(xq: np.ndarray, s: np.ndarray, codes: np.ndarray, beta: float,
              want_acc: bool = True) -> Tuple[Optional[np.ndarray], np.ndarray]:
    """Plain triple loop: acc = x_q c^T (int32), y = acc * (beta / s_m)."""
    xq = np.ascontiguousarray(xq, np.int8)
    s = _f32(s)
    codes = np.ascontiguousarray(codes, np.int8)
    M, K = xq.shape
    N = codes.shape[0]
    assert codes.shape[1] == K
    acc = np.empty((M, N), np.int32) if want_acc else None
    y = np.empty((M, N), np.float32)
    lib().orc_bitlinear(_p(xq), _p(s), _p(codes), float(beta), M, K, N,
                        _p(acc) if acc is not None else None, _p(y))
    return acc, y


def bitlinear_matmul(xq: np.ndarray, s: np.ndarray, codes: np.ndarray, beta: float):
    """Same result as ``bitlinear`` with the integer contraction done by a
    library fp32 matmul.  Exact: every term is an integer of magnitude <= 128
    and every partial sum is bounded by 128 K < 2^24 for K < 131072, so all
    fp32 additions (in any order, with or without fma) are exact."""
    M, K = xq.shape
    assert K < 131072
    accf = np.matmul(xq.astype(np.float32), codes.astype(np.float32).T)
    acc = accf.astype(np.int32)
    r = (np.float32(beta) / _f32(s)).astype(np.float32)
    y = (acc.astype(np.float32) * r[:, None]).astype(np.float32)
    return acc, y


def mse(y: np.ndarray, target: np.ndarray) -> float:
    """MSE loss of the single-layer workload: e = y - t and e^2 in fp32, the mean accumulated in fp64."""
    e = (_f32(y) - _f32(target)).astype(np.float32)
    e2 = (e * e).astype(np.float32)
    return float(np.float32(np.sum(e2.astype(np.float64)) / e2.size))


def projected_grad(f_plus: float, f_minus: float, eps: float) -> float:
    """g = (F+ - F-) / (2 eps) in fp32 (eq. spsa, Algorithm 1)."""
    fp, fm, e = np.float32(f_plus), np.float32(f_minus), np.float32(eps)
    return float(np.float32(np.float32(fp - fm) / np.float32(np.float32(2.0) * e)))


# --------------------------------------------------------------------------
# Algorithm-1 state
# --------------------------------------------------------------------------
def eq_memory(m_mezo: float, d: float, rho0: float, B: float = 2.0, B_Q: float = 0.25,
              mask: str = "min") -> float:
    """Peak memory of TerMeZO in bytes from that of MeZO (Sec. 5, eq. memory): the frozen
    fraction of the d latents drops from B to B_Q bytes, the rho0 d active ones keep a
    B_Q-byte quantised copy besides their B bytes, plus the mask -- a bitmask of ceil(d/8)
    bytes, an index list of ceil(rho0 d ceil(log2 d) / 8) bytes, or the smaller of the two
    ("min", as the paper states it)."""
    frozen = math.ceil(d * (1.0 - rho0) * (B - B_Q))
    active_codes = math.ceil(rho0 * d * B_Q)
    bitmask = math.ceil(d / 8.0)
    index_list = math.ceil(rho0 * d * math.ceil(math.log2(d)) / 8.0)
    m_mask = {"bitmask": bitmask, "index": index_list, "min": min(bitmask, index_list)}[mask]
    return m_mezo - frozen + active_codes + m_mask


@dataclass
class Layer:
    d_out: int
    d_in: int

    @property
    def n(self) -> int:
        return self.d_out * self.d_in


@dataclass
class TerMeZOOracle:
    """Latent weights of the ternary projections and the TerMeZO state.

    ``w`` holds every latent in global-id order as fp32 (bf16 latents are held
    widened, and updates round back to bf16)."""
    layers: List[Layer]
    w: np.ndarray
    bf16: bool = False
    delta: float = 1e-5
    offsets: np.ndarray = field(init=False)
    S: List[int] = field(init=False)          # exact fixed-point |w| sums (clean)
    tau: List[float] = field(init=False)
    beta: List[float] = field(init=False)
    active: List[np.ndarray] = field(init=False)  # ascending local indices per layer
    xi0: Optional[float] = None
    k0: int = 0
    last_seed: Optional[int] = None
    last_eps: Optional[float] = None
    # full-precision parameters theta (all registered tensors concatenated in
    # registration order, held as fp32; bf16 storage rounds perturbed and
    # updated values back to bf16).  None: theta frozen.
    theta: Optional[np.ndarray] = None
    theta_bf16: bool = False
    theta_cur: Optional[np.ndarray] = field(init=False, default=None)

    def __post_init__(self):
        if self.theta is not None:
            self.theta = _f32(self.theta).ravel().copy()
            if self.theta_bf16:
                assert np.array_equal(bf16_round(self.theta), self.theta), "bf16 theta must be bf16 values"
            self.theta_cur = self.theta.copy()
        self.w = _f32(self.w).ravel().copy()
        sizes = [l.n for l in self.layers]
        self.offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
        assert self.offsets[-1] == self.w.size
        if self.bf16:
            assert np.array_equal(bf16_round(self.w), self.w), "bf16 latents must be bf16 values"
        self.active = [np.empty(0, np.int64) for _ in self.layers]
        self._refresh_thresholds()

    # -- helpers ----------------------------------------------------------
    @property
    def D(self) -> int:
        return int(self.offsets[-1])

    def layer_w(self, l: int) -> np.ndarray:
        return self.w[self.offsets[l]: self.offsets[l + 1]]

    def _refresh_thresholds(self):
        self.S, self.tau, self.beta = [], [], []
        for l, L in enumerate(self.layers):
            S = layer_abs_sum(self.layer_w(l))
            tau, beta = threshold(S, L.n, self.delta)
            self.S.append(S)
            self.tau.append(tau)
            self.beta.append(beta)

    def clean_codes(self, l: int) -> np.ndarray:
        L = self.layers[l]
        return quantize(self.layer_w(l), self.tau[l]).reshape(L.d_out, L.d_in)

    @property
    def k(self) -> int:
        return int(sum(a.size for a in self.active))

    # -- eq. selection_init --------------------------------------------------
    def build_mask(self, rho0: float, inclusive: bool = False) -> Tuple[int, float]:
        self._refresh_thresholds()
        d_all = np.concatenate([distance(self.layer_w(l), self.tau[l])
                                for l in range(len(self.layers))])
        k0 = int(np.floor(np.float64(np.float32(rho0)) * np.float64(self.D)))
        if k0 <= 0:
            raise ValueError("rho0 * D rounds down to an empty mask")
        gids, xi0 = select(d_all, k0, inclusive)
        self.active = []
        for l in range(len(self.layers)):
            lo, hi = self.offsets[l], self.offsets[l + 1]
            sel = gids[(gids >= lo) & (gids < hi)] - lo
            self.active.append(sel.astype(np.int64))
        self.xi0, self.k0 = xi0, int(gids.size)
        return self.k0, xi0

    # -- Algorithm 1: perturbed evaluation ----------------------------------
    def perturbed_layer(self, l: int, seed: int, eps: float, sign: int) -> np.ndarray:
        L = self.layers[l]
        w = self.layer_w(l)
        out = np.empty_like(w)
        act = _i64(self.active[l])
        lib().orc_perturbed_layer(_p(w), w.size, _p(act), act.size, int(self.offsets[l]),
                                  seed & (2**64 - 1), float(eps), int(sign), _p(out))
        return out

    def perturb(self, seed: int, eps: float, sign: int):
        """Codes, tau' and beta' of every layer at w + sign eps m (.) z(seed)."""
        codes, taus, betas = [], [], []
        for l, L in enumerate(self.layers):
            wp = self.perturbed_layer(l, seed, eps, sign)
            S = layer_abs_sum(wp)
            tau, beta = threshold(S, L.n, self.delta)
            codes.append(quantize(wp, tau).reshape(L.d_out, L.d_in))
            taus.append(tau)
            betas.append(beta)
        if self.theta is not None:
            self.theta_cur = (theta_perturbed(self.theta, 0, seed, eps, sign, self.theta_bf16)
                              if sign != 0 else self.theta.copy())
        self.last_seed, self.last_eps = seed, eps
        return codes, taus, betas

    # -- Algorithm 1 with K directions: all estimates at w_t, then the K updates
    def update_multi(self, seeds: Sequence[int], gs: Sequence[float], lr: float) -> int:
        """w <- rnd(fma chain over k of -(lr/K) g_k z_k) at the actives (and theta
        densely, stream 1), then the thresholds and eq. selection_."""
        K = len(seeds)
        assert K == len(gs) and K >= 1
        sd = np.array([s & (2**64 - 1) for s in seeds], dtype=np.uint64)
        gg = np.array(gs, dtype=np.float32)
        for l in range(len(self.layers)):
            w = self.layer_w(l)
            act = _i64(self.active[l])
            lib().orc_update_layer_multi(_p(w), _p(act), act.size, int(self.offsets[l]), _p(sd),
                                         _p(gg), K, float(lr), int(self.bf16))
        if self.theta is not None:
            lib().orc_theta_update_multi(_p(self.theta), self.theta.size, 0, _p(sd), _p(gg), K,
                                         float(lr), int(self.theta_bf16))
            self.theta_cur = self.theta.copy()
        self._refresh_thresholds()
        for l in range(len(self.layers)):
            act = _i64(self.active[l]).copy()
            n = lib().orc_shrink_layer(_p(self.layer_w(l)), _p(act), act.size,
                                       float(self.tau[l]), float(self.xi0))
            self.active[l] = act[:n].copy()
        self.last_seed = None
        return self.k

    def es_update(self, seeds: Sequence[int], rewards: Sequence[float], lr: float,
                  standardize: bool = True) -> int:
        """Evolution strategies on the mask (RL appendix): w <- rnd(fma chain over n
        of a_n z_n) at the actives (theta densely, stream 1), a_n = (lr/N) Rt_n,
        then the thresholds and eq. selection_ as after any update."""
        N = len(seeds)
        assert N == len(rewards) and N >= 1
        sd = np.array([s & (2**64 - 1) for s in seeds], dtype=np.uint64)
        a = es_coeffs(rewards, lr, standardize)
        for l in range(len(self.layers)):
            w = self.layer_w(l)
            act = _i64(self.active[l])
            lib().orc_update_layer_coeffs(_p(w), _p(act), act.size, int(self.offsets[l]), _p(sd),
                                          _p(a), N, int(self.bf16))
        if self.theta is not None:
            lib().orc_theta_update_coeffs(_p(self.theta), self.theta.size, 0, _p(sd), _p(a), N,
                                          int(self.theta_bf16))
            self.theta_cur = self.theta.copy()
        self._refresh_thresholds()
        for l in range(len(self.layers)):
            act = _i64(self.active[l]).copy()
            n = lib().orc_shrink_layer(_p(self.layer_w(l)), _p(act), act.size,
                                       float(self.tau[l]), float(self.xi0))
            self.active[l] = act[:n].copy()
        self.last_seed = None
        return self.k

    # -- Algorithm 1: update, then eq. selection_ ---------------------------
    def update(self, g: float, lr: float) -> int:
        assert self.last_seed is not None, "update needs a preceding perturbation"
        for l in range(len(self.layers)):
            w = self.layer_w(l)
            act = _i64(self.active[l])
            lib().orc_update_layer(_p(w), _p(act), act.size, int(self.offsets[l]),
                                   self.last_seed & (2**64 - 1), float(lr), float(g),
                                   int(self.bf16))
        if self.theta is not None:
            self.theta = theta_updated(self.theta, 0, self.last_seed, lr, g, self.theta_bf16)
            self.theta_cur = self.theta.copy()
        self._refresh_thresholds()
        for l in range(len(self.layers)):
            act = _i64(self.active[l]).copy()
            n = lib().orc_shrink_layer(_p(self.layer_w(l)), _p(act), act.size,
                                       float(self.tau[l]), float(self.xi0))
            self.active[l] = act[:n].copy()
        self.last_seed = None
        return self.k
