"""Python binding of the TerMeZO C ABI (libtermezo.so).

Argument marshalling only: every step of the TerMeZO path runs in the HIP
kernels of libtermezo.so.  PyTorch tensors supply device memory and the HIP
stream.  The library must be built (``python -m paper_2609_33548_amd.build``);
importing this module without it raises ImportError.
"""
from __future__ import annotations

import atexit
import ctypes
import os
import sys
import weakref
from typing import List, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtermezo.so")

OK, ERR_INVALID_ARG, ERR_STATE, ERR_DEVICE, ERR_OOM, ERR_NUMERIC = range(6)
F32, BF16, I8, I32 = range(4)
STATUS_NAMES = {0: "OK", 1: "INVALID_ARG", 2: "STATE", 3: "DEVICE", 4: "OOM", 5: "NUMERIC"}


class TermezoError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"termezo {STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class Layer(ctypes.Structure):
    _fields_ = [("latent", ctypes.c_void_p), ("d_out", ctypes.c_int64), ("d_in", ctypes.c_int64)]


class Theta(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("n", ctypes.c_int64), ("dtype", ctypes.c_int32)]


class ModelConfig(ctypes.Structure):
    _fields_ = [("n_blocks", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("d_ffn", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("rope_base", ctypes.c_float), ("norm_eps", ctypes.c_float),
                ("act_dtype", ctypes.c_int32)]


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_33548_amd.build`")

_lib = ctypes.CDLL(LIB_PATH)
_P = ctypes.c_void_p
_i32, _i64, _u64, _f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_float
_SIGS = {
    "termezo_create": [ctypes.POINTER(Layer), _i32, _i32, _P, ctypes.POINTER(_P)],
    "termezo_destroy": [_P],
    "termezo_last_error": [_P],
    "termezo_build_mask": [_P, _f32, _f32, _i32, ctypes.POINTER(_i64), ctypes.POINTER(_f32)],
    "termezo_perturb": [_P, _u64, _f32, _i32],
    "termezo_bitlinear_forward": [_P, _i32, _P, _i32, _i64, _P, _i32, _P, _P, _P],
    "termezo_update": [_P, _f32, _f32, ctypes.POINTER(_i64)],
    "termezo_sync": [_P],
    "termezo_mask_export": [_P, _i32, _P, _i64, ctypes.POINTER(_i64)],
    "termezo_codes_export": [_P, _i32, _P],
    "termezo_layer_stats": [_P, _i32, ctypes.POINTER(_f32), ctypes.POINTER(_f32),
                            ctypes.POINTER(_i64), ctypes.POINTER(_f32), ctypes.POINTER(_f32)],
    "termezo_mse_loss": [_P, _P, _P, _i64, ctypes.POINTER(_f32)],
    "termezo_mse_loss_dev": [_P, _P, _P, _i64, _P],
    "termezo_bitlinear_forward_noalloc": [_P, _i32, _P, _i32, _i64, _P, _i32],
    "termezo_active_count": [_P, ctypes.POINTER(_i64)],
    "termezo_gauss": [_P, _u64, _P, _i64, _P],
    "termezo_update_from_losses": [_P, _P, _P, _f32, _f32],
    "termezo_update_multi": [_P, _P, _P, _i32, _f32, ctypes.POINTER(_i64)],
    "termezo_update_multi_from_losses": [_P, _P, _P, _i32, _f32, _f32],
    "termezo_es_update": [_P, _P, _P, _i32, _f32, _i32, ctypes.POINTER(_i64)],
    "termezo_es_update_from_rewards": [_P, _P, _P, _i32, _f32, _i32],
    "termezo_theta_register": [_P, ctypes.POINTER(Theta), _i32],
    "termezo_set_dense_requant": [_P, _i32],
    "termezo_compact": [_P],
    "termezo_active_values": [_P, _i32, _P, _i64, ctypes.POINTER(_i64)],
    "termezo_memory_footprint": [_P, ctypes.POINTER(_i64), ctypes.POINTER(_i64)],
    "termezo_theta_current": [_P, _i32, ctypes.POINTER(_P)],
    "termezo_theta_copy": [_P, _i32, _P],
    "termezo_model_create": [_P, _P, _P, ctypes.POINTER(_P)],
    "termezo_model_set_norm_weights": [_P, _P],
    "termezo_model_destroy": [_P],
    "termezo_model_loss": [_P, _P, _i32, _i32, _P, _P, ctypes.POINTER(_f32)],
    "termezo_model_set_timing": [_P, _i32],
    "termezo_model_timing": [_P, _i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_i64),
                             ctypes.POINTER(ctypes.c_double)],
    "termezo_codes_snapshot": [_P],
    "termezo_model_set_stream": [_P, _P],
    "termezo_model_use_snapshot": [_P, _i32],
    "termezo_model_join": [_P],
}
for _name, _args in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.argtypes = _args
    _fn.restype = None if _name in ("termezo_destroy", "termezo_model_destroy") else (
        ctypes.c_char_p if _name == "termezo_last_error" else ctypes.c_int)

lib = _lib
_is_finalizing = sys.is_finalizing   # bound now: module globals may be gone at teardown

# Contexts still open; closed (models first) before interpreter teardown, while
# the HIP runtime is still alive.
_LIVE = weakref.WeakSet()


@atexit.register
def _close_all():
    for ctx in list(_LIVE):
        try:
            ctx.close()
        except Exception:
            pass


def _ptr(t) -> Optional[int]:
    """Device address of a torch tensor (None passes NULL)."""
    return None if t is None else int(t.data_ptr())


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


# --------------------------------------------------------------------------
# Thin wrappers with the C names
# --------------------------------------------------------------------------
def termezo_create(layers: Sequence[Tuple[int, int, int]], latent_dtype: int, stream: Optional[int]):
    arr = (Layer * len(layers))(*[Layer(p, o, i) for p, o, i in layers])
    out = _P()
    st = _lib.termezo_create(arr, len(layers), latent_dtype, stream, ctypes.byref(out))
    if st != OK:
        raise TermezoError(st, "termezo_create failed")
    return out.value


class Context:
    """A registered set of ternary projections and its TerMeZO state.

    ``latents`` are torch device tensors [d_out, d_in] (all fp32 or all bf16)
    that the caller keeps alive; the library updates them in place."""

    def __init__(self, latents, stream=None):
        import torch
        if not latents:
            raise ValueError("at least one layer")
        dt = latents[0].dtype
        for w in latents:
            if w.dtype != dt or w.dim() != 2 or not w.is_contiguous() or not w.is_cuda:
                raise ValueError("latents must be contiguous 2-D device tensors of one dtype")
        self.latents = list(latents)
        self.dtype_code = _dtype_code(latents[0])
        self.shapes = [tuple(w.shape) for w in latents]
        self._stream = stream if stream is not None else torch.cuda.current_stream()
        self.handle = termezo_create([(w.data_ptr(), w.shape[0], w.shape[1]) for w in latents],
                                     self.dtype_code, int(self._stream.cuda_stream))
        self._models = weakref.WeakSet()
        _LIVE.add(self)

    def _check(self, st: int, what: str):
        if st != OK:
            msg = _lib.termezo_last_error(self.handle)
            raise TermezoError(st, f"{what}: {msg.decode() if msg else ''}")

    def close(self):
        for m in list(getattr(self, "_models", ())):
            m.close()
        if getattr(self, "handle", None):
            _lib.termezo_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            if _is_finalizing():
                return
            self.close()
        except Exception:
            pass

    # -- the four hot-path calls ----------------------------------------------
    def build_mask(self, rho0: float, delta: float = 1e-5, tie_inclusive: bool = False):
        k0 = _i64()
        xi0 = _f32()
        self._check(_lib.termezo_build_mask(self.handle, rho0, delta, int(tie_inclusive),
                                            ctypes.byref(k0), ctypes.byref(xi0)), "build_mask")
        return int(k0.value), float(np.float32(xi0.value))

    def perturb(self, seed: int, eps: float, sign: int):
        self._check(_lib.termezo_perturb(self.handle, seed & (2**64 - 1), eps, sign), "perturb")

    def bitlinear_forward(self, layer: int, x, y, xq_out=None, xscale_out=None, acc_out=None):
        M = x.shape[0]
        self._check(_lib.termezo_bitlinear_forward(
            self.handle, layer, _ptr(x), _dtype_code(x), M, _ptr(y), _dtype_code(y),
            _ptr(xq_out), _ptr(xscale_out), _ptr(acc_out)), "bitlinear_forward")

    def bitlinear_forward_noalloc(self, layer: int, x, y):
        """BitLinear forward whose quantisation scratch is the library's fixed device
        array (no allocation; M * d_in + 4 M bytes must fit 16 MiB)."""
        self._check(_lib.termezo_bitlinear_forward_noalloc(
            self.handle, layer, _ptr(x), _dtype_code(x), x.shape[0], _ptr(y), _dtype_code(y)),
            "bitlinear_forward_noalloc")

    def update(self, proj_grad: float, lr: float, want_k: bool = True) -> Optional[int]:
        k = _i64()
        self._check(_lib.termezo_update(self.handle, proj_grad, lr,
                                        ctypes.byref(k) if want_k else None), "update")
        return int(k.value) if want_k else None

    # -- support calls ----------------------------------------------------------
    def sync(self):
        self._check(_lib.termezo_sync(self.handle), "sync")

    def active_count(self) -> int:
        k = _i64()
        self._check(_lib.termezo_active_count(self.handle, ctypes.byref(k)), "active_count")
        return int(k.value)

    def mask(self, layer: int) -> np.ndarray:
        n = _i64()
        d_out, d_in = self.shapes[layer]
        buf = np.empty(max(1, d_out * d_in), np.uint32)
        self._check(_lib.termezo_mask_export(self.handle, layer, buf.ctypes.data, buf.size,
                                             ctypes.byref(n)), "mask_export")
        return buf[: n.value].astype(np.int64)

    def codes(self, layer: int) -> np.ndarray:
        d_out, d_in = self.shapes[layer]
        buf = np.empty((d_out, d_in), np.int8)
        self._check(_lib.termezo_codes_export(self.handle, layer, buf.ctypes.data), "codes_export")
        return buf

    def layer_stats(self, layer: int):
        tau, beta, tc, bc = _f32(), _f32(), _f32(), _f32()
        S = _i64()
        self._check(_lib.termezo_layer_stats(self.handle, layer, ctypes.byref(tau), ctypes.byref(beta),
                                             ctypes.byref(S), ctypes.byref(tc), ctypes.byref(bc)),
                    "layer_stats")
        f = lambda v: float(np.float32(v.value))
        return {"tau": f(tau), "beta": f(beta), "S": int(S.value), "tau_cur": f(tc), "beta_cur": f(bc)}

    def update_from_losses(self, loss_plus, loss_minus, eps: float, lr: float):
        """Device-side g = (F+ - F-) / (2 eps) and update; no host round trip."""
        self._check(_lib.termezo_update_from_losses(self.handle, _ptr(loss_plus), _ptr(loss_minus),
                                                    eps, lr), "update_from_losses")

    def compact(self):
        """Memory-optimal storage: keep only the active latents (library-owned); the
        registered latent tensors are no longer read or written."""
        self._check(_lib.termezo_compact(self.handle), "compact")
        self.latents = None                 # the caller may now free its latent tensors

    def active_values(self, layer: int) -> np.ndarray:
        """fp32 values of one layer's active latents in list order."""
        d_out, d_in = self.shapes[layer]
        buf = np.empty(max(1, d_out * d_in), np.float32)
        n = _i64()
        self._check(_lib.termezo_active_values(self.handle, layer, buf.ctypes.data, buf.size,
                                               ctypes.byref(n)), "active_values")
        return buf[: n.value].copy()

    def memory_footprint(self):
        """(library-owned device bytes, caller latent bytes still needed)."""
        lb, wb = _i64(), _i64()
        self._check(_lib.termezo_memory_footprint(self.handle, ctypes.byref(lb), ctypes.byref(wb)),
                    "memory_footprint")
        return int(lb.value), int(wb.value)

    def set_dense_requant(self, on: bool):
        """Re-quantise every latent on each perturbation (default: only the actives'
        codes while the threshold drift guard proves the frozen codes unchanged)."""
        self._check(_lib.termezo_set_dense_requant(self.handle, int(bool(on))), "set_dense_requant")

    def theta_register(self, tensors):
        """Register full-precision parameters theta (contiguous fp32 or bf16 device
        tensors, kept alive by the caller): from now on perturb and update move them
        with the latents (Algorithm 1)."""
        for t in tensors:
            if not t.is_cuda or not t.is_contiguous():
                raise ValueError("theta tensors must be contiguous device tensors")
        arr = (Theta * len(tensors))(*[Theta(t.data_ptr(), t.numel(), _dtype_code(t)) for t in tensors])
        self._check(_lib.termezo_theta_register(self.handle, arr, len(tensors)), "theta_register")
        self.theta = list(tensors)

    def theta_current_ptr(self, i: int) -> int:
        """Device address of the values the forward reads now for theta tensor i."""
        out = _P()
        self._check(_lib.termezo_theta_current(self.handle, i, ctypes.byref(out)), "theta_current")
        return int(out.value)

    def theta_current(self, i: int):
        """A copy (new device tensor) of the values the forward reads now for theta
        tensor i: the perturbed copy while a +- perturbation is current."""
        import torch
        out = torch.empty_like(self.theta[i])
        self._check(_lib.termezo_theta_copy(self.handle, i, _ptr(out)), "theta_copy")
        return out

    def update_multi(self, seeds, proj_grads, lr: float, want_k: bool = True) -> Optional[int]:
        """K directions (Algorithm 1): one update from the K seeds and projected gradients."""
        K = len(seeds)
        sd = (ctypes.c_uint64 * K)(*[s & (2**64 - 1) for s in seeds])
        gg = (ctypes.c_float * K)(*[float(g) for g in proj_grads])
        k = _i64()
        self._check(_lib.termezo_update_multi(self.handle, sd, gg, K, lr,
                                              ctypes.byref(k) if want_k else None), "update_multi")
        return int(k.value) if want_k else None

    def update_multi_from_losses(self, seeds, losses, eps: float, lr: float):
        """K directions with g_k formed on the device from losses [2K] (F+_k, F-_k pairs)."""
        K = len(seeds)
        sd = (ctypes.c_uint64 * K)(*[s & (2**64 - 1) for s in seeds])
        self._check(_lib.termezo_update_multi_from_losses(self.handle, sd, _ptr(losses), K, eps, lr),
                    "update_multi_from_losses")

    def es_update(self, seeds, rewards, lr: float, standardize: bool = True,
                  want_k: bool = True) -> Optional[int]:
        """Evolution strategies on the mask: the reward-weighted sum of the N
        directions (host rewards), then the shrink."""
        N = len(seeds)
        sd = (ctypes.c_uint64 * N)(*[s & (2**64 - 1) for s in seeds])
        rr = (ctypes.c_float * N)(*[float(r) for r in rewards])
        k = _i64()
        self._check(_lib.termezo_es_update(self.handle, sd, rr, N, lr, int(bool(standardize)),
                                           ctypes.byref(k) if want_k else None), "es_update")
        return int(k.value) if want_k else None

    def es_update_from_rewards(self, seeds, rewards, lr: float, standardize: bool = True):
        """The same with the rewards in a device fp32 tensor [N]; never waits."""
        N = len(seeds)
        sd = (ctypes.c_uint64 * N)(*[s & (2**64 - 1) for s in seeds])
        self._check(_lib.termezo_es_update_from_rewards(self.handle, sd, _ptr(rewards), N, lr,
                                                        int(bool(standardize))),
                    "es_update_from_rewards")

    def codes_snapshot(self):
        """Copy the current codes and output scales into the library's snapshot (no wait)."""
        self._check(_lib.termezo_codes_snapshot(self.handle), "codes_snapshot")

    def mse_loss(self, y, target) -> float:
        out = _f32()
        self._check(_lib.termezo_mse_loss(self.handle, _ptr(y), _ptr(target), y.numel(),
                                          ctypes.byref(out)), "mse_loss")
        return float(np.float32(out.value))

    def mse_loss_dev(self, y, target, loss_dev):
        """The same loss written to the device fp32 scalar loss_dev (no wait)."""
        self._check(_lib.termezo_mse_loss_dev(self.handle, _ptr(y), _ptr(target), y.numel(),
                                              _ptr(loss_dev)), "mse_loss_dev")


class Model:
    """BitNet decoder bound to a Context whose layers are the 7 projections of
    each block (q, k, v, o, gate, up, down); ``embedding`` is the frozen tied
    token embedding [vocab, d_model] (device tensor in the activation dtype)."""

    def __init__(self, ctx: Context, n_blocks: int, d_model: int, n_heads: int, n_kv_heads: int,
                 d_ffn: int, vocab: int, embedding, rope_base: float = 10000.0,
                 norm_eps: float = 1e-5):
        self.ctx = ctx
        self.embedding = embedding
        cfg = ModelConfig(n_blocks, d_model, n_heads, n_kv_heads, d_ffn, vocab, rope_base,
                          norm_eps, _dtype_code(embedding))
        out = _P()
        st = _lib.termezo_model_create(ctx.handle, ctypes.byref(cfg), _ptr(embedding),
                                       ctypes.byref(out))
        if st != OK:
            raise TermezoError(st, "termezo_model_create failed")
        self.handle = out.value
        ctx._models.add(self)

    def set_norm_weights(self, norm_weights):
        """RMSNorm weights [2 n_blocks + 1, d_model] (device tensor in the activation
        dtype, kept alive by the caller); None restores weights one."""
        self.norm_weights = norm_weights
        self.ctx._check(_lib.termezo_model_set_norm_weights(self.handle, _ptr(norm_weights)),
                        "model_set_norm_weights")

    def loss(self, tokens, loss_dev=None, row_loss_dev=None, host: bool = True) -> Optional[float]:
        B, S = tokens.shape
        out = _f32()
        st = _lib.termezo_model_loss(self.handle, _ptr(tokens), B, S, _ptr(loss_dev),
                                     _ptr(row_loss_dev), ctypes.byref(out) if host else None)
        self.ctx._check(st, "model_loss")
        return float(np.float32(out.value)) if host else None

    def set_stream(self, stream):
        """Run this model's forwards on ``stream`` (a torch stream; None: the context's)."""
        self.stream = stream                      # kept alive with the model
        self.ctx._check(_lib.termezo_model_set_stream(
            self.handle, None if stream is None else int(stream.cuda_stream)), "model_set_stream")

    def use_snapshot(self, on: bool):
        self.ctx._check(_lib.termezo_model_use_snapshot(self.handle, int(on)), "model_use_snapshot")

    def join(self):
        self.ctx._check(_lib.termezo_model_join(self.handle), "model_join")

    GEMM, ATTENTION, LM_HEAD = 0, 1, 2

    def set_timing(self, enable: bool):
        self.ctx._check(_lib.termezo_model_set_timing(self.handle, int(enable)), "set_timing")

    def timing(self, cls: int):
        """(kernel ms summed, launches, algorithmic ops) recorded for one class."""
        ms, ops = ctypes.c_double(), ctypes.c_double()
        n = _i64()
        self.ctx._check(_lib.termezo_model_timing(self.handle, cls, ctypes.byref(ms), ctypes.byref(n),
                                                  ctypes.byref(ops)), "timing")
        return float(ms.value), int(n.value), float(ops.value)

    def close(self):
        if getattr(self, "handle", None):
            _lib.termezo_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            if _is_finalizing():
                return
            self.close()
        except Exception:
            pass


def gauss(seed: int, gids, stream=None):
    """z at the given global ids (torch int64 device tensor) as a device fp32 tensor."""
    import torch
    g = gids.to(torch.int64).contiguous()
    z = torch.empty(g.shape, dtype=torch.float32, device=g.device)
    st = _lib.termezo_gauss(_stream_handle(stream), seed & (2**64 - 1), g.data_ptr(), g.numel(),
                            z.data_ptr())
    if st != OK:
        raise TermezoError(st, "termezo_gauss failed")
    return z
