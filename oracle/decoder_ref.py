"""BitNet decoder forward and next-token loss -- CPU oracle, TEST INFRASTRUCTURE ONLY.

The paper fixes the BitNet structure only in outline (Sec. 3): every linear
projection of a transformer block (q, k, v, o and the MLP linears) is a ternary
BitLinear with 8-bit activations, while the embeddings, the normalisation
layers and the LM head stay in full precision (theta: frozen, or perturbed and
updated by the caller, which passes the values to evaluate).  The
objective is the batch mean of the per-sample loss (eq. objective_est); for
supervised fine-tuning that is next-token cross-entropy.  The remaining details
are readings (the paper is silent on them):

  * pre-norm blocks with RMSNorm (eps 1e-5; weights one unless given: row
    2 b scales the attention input of block b, row 2 b + 1 the MLP input, the
    last row the LM-head input);
  * rotary position embedding, base 10000, on (i, i + head_dim/2) pairs;
  * causal grouped-query attention with softmax scale 1/sqrt(head_dim);
  * SwiGLU MLP: down( silu(gate x) * up x );
  * LM head tied to the token embedding;
  * storage between kernels in the activation dtype (fp32 or bf16, rounded to
    nearest-even); the RMSNorm output feeding a BitLinear and the SwiGLU
    product are consumed in fp32 by the activation quantiser, never stored;
    residual adds round the projection output, then the sum.

Reference arithmetic is fp64 except where the paper's method fixes the
precision: activation quantisation and the BitLinear accumulation follow the
fp32 / int32 definitions of the oracle's C primitives.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np

from . import termezo_ref as orc


@dataclass
class DecoderConfig:
    n_blocks: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    d_ffn: int
    vocab: int
    bf16: bool = False
    rope_base: float = 10000.0
    norm_eps: float = 1e-5

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads

    def layer_shapes(self):
        """(d_out, d_in) of the seven ternary projections of one block, in the
        registration order q, k, v, o, gate, up, down."""
        d, hd, F = self.d_model, self.head_dim, self.d_ffn
        q, kv = self.n_heads * hd, self.n_kv_heads * hd
        blk = [(q, d), (kv, d), (kv, d), (d, q), (F, d), (F, d), (d, F)]
        return blk * self.n_blocks


def store(x: np.ndarray, bf16: bool) -> np.ndarray:
    """Round to the activation storage dtype (kept as fp32 values)."""
    x = np.asarray(x, dtype=np.float64).astype(np.float32)
    return orc.bf16_round(x) if bf16 else x


def rmsnorm(h: np.ndarray, eps: float, weight: Optional[np.ndarray] = None) -> np.ndarray:
    """weight * h / sqrt(mean(h^2) + eps) (weight one when None); fp32 result."""
    h64 = h.astype(np.float64)
    r = 1.0 / np.sqrt(np.mean(h64 * h64, axis=-1, keepdims=True) + eps)
    y = h64 * r
    if weight is not None:
        y = y * weight.astype(np.float64)
    return y.astype(np.float32)


def rope(x: np.ndarray, pos: np.ndarray, n_heads: int, head_dim: int, base: float) -> np.ndarray:
    """Rotate the pairs (i, i + head_dim/2) of every head by pos * base^(-2i/head_dim)."""
    M = x.shape[0]
    half = head_dim // 2
    inv = base ** (-2.0 * np.arange(half, dtype=np.float64) / head_dim)
    ang = pos.astype(np.float64)[:, None] * inv[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    xh = x.astype(np.float64).reshape(M, n_heads, head_dim)
    a, b = xh[..., :half], xh[..., half:]
    out = np.concatenate([a * c - b * s, a * s + b * c], axis=-1)
    return out.reshape(M, n_heads * head_dim)


def attention(q, k, v, B, S, Hq, Hkv, hd) -> np.ndarray:
    """Causal grouped-query attention; query head h reads kv head h // (Hq/Hkv)."""
    group = Hq // Hkv
    q = q.astype(np.float64).reshape(B, S, Hq, hd)
    k = k.astype(np.float64).reshape(B, S, Hkv, hd)
    v = v.astype(np.float64).reshape(B, S, Hkv, hd)
    out = np.empty((B, S, Hq, hd))
    causal = np.tril(np.ones((S, S), bool))
    for b in range(B):
        for h in range(Hq):
            kh = h // group
            sc = q[b, :, h, :] @ k[b, :, kh, :].T / np.sqrt(hd)
            sc = np.where(causal, sc, -np.inf)
            sc -= sc.max(axis=1, keepdims=True)
            p = np.exp(sc)
            p /= p.sum(axis=1, keepdims=True)
            out[b, :, h, :] = p @ v[b, :, kh, :]
    return out.reshape(B * S, Hq * hd)


def silu_mul(g: np.ndarray, u: np.ndarray) -> np.ndarray:
    g64 = g.astype(np.float64)
    return (g64 / (1.0 + np.exp(-g64)) * u.astype(np.float64)).astype(np.float32)


def bitlinear_fp32_in(x32: np.ndarray, codes: np.ndarray, beta: float) -> np.ndarray:
    """BitLinear on an fp32 input: 8-bit activation quantisation, exact integer
    contraction, rescale (the oracle's C primitives plus an exact matmul)."""
    xq, s = orc.act_quant(x32)
    _, y = orc.bitlinear_matmul(xq, s, codes, beta)
    return y


def forward_row_losses(cfg: DecoderConfig, emb: np.ndarray, tokens: np.ndarray,
                       codes: Sequence[np.ndarray], betas: Sequence[float],
                       norm_w: Optional[np.ndarray] = None) -> np.ndarray:
    """Per-position cross-entropy [B, S] (position S-1 has no label: 0).

    emb: [V, d] fp32 values (bf16 values when cfg.bf16); tokens: [B, S];
    codes/betas: ternary codes and scales of the 7 * n_blocks projections;
    norm_w: RMSNorm weights [2 n_blocks + 1, d] (None: one)."""
    nw = (lambda i: None) if norm_w is None else (lambda i: norm_w.reshape(-1, cfg.d_model)[i])
    B, S = tokens.shape
    d, Hq, Hkv, hd = cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    bf = cfg.bf16
    M = B * S
    pos = np.tile(np.arange(S), B)
    h = store(emb[tokens.reshape(-1)], bf)
    for blk in range(cfg.n_blocks):
        c = codes[7 * blk: 7 * blk + 7]
        be = betas[7 * blk: 7 * blk + 7]
        x = rmsnorm(h, cfg.norm_eps, nw(2 * blk))
        q = store(bitlinear_fp32_in(x, c[0], be[0]), bf)
        k = store(bitlinear_fp32_in(x, c[1], be[1]), bf)
        v = store(bitlinear_fp32_in(x, c[2], be[2]), bf)
        q = store(rope(q, pos, Hq, hd, cfg.rope_base), bf)
        k = store(rope(k, pos, Hkv, hd, cfg.rope_base), bf)
        a = store(attention(q, k, v, B, S, Hq, Hkv, hd), bf)
        o = store(bitlinear_fp32_in(a, c[3], be[3]), bf)
        h = store(h.astype(np.float64) + o, bf)
        x = rmsnorm(h, cfg.norm_eps, nw(2 * blk + 1))
        g = store(bitlinear_fp32_in(x, c[4], be[4]), bf)
        u = store(bitlinear_fp32_in(x, c[5], be[5]), bf)
        m = store(silu_mul(g, u), bf)
        dn = store(bitlinear_fp32_in(m, c[6], be[6]), bf)
        h = store(h.astype(np.float64) + dn, bf)
    xf = store(rmsnorm(h, cfg.norm_eps, nw(2 * cfg.n_blocks)), bf)
    logits = xf.astype(np.float64) @ emb.astype(np.float64).T          # [M, V]
    lab = np.zeros((B, S), np.int64)
    lab[:, :-1] = tokens[:, 1:]
    row = cross_entropy_rows(logits, lab.reshape(-1))
    row = row.reshape(B, S)
    row[:, -1] = 0.0
    return row


def cross_entropy_rows(logits: np.ndarray, labels: np.ndarray) -> np.ndarray:
    """logsumexp(logits_m) - logits_m[label_m] per row, with max subtraction."""
    mx = logits.max(axis=1, keepdims=True)
    lse = mx[:, 0] + np.log(np.exp(logits - mx).sum(axis=1))
    return lse - logits[np.arange(logits.shape[0]), labels]


def mean_loss(row_losses: np.ndarray) -> float:
    """Batch mean over the B (S - 1) labelled positions (eq. objective_est)."""
    B, S = row_losses.shape
    return float(np.float32(row_losses.sum() / (B * (S - 1))))
