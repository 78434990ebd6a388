"""Pins of the decoder oracle (the BitNet forward around the ternary
projections) against textbook definitions in independent library routines
(torch CPU, fp64) and invariants (rotation norms, relative positions,
causality, uniform logits)."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import decoder_ref as dec
from paper_2609_33548_amd import synth


def test_rmsnorm_matches_torch():
    h = synth.activations(1, 7, 96) * np.float32(3.0)
    ref = F.rms_norm(torch.from_numpy(h).double(), (96,), eps=1e-5).numpy()
    assert np.allclose(dec.rmsnorm(h, 1e-5), ref, rtol=1e-6, atol=1e-7)


def test_weighted_rmsnorm_matches_torch_and_unit_weight():
    rng = np.random.default_rng(1)
    h = rng.standard_normal((5, 48)).astype(np.float32)
    w = (1.0 + 0.1 * rng.standard_normal(48)).astype(np.float32)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(h).double(), (48,),
                                       torch.from_numpy(w).double(), eps=1e-5).numpy()
    assert np.allclose(dec.rmsnorm(h, 1e-5, w), ref, rtol=1e-6, atol=1e-7)
    assert np.array_equal(dec.rmsnorm(h, 1e-5, np.ones(48, np.float32)), dec.rmsnorm(h, 1e-5))


def test_rope_is_complex_rotation_and_relative():
    M, H, hd = 6, 3, 16
    x = synth.activations(2, M, H * hd).astype(np.float64)
    pos = np.array([0, 1, 5, 17, 100, 511])
    got = dec.rope(x, pos, H, hd, 10000.0)
    half = hd // 2
    xc = x.reshape(M, H, 2, half)
    z = xc[:, :, 0, :] + 1j * xc[:, :, 1, :]
    theta = 10000.0 ** (-np.arange(half) * 2.0 / hd)
    zr = z * np.exp(1j * pos[:, None, None] * theta[None, None, :])
    ref = np.concatenate([zr.real, zr.imag], axis=-1).reshape(M, H * hd)
    assert np.allclose(got, ref, atol=1e-12)
    assert np.allclose(np.linalg.norm(got, axis=1), np.linalg.norm(x, axis=1))
    q = synth.activations(3, 1, hd).astype(np.float64)
    k = synth.activations(4, 1, hd).astype(np.float64)
    dots = [float((dec.rope(q, np.array([p + 7]), 1, hd, 1e4) @ dec.rope(k, np.array([p]), 1, hd, 1e4).T)[0, 0])
            for p in (0, 3, 50)]
    assert np.allclose(dots, dots[0])


@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (4, 1), (6, 2)])
def test_attention_matches_torch_sdpa(Hq, Hkv):
    B, S, hd = 2, 9, 8
    q = synth.activations(5, B * S, Hq * hd)
    k = synth.activations(6, B * S, Hkv * hd)
    v = synth.activations(7, B * S, Hkv * hd)
    got = dec.attention(q, k, v, B, S, Hq, Hkv, hd)
    tq = torch.from_numpy(q).double().reshape(B, S, Hq, hd).transpose(1, 2)
    tk = torch.from_numpy(k).double().reshape(B, S, Hkv, hd).transpose(1, 2)
    tv = torch.from_numpy(v).double().reshape(B, S, Hkv, hd).transpose(1, 2)
    tk = tk.repeat_interleave(Hq // Hkv, dim=1)
    tv = tv.repeat_interleave(Hq // Hkv, dim=1)
    ref = F.scaled_dot_product_attention(tq, tk, tv, is_causal=True)
    ref = ref.transpose(1, 2).reshape(B * S, Hq * hd).numpy()
    assert np.allclose(got, ref, atol=1e-12)


def test_silu_mul_matches_torch():
    g = synth.activations(8, 5, 33)
    u = synth.activations(9, 5, 33)
    ref = (F.silu(torch.from_numpy(g).double()) * torch.from_numpy(u).double()).numpy()
    assert np.allclose(dec.silu_mul(g, u), ref, rtol=1e-6, atol=1e-7)


def _tiny(bf16=False):
    cfg = dec.DecoderConfig(n_blocks=2, d_model=64, n_heads=4, n_kv_heads=2, d_ffn=96,
                            vocab=50, bf16=bf16)
    shapes = cfg.layer_shapes()
    rng = np.random.default_rng(0)
    codes = [rng.integers(-1, 2, size=s).astype(np.int8) for s in shapes]
    betas = [0.016] * len(shapes)
    emb = synth.latents(11, [cfg.vocab * cfg.d_model], bf16=bf16).reshape(cfg.vocab, cfg.d_model)
    return cfg, codes, betas, emb


def test_cross_entropy_matches_torch_and_causality():
    cfg, codes, betas, emb = _tiny()
    tok = synth.tokens(1, 2, 12, cfg.vocab)
    rows = dec.forward_row_losses(cfg, emb, tok, codes, betas)
    assert np.all(rows[:, -1] == 0.0) and np.all(rows[:, :-1] > 0)
    # changing the last input token changes only the last labelled position
    tok2 = tok.copy()
    tok2[:, -1] = (tok2[:, -1] + 1) % cfg.vocab
    rows2 = dec.forward_row_losses(cfg, emb, tok2, codes, betas)
    assert np.array_equal(rows[:, :-2], rows2[:, :-2])
    assert not np.array_equal(rows[:, -2], rows2[:, -2])
    # changing a middle token leaves every earlier position untouched
    tok3 = tok.copy()
    tok3[:, 6] = (tok3[:, 6] + 3) % cfg.vocab
    rows3 = dec.forward_row_losses(cfg, emb, tok3, codes, betas)
    assert np.array_equal(rows[:, :5], rows3[:, :5])
    assert dec.mean_loss(rows) == pytest.approx(rows.sum() / (2 * 11), rel=1e-6)


def test_loss_is_log_vocab_for_uniform_logits():
    cfg, codes, betas, _ = _tiny()
    emb = np.ones((cfg.vocab, cfg.d_model), np.float32) * np.float32(0.02)
    tok = synth.tokens(2, 2, 8, cfg.vocab)
    rows = dec.forward_row_losses(cfg, emb, tok, codes, betas)
    assert np.allclose(rows[:, :-1], math.log(cfg.vocab), rtol=1e-12)


def test_cross_entropy_rows_match_torch():
    logits = synth.activations(12, 20, 77).astype(np.float64) * 3.0
    labels = synth.tokens(13, 1, 20, 77)[0].astype(np.int64)
    ref = F.cross_entropy(torch.from_numpy(logits), torch.from_numpy(labels), reduction="none")
    assert np.allclose(dec.cross_entropy_rows(logits, labels), ref.numpy(), rtol=1e-12)


def test_bf16_storage_rounds_every_stored_activation():
    cfg, codes, betas, emb = _tiny(bf16=True)
    tok = synth.tokens(4, 2, 8, cfg.vocab)
    r16 = dec.forward_row_losses(cfg, emb, tok, codes, betas)
    cfg32 = dec.DecoderConfig(**{**cfg.__dict__, "bf16": False})
    r32 = dec.forward_row_losses(cfg32, emb, tok, codes, betas)
    assert not np.array_equal(r16, r32)
    assert np.allclose(r16, r32, rtol=2e-2)


# --------------------------------------------------------------------------
# Block composition, written independently with torch fp64 library routines
# --------------------------------------------------------------------------
def _torch_rows(cfg, emb, tokens, codes, betas, mutant=None):
    """Per-position next-token cross-entropy of the pre-norm BitNet decoder, composed
    from torch CPU routines (F.embedding, F.rms_norm, rotate-half RoPE, SDPA with K/V
    heads repeated, F.silu, F.cross_entropy); the ternary projections use the oracle's
    activation quantiser (pinned on its own) and an int64 matmul.  Rounding points: the
    activation dtype wherever a tensor is stored (fp32 first, then bf16), the RMSNorm
    output feeding a projection kept at fp32.  `mutant` swaps in one plausible wiring
    mistake, to show the comparison detects it."""
    from oracle import termezo_ref as orc
    f64 = torch.float64
    act = torch.bfloat16 if cfg.bf16 else torch.float32

    def stored(x):
        return x.to(torch.float32).to(act).to(f64)

    def bitlinear(x, c, beta):
        xq, s = orc.act_quant(x.to(torch.float32).numpy())
        acc = torch.from_numpy(xq).to(torch.int64) @ torch.from_numpy(c).to(torch.int64).T
        r = torch.tensor(beta, dtype=torch.float32) / torch.from_numpy(s)
        return (acc.to(torch.float32) * r[:, None]).to(f64)

    B, S = tokens.shape
    d, Hq, Hkv, hd = cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    E = torch.from_numpy(emb).to(f64)
    tok = torch.from_numpy(tokens).to(torch.int64)
    half = hd // 2
    inv = cfg.rope_base ** (-torch.arange(half, dtype=f64) * 2.0 / hd)
    ang = torch.arange(S, dtype=f64)[:, None] * inv[None, :]
    cos = torch.cat([ang.cos(), ang.cos()], -1)           # [S, hd]
    sin = torch.cat([ang.sin(), ang.sin()], -1)

    def rope(x, H):                                         # x [B, S, H*hd]
        x = x.view(B, S, H, hd)
        if mutant == "interleaved_rope":                    # pairs (2i, 2i+1) instead
            x1, x2 = x[..., 0::2], x[..., 1::2]
            a = ang[None, :, None, :]
            y = torch.stack([x1 * a.cos() - x2 * a.sin(), x1 * a.sin() + x2 * a.cos()], -1)
            return y.reshape(B, S, H * hd)
        rot = torch.cat([-x[..., half:], x[..., :half]], -1)
        return (x * cos[None, :, None, :] + rot * sin[None, :, None, :]).reshape(B, S, H * hd)

    def norm(h):
        return F.rms_norm(h, (d,), eps=cfg.norm_eps)

    h = stored(F.embedding(tok, E))                         # [B, S, d]
    for blk in range(cfg.n_blocks):
        c = codes[7 * blk: 7 * blk + 7]
        be = betas[7 * blk: 7 * blk + 7]
        x = norm(h).reshape(B * S, d)
        q = stored(rope(stored(bitlinear(x, c[0], be[0])).view(B, S, -1), Hq))
        k = stored(rope(stored(bitlinear(x, c[1], be[1])).view(B, S, -1), Hkv))
        v = stored(bitlinear(x, c[2], be[2])).view(B, S, -1)
        qh = q.view(B, S, Hq, hd).transpose(1, 2)
        kh = k.view(B, S, Hkv, hd).transpose(1, 2)
        vh = v.view(B, S, Hkv, hd).transpose(1, 2)
        if mutant == "gqa_modulo":                          # query head h reads kv head h % Hkv
            kh = kh.repeat(1, Hq // Hkv, 1, 1)
            vh = vh.repeat(1, Hq // Hkv, 1, 1)
        else:
            kh = kh.repeat_interleave(Hq // Hkv, dim=1)
            vh = vh.repeat_interleave(Hq // Hkv, dim=1)
        a = F.scaled_dot_product_attention(qh, kh, vh, is_causal=(mutant != "no_causal_mask"))
        a = stored(a.transpose(1, 2).reshape(B * S, Hq * hd))
        o = stored(bitlinear(a, c[3], be[3])).view(B, S, d)
        h = stored(h + o)
        x = (h if mutant == "no_mlp_norm" else norm(h)).reshape(B * S, d)
        g = stored(bitlinear(x, c[4], be[4]))
        u = stored(bitlinear(x, c[5], be[5]))
        m = stored(F.silu(g) * u) if mutant != "gate_up_swapped" else stored(F.silu(u) * g)
        dn = stored(bitlinear(m, c[6], be[6])).view(B, S, d)
        h = stored(h + dn)
    xf = stored(norm(h)).reshape(B * S, d)
    logits = xf @ E.T
    labels = torch.zeros(B, S, dtype=torch.int64)
    labels[:, :-1] = tok[:, 1:]
    rows = F.cross_entropy(logits, labels.reshape(-1), reduction="none").view(B, S)
    rows[:, -1] = 0.0
    return rows.numpy()


@pytest.mark.parametrize("bf16", [False, True])
def test_block_composition_matches_independent_torch_composition(bf16):
    """Pins the wiring of the decoder oracle (pre-norm order, residual adds, RoPE pairs,
    GQA head mapping, causal mask, SwiGLU, tied head, rounding points) against a
    composition of library routines; each mutant of that composition, one wiring
    mistake each, must differ from the oracle far beyond the agreement bar."""
    cfg = dec.DecoderConfig(n_blocks=2, d_model=64, n_heads=4, n_kv_heads=2, d_ffn=96,
                            vocab=50, bf16=bf16)
    rng = np.random.default_rng(3)
    codes = [rng.integers(-1, 2, size=s).astype(np.int8) for s in cfg.layer_shapes()]
    betas = [0.05] * len(codes)
    # embedding of std 0.25 (logits of std ~2) so the losses vary strongly from position
    # to position without saturating
    emb = dec.store(synth.activations(21, cfg.vocab, cfg.d_model) * np.float32(0.25), bf16)
    tok = synth.tokens(22, 2, 16, cfg.vocab)
    ref = dec.forward_row_losses(cfg, emb, tok, codes, betas)
    got = _torch_rows(cfg, emb, tok, codes, betas)
    assert np.all(got[:, -1] == 0.0)
    # relative error, on a floor of 1 nat (a position whose label is the current token
    # has a loss near zero with a tied head)
    rel = np.abs(got[:, :-1] - ref[:, :-1]) / np.maximum(np.abs(ref[:, :-1]), 1.0)
    # the same rounding points and integer decisions on both sides: only fp64 summation
    # order differs (observed 1e-15)
    assert rel.max() <= 1e-12, rel.max()
    for mutant in ("interleaved_rope", "gqa_modulo", "no_causal_mask", "no_mlp_norm",
                   "gate_up_swapped"):
        bad = _torch_rows(cfg, emb, tok, codes, betas, mutant=mutant)
        drel = np.abs(bad[:, :-1] - ref[:, :-1]) / np.maximum(np.abs(ref[:, :-1]), 1.0)
        assert drel.max() > 1e-3, mutant
