"""GPU parity of the full-precision parameters theta (Algorithm 1 perturbs and
updates them densely with the masked latents, from the same seed) against the
CPU oracle, through the C ABI.

Bar: the perturbed copies theta +- eps z_theta and the updated theta are
bit-exact (both sides evaluate the same correctly rounded fp32 operations and
the same round-to-nearest-even bf16 conversion); decoder losses evaluated at the
perturbed theta within the decoder bar (1e-3 relative on the batch loss, 5e-3
per position for bf16 activations, 2e-3 for fp32)."""
import numpy as np
import pytest

from paper_2609_33548_amd import synth

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _dev(torch, a, bf16, shape=None):
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    t = t.to(torch.bfloat16) if bf16 else t
    return t.view(*shape) if shape else t


@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
def test_theta_perturb_and_update_are_bit_exact(orc, bf16):
    """Three theta tensors whose ids start at 0, 4 k + 2 and 4 k' + 3 (quads that
    straddle tensors), a 1e-2 mask over two latent layers; per step: +, -, the
    repeated + of the same pair, the clean point, then the update."""
    torch = _torch()
    from paper_2609_33548_amd import termezo
    print(f"theta bf16={bf16}", flush=True)
    shapes = [(64, 256), (96, 128)]
    w = synth.latents(11, [o * i for o, i in shapes], bf16=bf16)
    sizes = [4 * 1000 + 2, 2 * 3001 + 5, 777]
    th = [synth.latents(12 + j, [n], bf16=bf16) for j, n in enumerate(sizes)]
    ref = orc.TerMeZOOracle([orc.Layer(o, i) for o, i in shapes], w, bf16=bf16,
                            theta=np.concatenate(th), theta_bf16=bf16)
    lat, off = [], 0
    for o, i in shapes:
        lat.append(_dev(torch, w[off: off + o * i], bf16, (o, i)))
        off += o * i
    ctx = termezo.Context(lat)
    tdev = [_dev(torch, t, bf16) for t in th]
    ctx.theta_register(tdev)
    ctx.build_mask(0.01)
    ref.build_mask(0.01)
    tid0 = np.concatenate([[0], np.cumsum(sizes)])

    def check(expect, what):
        for j in range(len(sizes)):
            got = ctx.theta_current(j).float().cpu().numpy()
            exp = expect[tid0[j]: tid0[j + 1]]
            bad = np.count_nonzero(got != exp)
            assert bad == 0, f"{what}: tensor {j}: {bad} of {got.size} differ"

    eps, lr = 1e-3, 5e-2
    for t in range(3):
        seed = 1000 + t
        for sign in (1, -1, 1, 0):
            ctx.perturb(seed, eps, sign)
            ref.perturb(seed, eps, sign)
            check(ref.theta_cur, f"step {t} sign {sign}")
        g = 0.37 - 0.2 * t
        ctx.perturb(seed, eps, -1)
        ref.perturb(seed, eps, -1)
        ctx.update(g, lr)
        ref.update(g, lr)
        check(ref.theta, f"step {t} update")
        got = np.concatenate([x.float().cpu().numpy().ravel() for x in tdev])
        assert np.array_equal(got, ref.theta), f"step {t}: caller's theta"
        assert np.array_equal(np.concatenate([x.float().cpu().numpy().ravel() for x in lat]), ref.w)
    ctx.close()


@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
def test_decoder_with_perturbed_theta(orc, bf16):
    """theta = (tied embedding, RMSNorm weights): the loss at w +- eps m z,
    theta +- eps z_theta against the decoder oracle evaluated at the oracle's
    perturbed values; two steps with device-side g, theta and latents
    bit-exact after each update."""
    torch = _torch()
    from oracle import decoder_ref as dec
    from paper_2609_33548_amd import termezo
    print(f"decoder theta bf16={bf16}", flush=True)
    cfg = dec.DecoderConfig(n_blocks=2, d_model=256, n_heads=2, n_kv_heads=1, d_ffn=256, vocab=512,
                            bf16=bf16)
    B, S = 2, 128
    shapes = cfg.layer_shapes()
    w = synth.latents(60, [o * i for o, i in shapes], bf16=bf16)
    emb = synth.latents(61, [cfg.vocab * cfg.d_model], bf16=bf16)
    nw = (1.0 + 0.1 * synth.activations(62, 2 * cfg.n_blocks + 1, cfg.d_model)).astype(np.float32)
    if bf16:
        nw = orc.bf16_round(nw)
    nw = nw.ravel()
    ref = orc.TerMeZOOracle([orc.Layer(o, i) for o, i in shapes], w, bf16=bf16,
                            theta=np.concatenate([emb, nw]), theta_bf16=bf16)
    lat, off = [], 0
    for o, i in shapes:
        lat.append(_dev(torch, w[off: off + o * i], bf16, (o, i)))
        off += o * i
    ctx = termezo.Context(lat)
    E = _dev(torch, emb, bf16, (cfg.vocab, cfg.d_model))
    NW = _dev(torch, nw, bf16, (2 * cfg.n_blocks + 1, cfg.d_model))
    ctx.theta_register([E, NW])
    model = termezo.Model(ctx, cfg.n_blocks, cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.d_ffn,
                          cfg.vocab, E)
    model.set_norm_weights(NW)
    tok = synth.tokens(63, B, S, cfg.vocab)
    tokd = torch.from_numpy(tok).cuda()
    ctx.build_mask(0.01)
    ref.build_mask(0.01)
    rows = torch.empty(B * S, device="cuda")
    Fd = torch.zeros(2, device="cuda")
    eps, lr = 1e-3, 1e-2
    nE = cfg.vocab * cfg.d_model
    rtol = 5e-3 if bf16 else 2e-3
    for t in range(2):
        F = {}
        for j, sign in enumerate((1, -1)):
            ctx.perturb(t, eps, sign)
            F[sign] = model.loss(tokd, loss_dev=Fd[j: j + 1], row_loss_dev=rows)
            codes, _, betas = ref.perturb(t, eps, sign)
            emb_p = ref.theta_cur[:nE].reshape(cfg.vocab, cfg.d_model)
            rr = dec.forward_row_losses(cfg, emb_p, tok, codes, betas, norm_w=ref.theta_cur[nE:])
            rl = dec.mean_loss(rr)
            assert abs(F[sign] - rl) <= 1e-3 * abs(rl), (t, sign, F[sign], rl)
            got = rows.cpu().numpy().reshape(B, S)[:, :-1]
            rel = np.abs(got - rr[:, :-1]) / np.abs(rr[:, :-1])
            assert rel.max() <= rtol, f"step {t} sign {sign}: max rel {rel.max()}"
        ctx.update_from_losses(Fd[0:1], Fd[1:2], eps, lr)
        g = orc.projected_grad(F[1], F[-1], eps)
        ref.update(g, lr)
        got = np.concatenate([E.float().cpu().numpy().ravel(), NW.float().cpu().numpy().ravel()])
        assert np.array_equal(got, ref.theta), f"step {t}: theta after the update"
        assert np.array_equal(np.concatenate([x.float().cpu().numpy().ravel() for x in lat]), ref.w)
    model.close()
    ctx.close()
