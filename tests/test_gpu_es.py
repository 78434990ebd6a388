"""GPU parity of the evolution-strategies update restricted to the mask (appendix
on RL-based fine-tuning: N one-sided perturbations, a reward each, the
reward-weighted sum of the directions) against the CPU oracle, through the C ABI.

Bar: codes of every population member, latents, theta, thresholds and the
shrunk mask bit-exact (both sides standardise the rewards in fp64 in index
order, form a_n = (lr / N) Rt_n in fp32 and run the same fp32 fma chain); the
device-side reward path equals the host path bit for bit."""
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


def _setup(torch, termezo, orc, shapes, bf16, seed, theta_n=0):
    w = synth.latents(seed, [o * i for o, i in shapes], bf16=bf16)
    th = synth.latents(seed + 1, [theta_n], bf16=bf16) if theta_n else None
    ref = orc.TerMeZOOracle([orc.Layer(o, i) for o, i in shapes], w, bf16=bf16, theta=th,
                            theta_bf16=bf16)
    lat, off = [], 0
    for o, i in shapes:
        lat.append(_dev(torch, w[off: off + o * i], bf16, (o, i)))
        off += o * i
    ctx = termezo.Context(lat)
    T = None
    if theta_n:
        T = _dev(torch, th, bf16)
        ctx.theta_register([T])
    return ref, ctx, lat, T


def _host(lat):
    return np.concatenate([x.float().cpu().numpy().ravel() for x in lat])


@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
@pytest.mark.parametrize("N,standardize", [(8, True), (5, False), (30, True)])
def test_es_update_matches_oracle(orc, bf16, N, standardize):
    torch = _torch()
    from paper_2609_33548_amd import termezo
    print(f"ES N={N} standardize={standardize} bf16={bf16}", flush=True)
    shapes = [(128, 256), (64, 512), (256, 128)]
    ref, ctx, lat, T = _setup(torch, termezo, orc, shapes, bf16, 61, theta_n=4001)
    assert ctx.build_mask(0.02) == ref.build_mask(0.02)
    sigma, lr = 1e-3, 2e-2
    rng = np.random.default_rng(7)
    for t in range(3):
        seeds = [1000 * t + n for n in range(N)]
        for n, sd in enumerate(seeds):           # one-sided population members
            ctx.perturb(sd, sigma, 1)
            codes, _, _ = ref.perturb(sd, sigma, 1)
            if n < 3:
                for l in range(len(shapes)):
                    assert np.array_equal(ctx.codes(l), codes[l]), f"step {t} member {n} layer {l}"
        rewards = rng.normal(0.0, 1.0, N).astype(np.float32)
        k_dev = ctx.es_update(seeds, rewards, lr, standardize)
        assert k_dev == ref.es_update(seeds, rewards, lr, standardize)
        assert np.array_equal(_host(lat), ref.w), f"step {t}: latents"
        assert np.array_equal(T.float().cpu().numpy(), ref.theta), f"step {t}: theta"
        for l in range(len(shapes)):
            assert np.array_equal(ctx.mask(l), ref.active[l]), f"step {t} layer {l}: mask"
            st = ctx.layer_stats(l)
            assert st["S"] == ref.S[l] and st["tau"] == ref.tau[l], f"step {t} layer {l}"
    ctx.close()


@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
def test_es_device_rewards_equal_host_rewards(orc, bf16):
    """The rewards read from device memory (no host round trip) give the same
    latents, mask and theta as the host rewards; a negative lr (rewards taken as
    losses) is the ascent on the negated rewards."""
    torch = _torch()
    from paper_2609_33548_amd import termezo
    shapes = [(256, 256), (128, 512)]
    _, ca, la, Ta = _setup(torch, termezo, orc, shapes, bf16, 71, theta_n=999)
    _, cb, lb, Tb = _setup(torch, termezo, orc, shapes, bf16, 71, theta_n=999)
    _, cc, lc, Tc = _setup(torch, termezo, orc, shapes, bf16, 71, theta_n=999)
    for c in (ca, cb, cc):
        c.build_mask(0.01)
    N, lr = 6, 3e-2
    rng = np.random.default_rng(3)
    for t in range(3):
        seeds = [77 * t + n for n in range(N)]
        for c in (ca, cb, cc):
            for sd in seeds:
                c.perturb(sd, 1e-3, 1)
        r = rng.normal(0.5, 2.0, N).astype(np.float32)
        ka = ca.es_update(seeds, r, lr)
        cb.es_update_from_rewards(seeds, torch.from_numpy(r).cuda(), lr)
        cc.es_update_from_rewards(seeds, torch.from_numpy(-r).cuda(), -lr)
        assert cb.active_count() == ka == cc.active_count()
        assert np.array_equal(_host(la), _host(lb)) and np.array_equal(_host(la), _host(lc))
        assert torch.equal(Ta, Tb) and torch.equal(Ta, Tc)
        for l in range(len(shapes)):
            assert np.array_equal(ca.mask(l), cb.mask(l))
    for c in (ca, cb, cc):
        c.close()


def test_es_degenerate_and_error_cases(orc):
    """N = 1 or equal rewards with standardisation: the weights do not move (only
    the shrink runs); a non-finite device reward skips the update and reports
    NUMERIC; host-side argument errors leave the state untouched."""
    torch = _torch()
    from paper_2609_33548_amd import termezo
    shapes = [(128, 256)]
    ref, ctx, lat, _ = _setup(torch, termezo, orc, shapes, True, 81)
    assert ctx.build_mask(0.05) == ref.build_mask(0.05)
    w0 = _host(lat)
    ctx.perturb(1, 1e-3, 1)
    ref.perturb(1, 1e-3, 1)
    assert ctx.es_update([1], [3.0], 1e-1) == ref.es_update([1], [3.0], 1e-1)
    assert np.array_equal(_host(lat), w0)
    for sd in (2, 3, 4):
        ctx.perturb(sd, 1e-3, 1)
        ref.perturb(sd, 1e-3, 1)
    assert ctx.es_update([2, 3, 4], [0.5] * 3, 1e-1) == ref.es_update([2, 3, 4], [0.5] * 3, 1e-1)
    assert np.array_equal(_host(lat), w0)
    ctx.perturb(5, 1e-3, 1)
    with pytest.raises(termezo.TermezoError) as e:
        ctx.es_update([5, 6], [1.0, float("nan")], 1e-1)
    assert e.value.status == termezo.ERR_INVALID_ARG
    with pytest.raises(termezo.TermezoError) as e:
        ctx.es_update(list(range(33)), [1.0] * 33, 1e-1)
    assert e.value.status == termezo.ERR_INVALID_ARG
    ctx.es_update_from_rewards([5, 6], torch.tensor([1.0, float("inf")], device="cuda"), 1e-1)
    with pytest.raises(termezo.TermezoError) as e:
        ctx.sync()
    assert e.value.status == termezo.ERR_NUMERIC
    assert np.array_equal(_host(lat), w0)
    ctx.close()


def test_es_in_compact_mode(orc):
    """ES steps after compaction (caller latents overwritten with NaN): active
    latents, mask and codes equal the oracle's."""
    torch = _torch()
    from paper_2609_33548_amd import termezo
    shapes = [(256, 256), (128, 384)]
    ref, ctx, lat, _ = _setup(torch, termezo, orc, shapes, True, 91)
    assert ctx.build_mask(0.003) == ref.build_mask(0.003)
    ctx.compact()
    for x in lat:
        x.fill_(float("nan"))
    rng = np.random.default_rng(11)
    for t in range(3):
        seeds = [10 * t + n for n in range(4)]
        for sd in seeds:
            ctx.perturb(sd, 1e-3, 1)
            codes, _, _ = ref.perturb(sd, 1e-3, 1)
        for l in range(len(shapes)):
            assert np.array_equal(ctx.codes(l), codes[l]), f"step {t} layer {l}: codes"
        r = rng.normal(0.0, 1.0, 4).astype(np.float32)
        assert ctx.es_update(seeds, r, 1e-3) == ref.es_update(seeds, r, 1e-3)
        for l in range(len(shapes)):
            assert np.array_equal(ctx.mask(l), ref.active[l])
            assert np.array_equal(ctx.active_values(l), ref.layer_w(l)[ref.active[l]])
    ctx.close()
