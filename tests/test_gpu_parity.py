"""GPU parity of the TerMeZO hot path against the CPU oracle, through the C ABI.

Bar: bit-exact mask indices, thresholds, fixed-point sums, ternary codes, int8
activations, scales and int32 accumulators; bit-exact BitLinear outputs and
updated latents (both sides evaluate the same sequence of correctly rounded
fp32 operations); losses within 1e-6 relative (in practice identical).
Inputs are seeded synthetic draws (paper_2609_33548_amd.synth)."""
import numpy as np
import pytest

from paper_2609_33548_amd import synth

pytestmark = pytest.mark.gpu

TINY_DECODER_LAYERS = [(256, 256)] * 4 + [(688, 256), (688, 256), (256, 688)]
TINY_DECODER_LAYERS = TINY_DECODER_LAYERS * 2


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _ctx(shapes, w_all, bf16):
    torch = _torch()
    from paper_2609_33548_amd import termezo
    tensors, off = [], 0
    for o, i in shapes:
        t = torch.from_numpy(np.ascontiguousarray(w_all[off: off + o * i]).reshape(o, i)).cuda()
        tensors.append(t.to(torch.bfloat16) if bf16 else t)
        off += o * i
    return termezo.Context(tensors), tensors


def _latents_host(tensors):
    return np.concatenate([t.float().cpu().numpy().ravel() for t in tensors])


def _setup(orc, shapes, bf16, seed=0):
    sizes = [o * i for o, i in shapes]
    w = synth.latents(seed, sizes, bf16=bf16)
    ref = orc.TerMeZOOracle([orc.Layer(o, i) for o, i in shapes], w, bf16=bf16)
    ctx, tensors = _ctx(shapes, w, bf16)
    return ref, ctx, tensors


def _check_mask(ref, ctx):
    for l in range(len(ref.layers)):
        got = ctx.mask(l)
        assert np.array_equal(got, ref.active[l]), f"layer {l}: mask differs"


def _check_stats(ref, ctx, cur=None):
    for l in range(len(ref.layers)):
        s = ctx.layer_stats(l)
        assert s["S"] == ref.S[l], f"layer {l}: |w| sum"
        assert s["tau"] == ref.tau[l] and s["beta"] == ref.beta[l], f"layer {l}: tau/beta"
        if cur is not None:
            assert s["tau_cur"] == cur[0][l] and s["beta_cur"] == cur[1][l], f"layer {l}: tau'/beta'"


def test_gauss_is_bit_identical_to_oracle(orc):
    torch = _torch()
    from paper_2609_33548_amd import termezo
    rng = np.random.default_rng(0)
    gids = np.concatenate([np.arange(1 << 20), rng.integers(0, 1 << 40, 1 << 20)]).astype(np.int64)
    for seed in (0, 7, (3 << 32) | 5, 2**64 - 1):
        z = termezo.gauss(seed, torch.from_numpy(gids).cuda()).cpu().numpy()
        rz = orc.gauss(seed, gids)
        bad = np.nonzero(z.view(np.uint32) != rz.view(np.uint32))[0]
        assert bad.size == 0, (f"seed {seed}: {bad.size} differ; first gid {gids[bad[0]]} "
                               f"gpu {z[bad[0]]!r} oracle {rz[bad[0]]!r}")


@pytest.mark.parametrize("shapes", [[(256, 256)], TINY_DECODER_LAYERS], ids=["single_layer", "tiny_decoder"])
@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
@pytest.mark.parametrize("rho0,inclusive", [(0.01, False), (0.001, False), (0.01, True),
                                           (1.0, False)])
def test_build_mask_matches_oracle(orc, shapes, bf16, rho0, inclusive):
    print(f"mask shapes={len(shapes)} bf16={bf16} rho0={rho0} incl={inclusive}", flush=True)
    ref, ctx, _ = _setup(orc, shapes, bf16, seed=1)
    k0, xi0 = ctx.build_mask(rho0, 1e-5, inclusive)
    rk0, rxi0 = ref.build_mask(rho0, inclusive)
    assert (k0, xi0) == (rk0, rxi0)
    _check_mask(ref, ctx)
    _check_stats(ref, ctx)
    for l in range(len(shapes)):        # clean codes after the build
        assert np.array_equal(ctx.codes(l), ref.clean_codes(l))


@pytest.mark.parametrize("shapes", [[(256, 256)], TINY_DECODER_LAYERS], ids=["single_layer", "tiny_decoder"])
@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
# 0.002: the guarded path (actives' codes only); 0.9999: fully active tiles after ragged ones
@pytest.mark.parametrize("rho0", [0.002, 0.05, 0.9999, 1.0])
def test_perturb_codes_match_oracle(orc, shapes, bf16, rho0):
    print(f"perturb shapes={len(shapes)} bf16={bf16} rho0={rho0}", flush=True)
    ref, ctx, tensors = _setup(orc, shapes, bf16, seed=2)
    ctx.build_mask(rho0)
    ref.build_mask(rho0)
    before = [t.clone() for t in tensors]
    for seed, eps, sign in [(7, 1e-3, 1), (7, 1e-3, -1), (123456789, 5e-3, 1), (7, 1e-3, 0)]:
        ctx.perturb(seed, eps, sign)
        codes, taus, betas = ref.perturb(seed, eps, sign)
        for l in range(len(shapes)):
            got = ctx.codes(l)
            bad = np.count_nonzero(got != codes[l])
            assert bad == 0, f"layer {l} seed {seed} sign {sign}: {bad} codes differ"
        _check_stats(ref, ctx, (taus, betas))
    for a, b in zip(before, tensors):   # perturbation never writes the latents
        assert a.equal(b)


@pytest.mark.parametrize("M,K,N", [(1, 256, 256), (8, 256, 256), (16, 2560, 2560),
                                   (130, 688, 256), (257, 256, 688), (64, 6912, 2560),
                                   (300, 2560, 640),
                                   # small-M kernel: ragged features, K not a multiple of 64,
                                   # a partial token group, the largest token count, K = 16
                                   (1, 2560, 6912), (17, 688, 100), (128, 6912, 2560),
                                   (3, 16, 48), (100, 256, 200),
                                   # more decode-sized shapes: the largest projection K at 16
                                   # tokens, a long K on few features, K not a multiple of 64,
                                   # features not a multiple of 4
                                   (16, 6912, 2560), (1, 7168, 64), (5, 688, 100), (1, 256, 37),
                                   (2, 7184, 48)])
@pytest.mark.parametrize("xdt,ydt", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32")])
def test_bitlinear_matches_oracle(orc, M, K, N, xdt, ydt):
    torch = _torch()
    print(f"bitlinear M={M} K={K} N={N} x={xdt} y={ydt}", flush=True)
    ref, ctx, _ = _setup(orc, [(N, K)], bf16=False, seed=3)
    ctx.build_mask(0.01)
    ref.build_mask(0.01)
    ctx.perturb(11, 1e-3, 1)
    codes, _, betas = ref.perturb(11, 1e-3, 1)
    x = synth.activations(4, M, K, bf16=(xdt == "bf16"))
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16}
    xd = torch.from_numpy(x).cuda().to(tdt[xdt])
    y = torch.empty((M, N), dtype=tdt[ydt], device="cuda")
    xq = torch.empty((M, K), dtype=torch.int8, device="cuda")
    s = torch.empty(M, dtype=torch.float32, device="cuda")
    acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
    ctx.bitlinear_forward(0, xd, y, xq, s, acc)
    torch.cuda.synchronize()
    rxq, rs = orc.act_quant(x)
    racc, ry = orc.bitlinear(rxq, rs, codes[0], betas[0])
    assert np.array_equal(xq.cpu().numpy(), rxq)
    assert np.array_equal(s.cpu().numpy(), rs)
    assert np.array_equal(acc.cpu().numpy(), racc)
    if ydt == "bf16":
        ry = orc.bf16_round(ry)
    assert np.array_equal(y.float().cpu().numpy(), ry)


@pytest.mark.parametrize("K,N", [(256, 256), (2560, 6912), (6912, 2560), (7168, 64), (256, 37),
                                 (16, 48), (688, 100), (8192, 32),
                                 (8208, 16)])    # beyond the fused kernel's row: two kernels
@pytest.mark.parametrize("xdt,ydt", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32")])
def test_single_token_forward_matches_oracle(orc, K, N, xdt, ydt):
    """One token without inspection outputs: the activation quantisation runs inside the
    contraction kernel (one launch); the output must still be the oracle's bit for bit."""
    torch = _torch()
    print(f"bitlinear M=1 K={K} N={N} x={xdt} y={ydt} (fused)", flush=True)
    ref, ctx, _ = _setup(orc, [(N, K)], bf16=False, seed=5)
    ctx.build_mask(0.01)
    ref.build_mask(0.01)
    ctx.perturb(13, 1e-3, -1)
    codes, _, betas = ref.perturb(13, 1e-3, -1)
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16}
    for seed in (6, 7):
        x = synth.activations(seed, 1, K, bf16=(xdt == "bf16"))
        xd = torch.from_numpy(x).cuda().to(tdt[xdt])
        y = torch.empty((1, N), dtype=tdt[ydt], device="cuda")
        ctx.bitlinear_forward(0, xd, y)
        torch.cuda.synchronize()
        rxq, rs = orc.act_quant(x)
        _, ry = orc.bitlinear(rxq, rs, codes[0], betas[0])
        if ydt == "bf16":
            ry = orc.bf16_round(ry)
        assert np.array_equal(y.float().cpu().numpy(), ry), f"seed {seed}"


@pytest.mark.parametrize("M,K,N", [(2, 256, 256), (16, 2560, 2560), (5, 688, 100), (9, 256, 37),
                                   (3, 16, 48),
                                   (16, 2560, 6912),    # two feature groups per block
                                   (2, 2560, 6912),
                                   (16, 2048, 8200),    # two groups, the last one ragged
                                   (16, 6912, 2560),    # M K above the fused bound: two kernels
                                   (10, 4096, 64),      # the longest fp32 row of the fused kernel
                                   (2, 4112, 48),       # fp32: two kernels; bf16: fused
                                   (9, 4112, 48),       # a long row for more tokens than it holds
                                   (5, 8192, 32),       # the longest bf16 row of the fused kernel
                                   (7, 8208, 16)])      # beyond it: two kernels
@pytest.mark.parametrize("xdt,ydt", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32")])
def test_few_token_forward_matches_oracle(orc, M, K, N, xdt, ydt):
    """Two to sixteen tokens without inspection outputs: every block quantises the token
    rows itself and contracts its features in one launch; the outputs must be the
    oracle's bit for bit, two calls in a row with new activations."""
    torch = _torch()
    print(f"bitlinear M={M} K={K} N={N} x={xdt} y={ydt} (fused, few tokens)", flush=True)
    ref, ctx, _ = _setup(orc, [(N, K)], bf16=False, seed=9)
    ctx.build_mask(0.01)
    ref.build_mask(0.01)
    ctx.perturb(17, 1e-3, 1)
    codes, _, betas = ref.perturb(17, 1e-3, 1)
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16}
    for seed in (21, 22):
        x = synth.activations(seed, M, K, bf16=(xdt == "bf16"))
        xd = torch.from_numpy(x).cuda().to(tdt[xdt])
        y = torch.empty((M, N), dtype=tdt[ydt], device="cuda")
        ctx.bitlinear_forward(0, xd, y)
        torch.cuda.synchronize()
        rxq, rs = orc.act_quant(x)
        _, ry = orc.bitlinear(rxq, rs, codes[0], betas[0])
        if ydt == "bf16":
            ry = orc.bf16_round(ry)
        assert np.array_equal(y.float().cpu().numpy(), ry), f"seed {seed}"


@pytest.mark.parametrize("M,K,N,ydt", [(8192, 2560, 2560, "bf16"),   # 320 tiles: last 64 cut in quarters
                                       (8192, 1024, 2816, "bf16"),   # 352 tiles: last 96 cut in quarters
                                       (8192, 2560, 3840, "bf16"),   # 480 tiles: whole tiles only
                                       (8232, 2560, 2560, "bf16"),   # ragged M on the large-tile path
                                       (8192, 688, 8192, "bf16"),    # K not a multiple of the K step
                                       (4096, 6912, 4352, "bf16"),   # 272 tiles: last 16 cut in quarters
                                       (8192, 2560, 2560, "f32"),    # fp32 outputs, whole and quarter tiles
                                       (512, 256, 512, "f32"),       # 4 tiles: two 128 x 256 blocks per CU
                                       (2048, 2560, 6912, "bf16"),   # 216 tiles: two blocks per CU
                                       (8192, 2560, 6912, "bf16")])  # 864 tiles: two blocks per CU
def test_bitlinear_large_grid_sampled_rows(orc, M, K, N, ydt):
    """Launch sizes that select the large-tile kernels (with and without the
    quarter-tile tail); the oracle evaluates a sample of rows (rows are
    independent), including the first and last and a band of the last quarter
    of rows, where the tail tiles lie.  Two calls in a row with new inputs."""
    torch = _torch()
    print(f"bitlinear large M={M} K={K} N={N} y={ydt}", flush=True)
    ref, ctx, _ = _setup(orc, [(N, K)], bf16=True, seed=8)
    ctx.build_mask(0.001)
    ref.build_mask(0.001)
    ctx.perturb(21, 1e-3, -1)
    codes, _, betas = ref.perturb(21, 1e-3, -1)
    y = torch.empty((M, N), dtype=torch.bfloat16 if ydt == "bf16" else torch.float32, device="cuda")
    acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
    xq = torch.empty((M, K), dtype=torch.int8, device="cuda")
    s = torch.empty(M, dtype=torch.float32, device="cuda")
    rows = np.unique(np.concatenate([[0, 1, 255, 256, M - 256, M - 1],
                                     np.random.default_rng(0).integers(0, M, 40),
                                     np.random.default_rng(1).integers(M - M // 4, M, 16)]))
    for xseed in (9, 10):
        xd = synth.torch_normal(xseed, (M, K), torch.bfloat16, "cuda")
        ctx.bitlinear_forward(0, xd, y, xq, s, acc)
        torch.cuda.synchronize()
        x = xd[torch.from_numpy(rows).cuda()].float().cpu().numpy()
        rxq, rs = orc.act_quant(x)
        racc, ry = orc.bitlinear(rxq, rs, codes[0], betas[0])
        assert np.array_equal(xq.cpu().numpy()[rows], rxq)
        assert np.array_equal(s.cpu().numpy()[rows], rs)
        assert np.array_equal(acc.cpu().numpy()[rows], racc)
        assert np.array_equal(y.float().cpu().numpy()[rows], orc.bf16_round(ry) if ydt == "bf16" else ry)


@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
@pytest.mark.parametrize("rho0", [0.002, 0.01, 0.9999, 1.0])   # 0.002: guarded (actives-only) path
def test_update_and_shrink_match_oracle(orc, bf16, rho0):
    print(f"update bf16={bf16} rho0={rho0}", flush=True)
    ref, ctx, tensors = _setup(orc, TINY_DECODER_LAYERS, bf16, seed=5)
    ctx.build_mask(rho0)
    ref.build_mask(rho0)
    gs = [40.0, -25.0, 60.0, -80.0, 10.0, 120.0]
    for t, g in enumerate(gs):
        seed = t
        ctx.perturb(seed, 1e-3, 1)
        ref.perturb(seed, 1e-3, 1)
        before = _latents_host(tensors)
        prev = np.concatenate([a + ref.offsets[l] for l, a in enumerate(ref.active)])
        k = ctx.update(g, 1e-4)
        rk = ref.update(g, 1e-4)
        after = _latents_host(tensors)
        diff = np.nonzero(after != ref.w)[0]
        assert diff.size == 0, (f"step {t}: {diff.size} latents differ, first gid {diff[0]} "
                                f"gpu {after[diff[0]]!r} oracle {ref.w[diff[0]]!r} "
                                f"before {before[diff[0]]!r} in-mask {np.isin(diff[0], prev)}")
        assert k == rk
        # latents outside the mask of the step never move
        assert np.isin(np.nonzero(after != before)[0], prev).all()
        _check_mask(ref, ctx)
        _check_stats(ref, ctx)


def test_single_layer_trajectory_is_bit_exact(orc):
    """Single BitLinear 256x256, fp32 latents, 8 token rows, MSE to a N(0,1)
    target, rho0 = 1%, eps = 1e-3, lr = 1e-4, seeds s_t = t, 100 steps."""
    torch = _torch()
    shapes = [(256, 256)]
    ref, ctx, tensors = _setup(orc, shapes, bf16=False, seed=0)
    x = synth.activations(100, 8, 256)
    tgt = synth.activations(101, 8, 256)
    xd = torch.from_numpy(x).cuda()
    td = torch.from_numpy(tgt).cuda()
    y = torch.empty((8, 256), device="cuda")
    eps, lr = 1e-3, 1e-4
    assert ctx.build_mask(0.01) == ref.build_mask(0.01)
    xq, s = orc.act_quant(x)
    for t in range(100):
        f = {}
        rf = {}
        for sign in (1, -1):
            ctx.perturb(t, eps, sign)
            ctx.bitlinear_forward(0, xd, y)
            f[sign] = ctx.mse_loss(y, td)
            codes, _, betas = ref.perturb(t, eps, sign)
            _, ry = orc.bitlinear(xq, s, codes[0], betas[0], want_acc=False)
            rf[sign] = orc.mse(ry, tgt)
        assert f == rf, f"step {t}: losses {f} vs {rf}"
        g = orc.projected_grad(f[1], f[-1], eps)
        k = ctx.update(g, lr)
        rk = ref.update(g, lr)
        assert k == rk
    assert np.array_equal(_latents_host(tensors), ref.w)
    _check_mask(ref, ctx)


def test_single_layer_device_side_trajectory_is_bit_exact(orc):
    """The single-layer step as the bench runs it, with nothing on the host: MSE
    losses written to device scalars, g = (F+ - F-)/(2 eps) and the update formed on
    the device (Algorithm 1).  The oracle runs the same 100 steps from its own losses;
    losses, mask sizes and latents agree bit for bit."""
    torch = _torch()
    shapes = [(256, 256)]
    ref, ctx, tensors = _setup(orc, shapes, bf16=False, seed=0)
    x = synth.activations(100, 8, 256)
    tgt = synth.activations(101, 8, 256)
    xd = torch.from_numpy(x).cuda()
    td = torch.from_numpy(tgt).cuda()
    y = torch.empty((8, 256), device="cuda")
    Fd = torch.zeros(2, device="cuda")
    eps, lr = 1e-3, 1e-4
    assert ctx.build_mask(0.01) == ref.build_mask(0.01)
    xq, s = orc.act_quant(x)
    losses = []
    for t in range(100):
        rf = {}
        for j, sign in enumerate((1, -1)):
            ctx.perturb(t, eps, sign)
            ctx.bitlinear_forward(0, xd, y)
            ctx.mse_loss_dev(y, td, Fd[j: j + 1])
            codes, _, betas = ref.perturb(t, eps, sign)
            _, ry = orc.bitlinear(xq, s, codes[0], betas[0], want_acc=False)
            rf[sign] = orc.mse(ry, tgt)
        ctx.update_from_losses(Fd[0:1], Fd[1:2], eps, lr)
        losses.append(Fd.cpu().numpy().copy())
        ref.update(orc.projected_grad(rf[1], rf[-1], eps), lr)
        assert losses[-1].tolist() == [rf[1], rf[-1]], f"step {t}"
        if t % 25 == 0:
            assert ctx.active_count() == ref.k
    assert np.array_equal(_latents_host(tensors), ref.w)
    _check_mask(ref, ctx)


def test_state_and_numeric_errors(orc):
    torch = _torch()
    from paper_2609_33548_amd import termezo as T
    w = torch.from_numpy(synth.latents(9, [64 * 64])).cuda().reshape(64, 64)
    ctx = T.Context([w])
    with pytest.raises(T.TermezoError) as e:
        ctx.perturb(1, 1e-3, 1)
    assert e.value.status == T.ERR_STATE
    with pytest.raises(T.TermezoError) as e:
        ctx.update(1.0, 1e-3)
    assert e.value.status == T.ERR_STATE
    with pytest.raises(T.TermezoError) as e:
        ctx.build_mask(1.5)
    assert e.value.status == T.ERR_INVALID_ARG
    with pytest.raises(T.TermezoError) as e:
        ctx.build_mask(1e-6)           # floor(rho0 * D) == 0
    assert e.value.status == T.ERR_STATE
    ctx.build_mask(0.1)
    with pytest.raises(T.TermezoError) as e:
        ctx.perturb(1, 1e-3, 2)
    assert e.value.status == T.ERR_INVALID_ARG
    ctx.perturb(1, 1e-3, 1)
    ctx.update(1.0, 1e-3)
    x = torch.zeros((4, 64), device="cuda")
    y = torch.empty((4, 64), device="cuda")
    with pytest.raises(T.TermezoError) as e:   # codes invalid after an update
        ctx.bitlinear_forward(0, x, y)
    assert e.value.status == T.ERR_STATE
    w[3, 5] = float("nan")
    with pytest.raises(T.TermezoError) as e:
        ctx.build_mask(0.1)
    assert e.value.status == T.ERR_NUMERIC
    w[3, 5] = 0.0
    ctx.build_mask(0.1)                        # recovers once the latent is fixed
    ctx.close()


@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
@pytest.mark.parametrize("rho0,eps", [(0.003, 1e-3),    # drift far below xi0: actives only
                                      (0.012, 1e-3),    # denser set: code words tile by tile
                                      (0.02, 0.5),      # tile-by-tile and dense fallback
                                      (0.002, 0.5)])    # drift above xi0: dense fallback
def test_guarded_requant_equals_dense_requant(orc, bf16, rho0, eps):
    """The default perturbation (actives' codes only while the threshold-drift
    guard proves every frozen code unchanged, dense otherwise) gives the codes of
    the dense requantisation: three contexts on the same latents (default, forced
    dense, and switching between the two at every perturbation, so a guarded pass
    follows a forced one) against each other and the oracle over five steps
    (perturb +, -, 0, update)."""
    print(f"guarded requant bf16={bf16} rho0={rho0} eps={eps}", flush=True)
    shapes = [(256, 256), (128, 512), (384, 128)]
    ref, ctx, tensors = _setup(orc, shapes, bf16, seed=41)
    _, ctx_d, tensors_d = _setup(orc, shapes, bf16, seed=41)
    _, ctx_a, _ = _setup(orc, shapes, bf16, seed=41)
    ctx_d.set_dense_requant(True)
    ctx.build_mask(rho0)
    ctx_d.build_mask(rho0)
    ctx_a.build_mask(rho0)
    ref.build_mask(rho0)
    n_pert = 0
    for t in range(5):
        for sign in (1, -1, 0):
            ctx.perturb(t, eps, sign)
            ctx_d.perturb(t, eps, sign)
            ctx_a.set_dense_requant(n_pert % 2 == 0)
            ctx_a.perturb(t, eps, sign)
            n_pert += 1
            codes, taus, betas = ref.perturb(t, eps, sign)
            for l in range(len(shapes)):
                got, dense = ctx.codes(l), ctx_d.codes(l)
                assert np.array_equal(dense, codes[l]), f"step {t} sign {sign} layer {l}: dense path"
                bad = np.count_nonzero(got != codes[l])
                assert bad == 0, f"step {t} sign {sign} layer {l}: {bad} codes differ"
                bad = np.count_nonzero(ctx_a.codes(l) != codes[l])
                assert bad == 0, f"step {t} sign {sign} layer {l}: {bad} codes differ (switching)"
        g = 0.5 - 0.3 * t
        ctx.perturb(t, eps, 1)
        ctx_d.perturb(t, eps, 1)
        ctx_a.perturb(t, eps, 1)
        ref.perturb(t, eps, 1)
        k_ref = ref.update(g, 1e-2)
        assert ctx.update(g, 1e-2) == ctx_d.update(g, 1e-2) == ctx_a.update(g, 1e-2) == k_ref
        assert np.array_equal(_latents_host(tensors), ref.w)
        assert np.array_equal(_latents_host(tensors_d), ref.w)
    ctx.close()
    ctx_d.close()
    ctx_a.close()


@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
@pytest.mark.parametrize("rho0", [0.01, 1.0])
def test_update_reads_kept_draws_only_for_their_seed(orc, bf16, rho0):
    """The pair pass keeps its draws z for an update of the same seed over the same
    active list.  An update whose last perturbation had another seed (here a sign-0
    call after the pair) must draw z again; one whose seed matches reads them.  Both
    give the oracle's latents, over steps that shrink the list in between."""
    print(f"kept draws bf16={bf16} rho0={rho0}", flush=True)
    shapes = [(256, 256), (128, 512), (64, 128)]
    ref, ctx, tensors = _setup(orc, shapes, bf16, seed=23)
    assert ctx.build_mask(rho0) == ref.build_mask(rho0)
    steps = [((5, 1), (6, 0)),       # pair of seed 5, then a sign-0 call of seed 6: draw again
             ((7, 1), (7, -1)),      # the pair of seed 7: the kept draws apply
             ((8, -1), (8, 0)),      # sign 0 of the same seed after the pair: still apply
             ((9, 1), (10, 0))]
    for t, calls in enumerate(steps):
        for sd, sign in calls:
            ctx.perturb(sd, 1e-3, sign)
            ref.perturb(sd, 1e-3, sign)
        g = 30.0 - 17.0 * t
        assert ctx.update(g, 1e-2) == ref.update(g, 1e-2)
        assert np.array_equal(_latents_host(tensors), ref.w), f"step {t}: latents"
        _check_mask(ref, ctx)
    ctx.close()


@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
@pytest.mark.parametrize("rho0", [0.01, 1.0])
def test_perturbation_pair_reuse(orc, bf16, rho0):
    """The first call of a (seed, eps) pair also produces the other sign's values;
    the other sign, a repeat of either sign, a pair that starts with -1, a new eps
    for the same seed, sign 0 in between, and the update after the pair all give
    the oracle's codes, thresholds and latents."""
    print(f"pair reuse bf16={bf16} rho0={rho0}", flush=True)
    shapes = [(256, 256), (128, 512), (64, 128)]
    ref, ctx, tensors = _setup(orc, shapes, bf16, seed=17)
    assert ctx.build_mask(rho0) == ref.build_mask(rho0)
    calls = [(3, 1e-3, 1), (3, 1e-3, -1), (3, 1e-3, 1), (3, 1e-3, 1), (3, 2e-3, -1),
             (3, 2e-3, 1), (3, 2e-3, 0), (3, 2e-3, -1), (4, 1e-3, -1), (4, 1e-3, 1)]
    lr = 1e-2
    for step in range(2):
        for sd, eps, sign in calls:
            sd += 10 * step
            ctx.perturb(sd, eps, sign)
            codes, taus, betas = ref.perturb(sd, eps, sign)
            for l in range(len(shapes)):
                assert np.array_equal(ctx.codes(l), codes[l]), f"{(sd, eps, sign)} layer {l}"
                st = ctx.layer_stats(l)
                assert st["tau_cur"] == taus[l] and st["beta_cur"] == betas[l], f"{(sd, eps, sign)}"
        g = 0.7 - step
        assert ctx.update(g, lr) == ref.update(g, lr)
        assert np.array_equal(_latents_host(tensors), ref.w), f"step {step}: latents"
        _check_mask(ref, ctx)
    ctx.close()


@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
def test_degenerate_active_sets(orc, bf16):
    """A single active latent (k0 = 1), then updates large enough that the shrink
    empties the set: with k = 0 a perturbation gives the clean codes of the current
    latents, an update changes nothing, and both sides agree throughout (codes,
    thresholds, latents, masks)."""
    print(f"degenerate sets bf16={bf16}", flush=True)
    shapes = [(64, 128), (32, 256)]
    D = sum(o * i for o, i in shapes)
    ref, ctx, tensors = _setup(orc, shapes, bf16, seed=23)
    assert ctx.build_mask(1.0 / D) == ref.build_mask(1.0 / D)
    assert ref.k == 1
    emptied = False
    for t in range(12):
        for sign in (1, -1):
            ctx.perturb(t, 1e-3, sign)
            codes, taus, betas = ref.perturb(t, 1e-3, sign)
            for l in range(len(shapes)):
                assert np.array_equal(ctx.codes(l), codes[l]), f"step {t} sign {sign} layer {l}"
        g = 50.0 if t % 2 == 0 else -50.0
        assert ctx.update(g, 1e-2) == ref.update(g, 1e-2)
        assert np.array_equal(_latents_host(tensors), ref.w), f"step {t}"
        _check_mask(ref, ctx)
        _check_stats(ref, ctx)
        emptied = emptied or ref.k == 0
    assert emptied, "the set did not empty; the case is not exercised"
    ctx.close()
