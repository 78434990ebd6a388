"""termezo_bitlinear_forward_noalloc against termezo_bitlinear_forward, through the
C ABI: the same projection and inputs must give bit-identical outputs, on two
calls in a row with the second smaller than the first (the fixed scratch keeps the
first call's bytes beyond the second's), for bf16 and fp32 activations, small- and
large-M kernel paths; sizes beyond the fixed scratch are rejected before any work."""
import numpy as np
import pytest

from paper_2609_33548_amd import synth

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


@pytest.mark.parametrize("shape,Ms,dt", [
    ((2560, 2560), (1000, 40), "bf16"),
    ((640, 688), (300, 37), "f32"),
    ((6912, 2560), (2048, 1), "bf16"),
])
def test_noalloc_forward_matches_forward(shape, Ms, dt):
    torch = _torch()
    from paper_2609_33548_amd import termezo as T
    N, K = shape
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    w = torch.from_numpy(synth.latents(5, [N * K], bf16=(dt == "bf16"))).cuda().to(tdt).view(N, K)
    ctx = T.Context([w])
    ctx.build_mask(1e-2)
    ctx.perturb(3, 1e-3, 1)
    for i, M in enumerate(Ms):
        print(f"noalloc forward N={N} K={K} M={M} {dt}", flush=True)
        x = torch.from_numpy(synth.activations(40 + i, M, K)).cuda().to(tdt)
        y_ref = torch.empty((M, N), dtype=tdt, device="cuda")
        y = torch.full((M, N), float("nan"), dtype=tdt, device="cuda")
        ctx.bitlinear_forward(0, x, y_ref)
        ctx.bitlinear_forward_noalloc(0, x, y)
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16 if dt == "bf16" else torch.int32),
                           y_ref.view(torch.int16 if dt == "bf16" else torch.int32)), M
    ctx.close()


def test_noalloc_forward_rejects_sizes_beyond_the_scratch():
    torch = _torch()
    from paper_2609_33548_amd import termezo as T
    N, K = 256, 6912
    w = torch.from_numpy(synth.latents(6, [N * K], bf16=True)).cuda().to(torch.bfloat16).view(N, K)
    ctx = T.Context([w])
    ctx.build_mask(1e-2)
    ctx.perturb(1, 1e-3, 1)
    M = 2425                               # 2425 * 6912 + 9728 + 4 * 2425 bytes > 16 MiB
    x = torch.zeros((M, K), dtype=torch.bfloat16, device="cuda")
    y = torch.zeros((M, N), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(T.TermezoError) as e:
        ctx.bitlinear_forward_noalloc(0, x, y)
    assert e.value.status == T.ERR_INVALID_ARG and "16 MiB" in str(e.value)
    assert bool((y == 0).all())
    ctx.bitlinear_forward_noalloc(0, x[:2424], y[:2424])   # the largest M that fits
    ctx.sync()
    ctx.close()
