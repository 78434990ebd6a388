"""Helpers of the full-size parity tests: the latent tensors live on the GPU
(seeded device draws, as the bench makes them) and the oracle works layer by
layer on host copies, so no oracle call ever holds more than one layer's
latents at full width."""
import numpy as np

from paper_2609_33548_amd import synth

DELTA = 1e-5


def host(view):
    return view.float().cpu().numpy().ravel()


def build(torch, termezo, shapes, seed=1234):
    """The bench's latent tensor (one allocation, one view per projection) and a context."""
    D = sum(o * i for o, i in shapes)
    lat = synth.torch_latents(seed, D, torch.bfloat16, "cuda")
    views, offs, off = [], [], 0
    for o, i in shapes:
        views.append(lat[off: off + o * i].view(o, i))
        offs.append(off)
        off += o * i
    return {"ctx": termezo.Context(views), "lat": lat, "views": views, "offs": offs, "D": D,
            "shapes": shapes}


def oracle_mask(full, orc, rho, xi0):
    """The exact-k mask xi0 defines, from the oracle's thresholds and distances of
    every layer: everything below xi0, then the ties at xi0 in id order up to k0.
    Returns k0, the counts below / at or below xi0, every layer's tau and actives."""
    k0 = int(np.floor(np.float64(np.float32(rho)) * np.float64(full["D"])))
    less, leq, ties, taus, acts_lt = 0, 0, [], [], []
    for l, v in enumerate(full["views"]):
        if l % 30 == 0:
            print(f"  oracle distances, layer {l}", flush=True)
        w = host(v)
        tau, _ = orc.threshold(orc.layer_abs_sum(w), w.size, DELTA)
        d = orc.distance(w, tau)
        lt = np.nonzero(d < np.float32(xi0))[0]
        eq = np.nonzero(d == np.float32(xi0))[0]
        less += lt.size
        leq += lt.size + eq.size
        taus.append(tau)
        acts_lt.append(lt)
        ties.append(eq)
    quota = k0 - less
    acts = []
    for l in range(len(full["shapes"])):
        take = ties[l][: max(0, min(quota, ties[l].size))]
        quota -= take.size
        acts.append(np.sort(np.concatenate([acts_lt[l], take])).astype(np.int64))
    return k0, less, leq, taus, acts


def oracle_codes(full, orc, seed, eps, sign):
    """Every layer's codes and beta' at w + sign eps m (.) z(seed), by the oracle."""
    codes, betas = [], []
    for l, v in enumerate(full["views"]):
        if l % 30 == 0:
            print(f"  oracle codes, layer {l}", flush=True)
        w = host(v)
        wp = orc.perturbed_layer_values(w, full["acts"][l], full["offs"][l], seed, eps, sign)
        tau, beta = orc.threshold(orc.layer_abs_sum(wp), w.size, DELTA)
        codes.append(orc.quantize(wp, tau).reshape(full["shapes"][l]))
        betas.append(beta)
    return codes, betas


def decoder_config(dec, C):
    return dec.DecoderConfig(n_blocks=C["n_blocks"], d_model=C["d_model"], n_heads=C["n_heads"],
                             n_kv_heads=C["n_kv_heads"], d_ffn=C["d_ffn"], vocab=C["vocab"],
                             bf16=True)


def compare_losses(got_rows, ref_rows, got_batch, n_seq, what, pos_bar, mean_bar):
    """got_rows: the device's per-position losses [B, S] of the whole batch; ref_rows:
    the oracle's for the first n_seq sequences; got_batch: the device's batch loss F
    (the scalar the step consumes).  Checks that F is the mean of the device's own
    labelled positions, then the device against the oracle per position and on the
    mean over the n_seq sequences."""
    B, S = got_rows.shape
    assert np.all(got_rows[:, -1] == 0.0) and np.all(ref_rows[:, -1] == 0.0)
    own = float(np.float32(got_rows[:, :-1].astype(np.float64).sum() / (B * (S - 1))))
    assert abs(got_batch - own) <= 2e-7 * abs(own), (got_batch, own)
    g = got_rows[:n_seq, :-1].astype(np.float64)
    r = ref_rows[:, :-1].astype(np.float64)
    rel = np.abs(g - r) / np.abs(r)
    mean_rel = abs(g.mean() - r.mean()) / abs(r.mean())
    print(f"{what}: per-position max rel {rel.max():.2e} median {np.median(rel):.2e}; mean over "
          f"{n_seq} sequences rel {mean_rel:.2e} (device {g.mean():.6f}, oracle {r.mean():.6f}); "
          f"device batch F {got_batch:.6f}", flush=True)
    assert mean_rel <= mean_bar
    assert rel.max() <= pos_bar
    return g.mean(), r.mean()
