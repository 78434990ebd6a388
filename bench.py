#!/usr/bin/env python3
"""TerMeZO zeroth-order steps per second at the BitNet b1.58 2B shape, one MI355X.

One step (Algorithm 1 with K = 1, theta frozen) on synthetic inputs:
  perturb(+eps) -> decoder loss F+ -> perturb(-eps) -> decoder loss F- ->
  g = (F+ - F-)/(2 eps) on the device -> masked update + shrink.
Workload: 30 blocks, d = 2560, 20 query / 5 KV heads (head dim 128), SwiGLU FFN
6912, vocab 128256, sequence 512, batch 16 (8192 tokens per forward),
2,084,044,800 bf16 latent weights ~ N(0, 0.02^2), bf16 tied embedding
~ N(0, 0.02^2), uniform random token ids, mask ratio 1e-3, eps = 1e-3.
The mask is built once before the timed steps (its time is reported apart).

Prints one JSON line with the steps/s, the roofline of the dominant kernel
(the int8 BitLinear GEMM, timed with HIP events on the library's stream) and a
CPU baseline (the oracle on a bounded sample of the same step, host cores).
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

CONFIGS = {
    # headline workload: BitNet b1.58 2B shape, bf16 latents and activations
    "2b": dict(n_blocks=30, d_model=2560, n_heads=20, n_kv_heads=5, d_ffn=6912, vocab=128256,
               seq=512, batch=16, rho=1e-3, lr=1e-5),
    # 700M-class shape, 16 heads of 96 (MHA), bf16
    "700m": dict(n_blocks=24, d_model=1536, n_heads=16, n_kv_heads=16, d_ffn=4096, vocab=32000,
                 seq=512, batch=8, rho=1e-3, lr=1e-5),
    # tiny decoder, fp32 latents and activations
    "tiny": dict(n_blocks=2, d_model=256, n_heads=4, n_kv_heads=4, d_ffn=688, vocab=1024,
                 seq=64, batch=4, rho=1e-2, lr=1e-4, fp32=True),
}
# single-layer workload: one 256 x 256 BitLinear (fp32 latents), 8 token rows, MSE to a target
LAYER = dict(d_out=256, d_in=256, tokens=8, rho=1e-2, eps=1e-3, lr=1e-4)
PEAK_INT8_TOPS = 5000.0          # MI355X dense int8 MFMA, TOP/s
# HBM traffic of the GEMM launches measured with rocprofv3 counters (FETCH_SIZE,
# WRITE_SIZE), valid only for the kernel source it was measured on.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "bitlinear_gemm_traffic_2b_step.txt")
# the GEMM kernels and every header they include (tile order, direct-to-LDS loads, unpacking)
GEMM_SOURCES = [os.path.join(ROOT, "paper_2609_33548_amd", "csrc", f)
                for f in ("tmz_bitlinear.hip", "tmz_device.h", "tmz_internal.h")]
METRIC = "ZO steps/sec at 2B BitNet shape; perturb+requant GB/s; BitLinear int8 TOPS"


def layer_shapes(c):
    hd = c["d_model"] // c["n_heads"]
    d, F = c["d_model"], c["d_ffn"]
    q, kv = c["n_heads"] * hd, c["n_kv_heads"] * hd
    return [(q, d), (kv, d), (kv, d), (d, q), (F, d), (F, d), (d, F)] * c["n_blocks"]


def gemm_algorithmic_bytes(c):
    """HBM bytes a BitLinear GEMM launch must move, averaged over the four
    launches of a block: int8 activations + 2-bit codes read once, bf16 output
    written (read too for the residual projections o and down)."""
    M = c["batch"] * c["seq"]
    hd = c["d_model"] // c["n_heads"]
    d, F = c["d_model"], c["d_ffn"]
    dq, dkv = c["n_heads"] * hd, c["n_kv_heads"] * hd
    # (K, N code rows, output columns, output passes); gate|up writes only the SwiGLU product
    launches = [(d, dq + 2 * dkv, dq + 2 * dkv, 1), (dq, d, d, 2), (d, 2 * F, F, 1), (F, d, d, 2)]
    total = sum(M * K + N * K // 4 + passes * 2 * M * No for K, N, No, passes in launches)
    return total / len(launches)


def gemm_source_digest():
    """SHA-256 over the GEMM's source files, concatenated in a fixed order."""
    import hashlib
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()


def measured_traffic():
    """Counter-measured HBM bytes per GEMM launch, or None when the counters
    were taken on another version of the kernel source."""
    try:
        kv = dict(line.split(":", 1) for line in open(TRAFFIC_FILE) if ":" in line)
    except OSError:
        return None
    if kv.get("source_sha256", "").strip() != gemm_source_digest():
        return None
    return float(kv["fetch_bytes_per_launch"]) + float(kv["write_bytes_per_launch"])


def cpu_baseline(c, rho, seed=0, theta_n=0, K=1, es=0):
    """The oracle, as it stands, on a bounded sample of the same step; the
    full-step time is extrapolated by operation counts (stated in 'sample')."""
    import numpy as np
    from threadpoolctl import threadpool_info
    from oracle import decoder_ref as dec
    from oracle import termezo_ref as orc
    from paper_2609_33548_amd import synth

    shapes = layer_shapes(c)
    D = sum(o * i for o, i in shapes)
    # (1) perturb / requant / update / shrink on the seven projections of one block
    smp = shapes[:7]
    nsmp = sum(o * i for o, i in smp)
    w = synth.latents(seed, [o * i for o, i in smp], bf16=True)
    st = orc.TerMeZOOracle([orc.Layer(o, i) for o, i in smp], w, bf16=True)
    st.build_mask(rho)
    t0 = time.perf_counter()
    st.perturb(1, 1e-3, 1)
    st.perturb(1, 1e-3, -1)
    st.update(1.0, 1e-4)
    t_latent = (time.perf_counter() - t0) * D / nsmp
    # (2) one decoder block on n_seq sequences (vocab shrunk so the head is negligible)
    n_seq = 16
    cfg1 = dec.DecoderConfig(n_blocks=1, d_model=c["d_model"], n_heads=c["n_heads"],
                             n_kv_heads=c["n_kv_heads"], d_ffn=c["d_ffn"], vocab=64, bf16=True)
    rng = np.random.default_rng(seed)
    codes = [rng.integers(-1, 2, size=s).astype(np.int8) for s in cfg1.layer_shapes()]
    betas = [0.016] * 7
    emb = synth.latents(seed + 1, [64 * c["d_model"]], bf16=True).reshape(64, c["d_model"])
    tok = synth.tokens(seed + 2, n_seq, c["seq"], 64)
    t0 = time.perf_counter()
    dec.forward_row_losses(cfg1, emb, tok, codes, betas)
    t_block = (time.perf_counter() - t0) / n_seq
    # (3) LM head + cross-entropy for n_pos positions over the full vocabulary
    n_pos = 2048
    E = synth.latents(seed + 3, [c["vocab"] * c["d_model"]], bf16=True).reshape(c["vocab"], c["d_model"])
    x = synth.activations(seed + 4, n_pos, c["d_model"], bf16=True)
    t0 = time.perf_counter()
    logits = x.astype(np.float64) @ E.astype(np.float64).T
    dec.cross_entropy_rows(logits, np.zeros(n_pos, np.int64))
    t_head = time.perf_counter() - t0
    # (4) theta: perturbation at both signs and the update on a sample of ids
    t_theta, n_th = 0.0, 1 << 20
    if theta_n:
        th = synth.latents(seed + 5, [n_th], bf16=True)
        t0 = time.perf_counter()
        orc.theta_perturbed(th, 0, 1, 1e-3, 1, True)
        orc.theta_perturbed(th, 0, 1, 1e-3, -1, True)
        orc.theta_updated(th, 0, 1, 1e-4, 1.0, True)
        t_theta = (time.perf_counter() - t0) * theta_n / n_th
    ntok = c["batch"] * c["seq"]
    t_fwd = c["n_blocks"] * c["batch"] * t_block + (ntok / n_pos) * t_head
    # K directions: K perturbation pairs and 2K forwards; the update regenerates K directions
    t_step = K * (2 * t_fwd + t_latent + t_theta)
    if es:     # ES: es one-sided members, one forward and one perturbation each
        t_step = es * (t_fwd + 0.5 * (t_latent + t_theta))
    wall = t_latent * nsmp / D + t_block * n_seq + t_head + t_theta * n_th / max(theta_n, 1)
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {
        "value": 1.0 / t_step, "unit": "steps/s", "cores": int(threads), "kind": "oracle",
        "host": host_cpu(),
        "sample": (f"oracle perturb(+/-)+update+shrink on one block's 7 projections ({nsmp} bf16 "
                   f"latents) scaled to {D}; 1 decoder block x {n_seq} sequences of {c['seq']} tokens "
                   f"scaled x{c['n_blocks']} blocks x{c['batch'] / n_seq:g}; LM head+CE on {n_pos} "
                   f"positions scaled x{ntok // n_pos}; two forwards per step"
                   + (f"; theta perturb(+/-)+update on {n_th} ids scaled to {theta_n}" if theta_n else "")
                   + (f"; all of it x{K} directions" if K > 1 and not es else "")
                   + (f"; ES: {es} members x (one forward + half the perturb/update sample)"
                      if es else "")
                   + f"; sample wall {wall:.1f}s"),
        "extrapolated_step_s": t_step,
    }

def cpu_baseline_layer(n_steps=200, seed=0):
    """The oracle's full single-layer step (perturb +/-, BitLinear, MSE, update), timed."""
    import numpy as np
    from oracle import termezo_ref as orc
    from paper_2609_33548_amd import synth
    w = synth.latents(seed, [LAYER["d_out"] * LAYER["d_in"]])
    st = orc.TerMeZOOracle([orc.Layer(LAYER["d_out"], LAYER["d_in"])], w)
    x = synth.activations(100, LAYER["tokens"], LAYER["d_in"])
    tgt = synth.activations(101, LAYER["tokens"], LAYER["d_out"])
    st.build_mask(LAYER["rho"])
    xq, s = orc.act_quant(x)
    t0 = time.perf_counter()
    for t in range(n_steps):
        f = {}
        for sign in (1, -1):
            codes, _, betas = st.perturb(t, LAYER["eps"], sign)
            _, y = orc.bitlinear(xq, s, codes[0], betas[0], want_acc=False)
            f[sign] = orc.mse(y, tgt)
        st.update(orc.projected_grad(f[1], f[-1], LAYER["eps"]), LAYER["lr"])
    dt = (time.perf_counter() - t0) / n_steps
    return {"value": 1.0 / dt, "unit": "steps/s", "cores": 1, "kind": "oracle", "host": host_cpu(),
            "sample": f"{n_steps} full oracle steps of the same workload (single thread, C + numpy)"}


def cpu_baseline_full(c, rho, n_steps=8, seed=0, theta=False):
    """The oracle's full decoder step (perturb +/-, two forwards, update) on the same
    workload, for configurations small enough to run whole."""
    import numpy as np
    from threadpoolctl import threadpool_info
    from oracle import decoder_ref as dec
    from oracle import termezo_ref as orc
    from paper_2609_33548_amd import synth
    bf = not c.get("fp32", False)
    cfg = dec.DecoderConfig(n_blocks=c["n_blocks"], d_model=c["d_model"], n_heads=c["n_heads"],
                            n_kv_heads=c["n_kv_heads"], d_ffn=c["d_ffn"], vocab=c["vocab"], bf16=bf)
    shapes = cfg.layer_shapes()
    w = synth.latents(seed, [o * i for o, i in shapes], bf16=bf)
    emb = synth.latents(seed + 1, [c["vocab"] * c["d_model"]], bf16=bf).reshape(c["vocab"], c["d_model"])
    nE = emb.size
    nw = np.ones((2 * c["n_blocks"] + 1) * c["d_model"], np.float32)
    st = orc.TerMeZOOracle([orc.Layer(o, i) for o, i in shapes], w, bf16=bf,
                           theta=np.concatenate([emb.ravel(), nw]) if theta else None, theta_bf16=bf)
    tok = synth.tokens(seed + 2, c["batch"], c["seq"], c["vocab"])
    st.build_mask(rho)
    t0 = time.perf_counter()
    for t in range(n_steps):
        f = {}
        for sign in (1, -1):
            codes, _, betas = st.perturb(t, 1e-3, sign)
            e, n = ((st.theta_cur[:nE].reshape(emb.shape), st.theta_cur[nE:]) if theta else (emb, None))
            f[sign] = dec.mean_loss(dec.forward_row_losses(cfg, e, tok, codes, betas, norm_w=n))
        st.update(orc.projected_grad(f[1], f[-1], 1e-3), c["lr"])
    dt = (time.perf_counter() - t0) / n_steps
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"value": 1.0 / dt, "unit": "steps/s", "cores": int(threads), "kind": "oracle",
            "host": host_cpu(),
            "sample": f"{n_steps} full oracle steps of the same workload"}


def run_layer(args, torch, termezo, synth, dev):
    """Single-layer workload: one BitLinear 256 x 256 with fp32 latents, 8 token rows, MSE to a
    N(0, 1) target, mask ratio 1e-2; a step is perturb +/-, two forwards with the MSE
    read back, g on the host and the masked update."""
    import numpy as np
    w = synth.torch_latents(0, LAYER["d_out"] * LAYER["d_in"], torch.float32, dev).view(LAYER["d_out"], LAYER["d_in"])
    x = torch.from_numpy(synth.activations(100, LAYER["tokens"], LAYER["d_in"])).to(dev)
    tgt = torch.from_numpy(synth.activations(101, LAYER["tokens"], LAYER["d_out"])).to(dev)
    y = torch.empty((LAYER["tokens"], LAYER["d_out"]), device=dev)
    ctx = termezo.Context([w])
    k0, _ = ctx.build_mask(LAYER["rho"])
    eps32, two = np.float32(LAYER["eps"]), np.float32(2.0)

    def step(t):
        f = {}
        for sign in (1, -1):
            ctx.perturb(t, LAYER["eps"], sign)
            ctx.bitlinear_forward(0, x, y)
            f[sign] = np.float32(ctx.mse_loss(y, tgt))
        g = np.float32((f[1] - f[-1]) / (two * eps32))      # projected gradient, fp32
        ctx.update(float(g), LAYER["lr"], want_k=False)

    for t in range(args.warmup):
        step(t)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(args.warmup, args.warmup + args.steps):
        step(t)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    cpu = None if args.no_cpu_baseline else cpu_baseline_layer()
    out = {"metric": "ZO steps/sec, single BitLinear with MSE loss", "value": 1000.0 / ms,
           "unit": "steps/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": "int8xternary+f32", "data": "synthetic",
           "config": {"workload": "termezo_zo_step_bitlinear_256x256_mse", **LAYER, "k0": k0,
                      "parallelism": "single_gpu"},
           "roofline": None,
           "note": "launch-latency bound (two host read-backs of the loss per step); "
                   "wall-clock over the timed steps",
           "cpu_baseline": cpu}
    print(json.dumps(out), flush=True)
    ctx.close()


# ---------------------------------------------------------------------------
# Kernel sweeps (--sweep): the perturb/requant and update kernels over a
# 2.4e9-latent tensor at several mask ratios, and the BitLinear forward over
# small and large token counts.  Each point prints one JSON line.
# ---------------------------------------------------------------------------
HBM_PEAK_GBS = 8000.0


def host_cpu():
    """Model name of the host CPU and the logical CPUs this process may use."""
    name = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    name = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return {"model": name, "logical_cpus": n}
SWEEP_LAYER = (6912, 2560)           # 136 layers of this shape: 2,406,481,920 latents
SWEEP_LAYERS = 136
SWEEP_RATIOS = (1e-4, 1e-3, 1e-2, 1.0)
SWEEP_GEMM_KN = ((2560, 2560), (2560, 6912), (6912, 2560))
SWEEP_GEMM_M = (1, 16, 128, 2048, 8192)


def _emit(rec):
    print(json.dumps(rec), flush=True)


def cpu_latent_sweep(ratio, seed=0):
    """Oracle perturb(+)/update(+shrink) on one sweep layer; seconds per call."""
    from oracle import termezo_ref as orc
    from paper_2609_33548_amd import synth
    o, i = SWEEP_LAYER
    w = synth.latents(seed, [o * i], bf16=True)
    st = orc.TerMeZOOracle([orc.Layer(o, i)], w, bf16=True)
    st.build_mask(ratio)
    t0 = time.perf_counter()
    st.perturb(1, 1e-3, 1)
    t_p = time.perf_counter() - t0
    t0 = time.perf_counter()
    st.update(1.0, 1e-5)
    t_u = time.perf_counter() - t0
    return t_p, t_u


def sweep_latent(torch, termezo, synth, dev, cpu):
    o, i = SWEEP_LAYER
    D = SWEEP_LAYERS * o * i
    lat = synth.torch_latents(4321, D, torch.bfloat16, dev)
    layers = [lat[l * o * i:(l + 1) * o * i].view(o, i) for l in range(SWEEP_LAYERS)]
    torch.cuda.synchronize()
    ctx = termezo.Context(layers)
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 10
    for r in SWEEP_RATIOS:
        k0, _ = ctx.build_mask(r)
        ctx.perturb(0, 1e-3, 1)
        ctx.update(1.0, 1e-5, want_k=False)
        ctx.perturb(1, 1e-3, 1)          # warm
        k = ctx.active_count()

        def time_perturb(dense):
            # pairs as in a step: (s, +eps) then (s, -eps); the second call of a pair
            # reuses the values the first one wrote
            ctx.set_dense_requant(dense)
            ctx.perturb(99, 1e-3, 1)
            torch.cuda.synchronize()
            ev0.record(stream)
            for t in range(reps):
                ctx.perturb(100 + t // 2, 1e-3, 1 if t % 2 == 0 else -1)
            ev1.record(stream)
            torch.cuda.synchronize()
            return ev0.elapsed_time(ev1) / reps * 1e-3
        t_p = time_perturb(True)         # every latent re-quantised (the dense stream)
        t_g = time_perturb(False)        # default: actives' codes only while the guard holds
        up = 0.0
        for t in range(reps):
            ctx.perturb(200 + t, 1e-3, 1)
            ev0.record(stream)
            ctx.update(1.0, 1e-5, want_k=False)
            ev1.record(stream)
            torch.cuda.synchronize()
            up += ev0.elapsed_time(ev1) * 1e-3
        t_u = up / reps
        k_after = ctx.active_count()
        b_p = D * (2 + 0.25) + k * (4 + 2)
        b_u = 16 * k
        cp = cu = None
        if cpu:
            c_p, c_u = cpu_latent_sweep(r)
            cp = {"value": (o * i * 2.25 + (k / SWEEP_LAYERS) * 6) / c_p / 1e9, "unit": "GB/s",
                  "kind": "oracle", "sample": f"one {o}x{i} layer, perturb(+), same ratio"}
            cu = {"value": c_u * SWEEP_LAYERS * 1e6, "unit": "us (scaled x136)", "kind": "oracle",
                  "sample": f"one {o}x{i} layer, update+shrink, same ratio"}
        _emit({"sweep": "perturb_requant", "latents": D, "ratio": r, "k": k, "ms": t_p * 1e3,
               "algorithmic_bytes": b_p, "GB/s": b_p / t_p / 1e9,
               "frac_hbm": b_p / t_p / 1e9 / HBM_PEAK_GBS,
               "protocol": "dense requantisation of every latent (termezo_set_dense_requant); "
                           "mean over 5 (+eps, -eps) pairs of one seed each",
               "cpu_baseline": cp})
        # default path: the same codes; only the actives' codes are rewritten while the
        # threshold-drift guard holds (per active: 4 B index + 2 B latent read, 4 B w' written,
        # index and w' read again, the code word read and, where the code changes, written)
        # (above 1/256 active: the code words of the tiles with actives read and written,
        # 0.5 B per weight, plus 4 B index + 4 B w' + 6 B for the delta per active)
        b_g = k * 26 if k * 256 <= D else D * 0.5 + k * 14
        _emit({"sweep": "perturb_guarded", "latents": D, "ratio": r, "k": k, "ms": t_g * 1e3,
               "algorithmic_bytes": b_g, "GB/s": b_g / t_g / 1e9,
               "frac_hbm": b_g / t_g / 1e9 / HBM_PEAK_GBS,
               "speedup_vs_dense": t_p / t_g,
               "protocol": "default termezo_perturb (guarded: dense where the guard fails, "
                           "code words tile by tile when k > D/256); mean over 5 (+eps, -eps) pairs"})
        _emit({"sweep": "update", "latents": D, "ratio": r, "k": k, "k_after": k_after,
               "us": t_u * 1e6, "algorithmic_bytes": b_u, "GB/s": b_u / t_u / 1e9,
               "frac_hbm": b_u / t_u / 1e9 / HBM_PEAK_GBS, "cpu_baseline": cu})
    ctx.close()
    # memory-optimal storage: a fresh context per ratio (the compact form is kept until the
    # context ends); the actives live contiguously in list order
    for r in SWEEP_RATIOS:
        cc = termezo.Context(layers)
        k0, _ = cc.build_mask(r)
        cc.compact()
        lib_b, _ = cc.memory_footprint()
        cc.perturb(0, 1e-3, 1)
        cc.update(1.0, 1e-5, want_k=False)
        cc.perturb(1, 1e-3, 1)
        torch.cuda.synchronize()
        k = cc.active_count()
        ev0.record(stream)
        for t in range(reps):
            cc.perturb(100 + t // 2, 1e-3, 1 if t % 2 == 0 else -1)
        ev1.record(stream)
        torch.cuda.synchronize()
        t_c = ev0.elapsed_time(ev1) / reps * 1e-3
        up = 0.0
        for t in range(reps):
            cc.perturb(200 + t, 1e-3, 1)
            ev0.record(stream)
            cc.update(1.0, 1e-5, want_k=False)
            ev1.record(stream)
            torch.cuda.synchronize()
            up += ev0.elapsed_time(ev1) * 1e-3
        t_uc = up / reps
        k_after = cc.active_count()
        cc.sync()
        cc.close()
        b_g = k * 26 if k * 256 <= D else D * 0.5 + k * 14
        b_u = 16 * k
        _emit({"sweep": "perturb_compact", "latents": D, "ratio": r, "k": k, "ms": t_c * 1e3,
               "algorithmic_bytes": b_g, "GB/s": b_g / t_c / 1e9,
               "frac_hbm": b_g / t_c / 1e9 / HBM_PEAK_GBS, "library_bytes": lib_b,
               "protocol": "termezo_compact after the mask build; actives' codes only; mean over "
                           "5 (+eps, -eps) pairs"})
        _emit({"sweep": "update_compact", "latents": D, "ratio": r, "k": k, "k_after": k_after,
               "us": t_uc * 1e6, "algorithmic_bytes": b_u, "GB/s": b_u / t_uc / 1e9,
               "frac_hbm": b_u / t_uc / 1e9 / HBM_PEAK_GBS})
    del lat, layers
    torch.cuda.empty_cache()


def cpu_bitlinear(M, K, N, seed=0):
    """Oracle BitLinear (activation quantisation + exact integer product) on at
    most 16 rows; seconds for the full M by row scaling."""
    import numpy as np
    from oracle import termezo_ref as orc
    from paper_2609_33548_amd import synth
    m = min(M, 16)
    rng = np.random.default_rng(seed)
    codes = rng.integers(-1, 2, size=(N, K)).astype(np.int8)
    x = synth.activations(seed, m, K, bf16=True)
    t0 = time.perf_counter()
    xq, s = orc.act_quant(x)
    orc.bitlinear(xq, s, codes, 0.016)
    return (time.perf_counter() - t0) * M / m


def vendor_int8_gemm(torch, dev, M, K, N):
    """Context only, not part of the path: the vendor library's dense int8 GEMM
    (hipBLASLt through torch._int_mm) on int8 operands of the same shape, the
    weights as a dense int8 ternary matrix (one byte per weight, no unpacking),
    timed the same way (10 back-to-back calls after 2 untimed ones)."""
    try:
        g = torch.Generator(device=dev)
        g.manual_seed(7)
        a = torch.randint(-127, 128, (M, K), dtype=torch.int8, device=dev, generator=g)
        w = torch.randint(-1, 2, (N, K), dtype=torch.int8, device=dev, generator=g)
        b = w.t()                              # [K, N] view of the row-major weights
        for _ in range(2):
            torch._int_mm(a, b)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(10):
            torch._int_mm(a, b)
        e1.record()
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) * 1e-3 / 10
    except RuntimeError as ex:                 # library call unavailable for this shape
        return {"library": "hipBLASLt via torch._int_mm", "error": str(ex)[:120]}
    return {"library": "hipBLASLt via torch._int_mm", "operands": "int8 x int8, no quantisation",
            "us": t * 1e6, "TOP/s": 2.0 * M * K * N / t / 1e12}


def sweep_bitlinear(torch, termezo, synth, dev, cpu):
    for K, N in SWEEP_GEMM_KN:
        code_bytes = N * K // 4
        L = max(64, -(-(512 << 20) // code_bytes))       # >= 512 MB of codes: beyond the caches
        lat = synth.torch_latents(77, L * N * K, torch.bfloat16, dev)
        layers = [lat[l * N * K:(l + 1) * N * K].view(N, K) for l in range(L)]
        stream = torch.cuda.Stream()
        with torch.cuda.stream(stream):
            ctx = termezo.Context(layers, stream=stream)
            ctx.build_mask(1e-3)
            ctx.perturb(1, 1e-3, 1)
        for M in SWEEP_GEMM_M:
            x = synth.torch_normal(5, (M, K), torch.float32, dev).to(torch.bfloat16)
            y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
            torch.cuda.synchronize()
            ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            with torch.cuda.stream(stream):
                ctx.bitlinear_forward(0, x, y)          # sizes the scratch before any capture
                stream.synchronize()
                if M <= 128:
                    # one graph cycling over all L code buffers (cold caches), replayed 3 times
                    g = torch.cuda.CUDAGraph()
                    with torch.cuda.graph(g, stream=stream):
                        for l in range(L):
                            ctx.bitlinear_forward(l, x, y)
                    g.replay()
                    stream.synchronize()
                    ev0.record(stream)
                    for _ in range(3):
                        g.replay()
                    ev1.record(stream)
                    stream.synchronize()
                    calls = 3 * L
                    del g
                else:
                    for _ in range(2):
                        ctx.bitlinear_forward(0, x, y)
                    ev0.record(stream)
                    calls = 10
                    for _ in range(calls):
                        ctx.bitlinear_forward(0, x, y)
                    ev1.record(stream)
                    stream.synchronize()
            t = ev0.elapsed_time(ev1) * 1e-3 / calls
            ops = 2.0 * M * K * N
            byts = K * N / 4 + M * K + 4 * M + 2 * M * N
            vendor = vendor_int8_gemm(torch, dev, M, K, N) if M > 128 else None
            c = None
            if cpu:
                tc = cpu_bitlinear(M, K, N)
                c = {"value": ops / tc / 1e12, "unit": "TOP/s", "kind": "oracle",
                     "sample": f"{min(M, 16)} rows scaled to {M}"}
            _emit({"sweep": "bitlinear_forward", "M": M, "K": K, "N": N, "us": t * 1e6,
                   "TOP/s": ops / t / 1e12, "frac_int8_peak": ops / t / 1e12 / PEAK_INT8_TOPS,
                   "algorithmic_bytes": byts, "GB/s": byts / t / 1e9,
                   "frac_hbm": byts / t / 1e9 / HBM_PEAK_GBS,
                   "protocol": (f"graph over {L} code buffers ({L * code_bytes >> 20} MiB), "
                                "activation quantisation included") if M <= 128 else
                               "10 back-to-back calls, activation quantisation included",
                   "vendor_int8_gemm": vendor, "cpu_baseline": c})
        ctx.close()
        del lat, layers
        torch.cuda.empty_cache()



def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="2b", choices=sorted(CONFIGS) + ["layer"],
                    help="2b (default: the 2B decoder), 700m (700M-class decoder), tiny (tiny "
                         "fp32 decoder), layer (one 256 x 256 BitLinear with an MSE loss)")
    ap.add_argument("--rho", type=float, default=None, help="mask ratio (default: the config's)")
    ap.add_argument("--eps", type=float, default=1e-3)
    ap.add_argument("--lr", type=float, default=None, help="learning rate (default: the config's)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sweep", choices=["latent", "bitlinear", "all"],
                    help="run the kernel sweeps instead of the step benchmark")
    ap.add_argument("--K", type=int, default=1,
                    help="perturbation directions per step (Algorithm 1; the paper's runs use 5)")
    ap.add_argument("--es", type=int, default=0,
                    help="evolution strategies on the mask (RL appendix): N one-sided population "
                         "members per step, rewards = -loss, standardised")
    ap.add_argument("--compact", action="store_true",
                    help="memory-optimal storage: after the mask build keep only the active latents "
                         "(the full latent tensor is freed)")
    ap.add_argument("--theta", action="store_true",
                    help="also perturb and update the full-precision parameters (tied embedding and "
                         "RMSNorm weights) with the latents, as Algorithm 1 does")
    ap.add_argument("--calib-copy", action="store_true",
                    help="after the measurement, copy 1 GiB device to device (a kernel of known "
                         "traffic, for scaling hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the TerMeZO step "
              "here is measured on a single MI355X", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_33548_amd import synth, termezo

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.sweep:
        if args.sweep in ("latent", "all"):
            sweep_latent(torch, termezo, synth, dev, not args.no_cpu_baseline)
        if args.sweep in ("bitlinear", "all"):
            sweep_bitlinear(torch, termezo, synth, dev, not args.no_cpu_baseline)
        return
    if args.config == "layer":
        run_layer(args, torch, termezo, synth, dev)
        return
    c = CONFIGS[args.config]
    if args.rho is None:
        args.rho = c["rho"]
    if args.lr is None:
        args.lr = c["lr"]
    fp32 = c.get("fp32", False)
    adt = torch.float32 if fp32 else torch.bfloat16
    shapes = layer_shapes(c)
    D = sum(o * i for o, i in shapes)
    print(f"[bench] config {args.config}: {len(shapes)} ternary projections, {D} latents", flush=True)
    lat = synth.torch_latents(1234, D, adt, dev)
    layers, off = [], 0
    for o, i in shapes:
        layers.append(lat[off: off + o * i].view(o, i))
        off += o * i
    E = synth.torch_normal(1235, (c["vocab"], c["d_model"]), torch.float32, dev)
    E = (E * synth.LATENT_STD).to(adt)
    tok = synth.torch_tokens(1236, c["batch"], c["seq"], c["vocab"], dev)
    torch.cuda.synchronize()

    ctx = termezo.Context(layers)
    model = termezo.Model(ctx, c["n_blocks"], c["d_model"], c["n_heads"], c["n_kv_heads"],
                          c["d_ffn"], c["vocab"], E)
    n_theta = 0
    if args.theta:
        NW = torch.ones((2 * c["n_blocks"] + 1, c["d_model"]), dtype=adt, device=dev)
        model.set_norm_weights(NW)
        ctx.theta_register([E, NW])
        n_theta = E.numel() + NW.numel()
        print(f"[bench] theta: {n_theta} full-precision parameters perturbed and updated", flush=True)
    t0 = time.perf_counter()
    k0, xi0 = ctx.build_mask(args.rho)
    mask_ms = (time.perf_counter() - t0) * 1e3
    print(f"[bench] mask: k0={k0} xi0={xi0:.3e} built in {mask_ms:.1f} ms", flush=True)
    if args.compact:
        ctx.compact()
        del lat, layers                  # frozen latents live on only as their ternary codes
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    lib_b, lat_b = ctx.memory_footprint()
    bsz = 4 if fp32 else 2
    # eq. memory of the paper for the latent side: every latent as a 2-bit code, the active
    # latents at full width, the mask as an index list or a bitmask (whichever is smaller)
    idx_bits = math.ceil(math.log2(D))
    eq_mem = D * 0.25 + k0 * bsz + min(-(-D // 8), -(-k0 * idx_bits // 8))
    print(f"[bench] memory: library {lib_b / 2**20:.1f} MiB, caller latents {lat_b / 2**20:.1f} MiB, "
          f"eq. memory estimate {eq_mem / 2**20:.1f} MiB", flush=True)
    F = torch.zeros(max(2 * args.K, args.es), device=dev)

    def step(t):
        if args.es:
            seeds = [t * args.es + n for n in range(args.es)]
            for n, sd in enumerate(seeds):
                ctx.perturb(sd, args.eps, 1)
                model.loss(tok, loss_dev=F[n: n + 1], host=False)
            # the losses are the rewards of the descent: -lr ascends on -loss
            ctx.es_update_from_rewards(seeds, F[:args.es], -args.lr)
            return
        if args.K == 1:
            ctx.perturb(t, args.eps, 1)
            model.loss(tok, loss_dev=F[0:1], host=False)
            ctx.perturb(t, args.eps, -1)
            model.loss(tok, loss_dev=F[1:2], host=False)
            ctx.update_from_losses(F[0:1], F[1:2], args.eps, args.lr)
            return
        seeds = [t * args.K + k for k in range(args.K)]     # seed s_{t,k}
        for k, sd in enumerate(seeds):
            ctx.perturb(sd, args.eps, 1)
            model.loss(tok, loss_dev=F[2 * k: 2 * k + 1], host=False)
            ctx.perturb(sd, args.eps, -1)
            model.loss(tok, loss_dev=F[2 * k + 1: 2 * k + 2], host=False)
        ctx.update_multi_from_losses(seeds, F, args.eps, args.lr)

    for t in range(args.warmup):
        step(t)
    torch.cuda.synchronize()
    print(f"[bench] warmup done ({args.warmup} steps)", flush=True)

    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for t in range(args.warmup, args.warmup + args.steps):
        step(t)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = ev0.elapsed_time(ev1) / args.steps
    print(f"[bench] {args.steps} steps: {ms_per_step:.2f} ms/step", flush=True)

    # dominant kernel: the int8 BitLinear GEMM, event-timed on the same stream
    model.set_timing(True)
    ev0.record(stream)
    for t in range(args.warmup + args.steps, args.warmup + 2 * args.steps):
        step(t)
    ev1.record(stream)
    torch.cuda.synchronize()
    timed_ms_per_step = ev0.elapsed_time(ev1) / args.steps
    g_ms, g_n, g_ops = model.timing(model.GEMM)
    a_ms, a_n, a_ops = model.timing(model.ATTENTION)
    h_ms, h_n, h_ops = model.timing(model.LM_HEAD)
    model.set_timing(False)
    k_final = ctx.active_count()
    gemm_tops = g_ops / (g_ms * 1e-3) / 1e12
    print(f"[bench] gemm {g_n} launches, {g_ms / g_n * 1e3:.1f} us avg, {gemm_tops:.1f} TOP/s; "
          f"attention {a_ms / max(1, a_n) * 1e3:.1f} us avg; lm head {h_ms / max(1, h_n) * 1e3:.1f} us avg",
          flush=True)

    if args.calib_copy:
        src = torch.empty(1 << 29, dtype=torch.bfloat16, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print("[bench] calibration copy: 1073741824 bytes read, 1073741824 bytes written", flush=True)
        del src, dst

    cpu = None
    if not args.no_cpu_baseline:
        t0 = time.perf_counter()
        cpu = (cpu_baseline_full(c, args.rho, theta=args.theta) if args.config == "tiny"
               else cpu_baseline(c, args.rho, theta_n=n_theta, K=args.K, es=args.es))
        print(f"[bench] cpu baseline sample took {time.perf_counter() - t0:.1f} s", flush=True)

    metric = METRIC if args.config == "2b" else {
        "700m": "ZO steps/sec at the 700M-class decoder shape (24 blocks, d 1536, 16 heads of 96)",
        "tiny": "ZO steps/sec, tiny decoder (2 blocks, d 256, fp32)"}[args.config]
    out = {
        "metric": metric,
        "value": 1000.0 / ms_per_step,
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8xternary+f32" if fp32 else "int8xternary+bf16",
        "data": "synthetic",
        "config": {"workload": (f"termezo_zo_step_tiny_decoder" if args.config == "tiny"
                                else f"termezo_zo_step_bitnet_{args.config}")
                               + ("_with_theta" if args.theta else "")
                               + (f"_K{args.K}" if args.K > 1 and not args.es else "")
                               + (f"_es{args.es}" if args.es else "")
                               + ("_compact" if args.compact else ""),
                   "theta_params": n_theta,
                   "directions_per_step": args.es if args.es else args.K,
                   "estimator": "es_one_sided" if args.es else "spsa_two_point",
                   "storage": "compact" if args.compact else "full_latents",
                   **{k: v for k, v in c.items() if k not in ("rho", "lr", "fp32")},
                   "tokens_per_forward": c["batch"] * c["seq"], "latents": D,
                   "mask_ratio": args.rho, "k0": k0, "k_final": k_final, "eps": args.eps,
                   "lr": args.lr, "parallelism": "single_gpu"},
        "roofline": {"bound": "mfma",
                     "kernel": "k_gemm_i8_dma + k_gemm_i8_dma_h (BitLinear int8 x ternary "
                               "GEMM, all four projections of a block)",
                     "achieved": gemm_tops, "peak": PEAK_INT8_TOPS, "unit": "TOP/s",
                     "frac": gemm_tops / PEAK_INT8_TOPS, "traffic": measured_traffic(),
                     "traffic_unit": "HBM bytes per launch",
                     "algorithmic_bytes_per_launch": gemm_algorithmic_bytes(c),
                     "launches": g_n, "avg_launch_us": g_ms / g_n * 1e3,
                     "ops_per_launch": g_ops / g_n},
        "kernels_ms_per_step": {"bitlinear_gemm": g_ms / args.steps,
                                "attention": a_ms / args.steps,
                                "lm_head_ce": h_ms / args.steps,
                                "event_timed_step_ms": timed_ms_per_step},
        "mask_build_ms": mask_ms,
        "memory": {"library_bytes": lib_b, "latent_bytes_needed": lat_b,
                   "method_state_bytes": lib_b + lat_b,
                   "eq_memory_latent_side_bytes": int(eq_mem),
                   "torch_allocated_bytes": int(torch.cuda.memory_allocated())},
        "cpu_baseline": cpu,
    }
    if args.config == "tiny":
        out["note"] = "launch-latency bound; the roofline figures are those of its tiny GEMMs"
    print(json.dumps(out), flush=True)
    model.close()
    ctx.close()


if __name__ == "__main__":
    main()
