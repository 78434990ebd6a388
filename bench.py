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

The default run prints ONE JSON line: the headline step (steps/s, the roofline
of the dominant kernel -- the int8 BitLinear GEMM, each launch timed by HIP events
that take the kernel's own start and end on the library's stream -- and the
oracle baseline on the host cores), and under "rows" every other measured workload of the hot path, each with its own
roofline fraction and oracle baseline (single-threaded and on all host cores):
  d1  single BitLinear layer (256 x 256, fp32, MSE), 100 steps
  d2  tiny fp32 decoder (2 blocks, d 256)
  d3  700M-class decoder (24 blocks, d 1536, 16 heads of 96)
  d4  the 2B step with every latent active (mask ratio 1: dense MeZO)
  d5a/d5b  perturb+requant and update+shrink over 2.4e9 bf16 latents at mask
      ratios 1e-4, 1e-3, 1e-2, 1
  d5c/d5d  BitLinear forward at M in {1, 16, 128} (cold caches) and {2048, 8192}
      tokens for (K, N) in {(2560, 2560), (2560, 6912), (6912, 2560)}
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
HBM_PEAK_GBS = 8000.0            # MI355X HBM3E, GB/s
PEAK_BF16_TFLOPS = 2500.0        # MI355X dense bf16 MFMA, TFLOP/s
PEAK_FP32_TFLOPS = 157.3         # MI355X fp32 vector, TFLOP/s
# HBM traffic of the GEMM launches measured with rocprofv3 counters (FETCH_SIZE,
# WRITE_SIZE), valid only for the kernel source it was measured on.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "bitlinear_gemm_traffic_2b_step.txt")
# the GEMM kernels and every header they include (tile order, direct-to-LDS loads, unpacking)
GEMM_SOURCES = [os.path.join(ROOT, "paper_2609_33548_amd", "csrc", f)
                for f in ("tmz_bitlinear.hip", "tmz_device.h", "tmz_internal.h")]
METRIC = "ZO steps/sec at 2B BitNet shape; perturb+requant GB/s; BitLinear int8 TOPS"
ROWS = ("d1", "d2", "d3", "d4", "d5ab", "d5cd")


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


def calibration_copy(torch, dev):
    """A 1 GiB device-to-device copy: a kernel of known traffic, by which hardware
    byte counters taken in the same run are scaled to bytes."""
    src = torch.empty(1 << 29, dtype=torch.bfloat16, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    log("calibration copy: 1073741824 bytes read, 1073741824 bytes written")
    del src, dst


def log(msg):
    print(f"[bench] {msg}", flush=True)


def _emit(rec):
    print(json.dumps(rec), flush=True)


# ---------------------------------------------------------------------------
# CPU baselines: the oracle as it stands, on a bounded sample of each workload,
# once on one host thread and once on all host cores (the oracle's OpenMP build
# for its C loops, numpy's BLAS pool for its matrix products).
# ---------------------------------------------------------------------------
def all_cores():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        n = min(n, int(env))
    return n


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
    return {"model": name, "logical_cpus": all_cores()}


def run_leg(threads, fn, *a, **kw):
    """fn(*a, **kw) with the oracle's C loops and numpy's BLAS on `threads` threads."""
    from threadpoolctl import threadpool_limits
    from oracle import termezo_ref as orc
    with threadpool_limits(limits=threads):
        orc.use_threads(threads)
        try:
            return fn(*a, **kw)
        finally:
            orc.use_threads(1)


def _public(d):
    return {k: v for k, v in d.items() if not k.startswith("_")}


def _faster(a, b):
    """The better of two legs by the metric's direction (time-like units are lower-better)."""
    lower = a["unit"].startswith("us")
    return (a if a["value"] <= b["value"] else b) if lower else (a if a["value"] >= b["value"] else b)


def combine_legs(st, mt, n):
    """Baseline record of two legs: both with their thread counts, and at the top
    the faster one (its value, unit, sample and thread count)."""
    legs = {"single_thread": {**_public(st), "cores": 1}, "all_cores": {**_public(mt), "cores": n}}
    best = _faster(legs["single_thread"], legs["all_cores"])
    return {**best, "kind": "oracle", "host": host_cpu(), **legs}


def two_legs(fn, st_kw, mt_kw):
    """The baseline on one thread and on all host cores.  Returns (baseline dict,
    single-thread result, all-core result)."""
    t0 = time.perf_counter()
    n = all_cores()
    st = run_leg(1, fn, **st_kw)
    mt = run_leg(n, fn, **mt_kw)
    log(f"cpu baseline ({fn.__name__}) took {time.perf_counter() - t0:.1f} s")
    combined = combine_legs(st, mt, n) if "value" in st else None   # nested results: caller combines
    return combined, st, mt


_INPUTS = {}


def _cached(key, make):
    """Synthetic inputs of the oracle samples, drawn once per run (both legs time the
    oracle on the same inputs; drawing them is not part of the timed work)."""
    if key not in _INPUTS:
        _INPUTS[key] = make()
    return _INPUTS[key]


def cpu_decoder_step(c, rho, n_lat_layers=1, n_seq=1, n_pos=256, theta_n=0, K=1, es=0,
                     seed=0, fwd=None):
    """The oracle's decoder step, extrapolated from a sample (stated in 'sample'):
    perturb(+), perturb(-), update + shrink on the first n_lat_layers projections
    scaled to all latents; one decoder block on n_seq sequences scaled to all
    blocks and the batch; the LM head + cross-entropy on n_pos positions scaled to
    all tokens.  fwd: a forward time measured before (only the latent part is then
    sampled)."""
    import numpy as np
    from oracle import decoder_ref as dec
    from oracle import termezo_ref as orc
    from paper_2609_33548_amd import synth

    shapes = layer_shapes(c)
    D = sum(o * i for o, i in shapes)
    smp = shapes[:n_lat_layers]
    nsmp = sum(o * i for o, i in smp)
    w = synth.latents(seed, [o * i for o, i in smp], bf16=True)
    st = orc.TerMeZOOracle([orc.Layer(o, i) for o, i in smp], w, bf16=True)
    st.build_mask(rho)
    t0 = time.perf_counter()
    st.perturb(1, 1e-3, 1)
    st.perturb(1, 1e-3, -1)
    st.update(1.0, 1e-4)
    t_latent = (time.perf_counter() - t0) * D / nsmp
    wall = t_latent * nsmp / D
    ntok = c["batch"] * c["seq"]
    if fwd is None:
        cfg1 = dec.DecoderConfig(n_blocks=1, d_model=c["d_model"], n_heads=c["n_heads"],
                                 n_kv_heads=c["n_kv_heads"], d_ffn=c["d_ffn"], vocab=64, bf16=True)
        rng = np.random.default_rng(seed)
        codes = [rng.integers(-1, 2, size=s).astype(np.int8) for s in cfg1.layer_shapes()]
        emb = synth.latents(seed + 1, [64 * c["d_model"]], bf16=True).reshape(64, c["d_model"])
        tok = synth.tokens(seed + 2, n_seq, c["seq"], 64)
        t0 = time.perf_counter()
        dec.forward_row_losses(cfg1, emb, tok, codes, [0.016] * 7)
        t_block = (time.perf_counter() - t0) / n_seq
        # the LM head on a slice of the vocabulary (its cost is linear in the vocabulary)
        vs = -(-c["vocab"] // 8)
        E = _cached(("E", seed, vs, c["d_model"]), lambda: synth.latents(
            seed + 3, [vs * c["d_model"]], bf16=True).reshape(vs, c["d_model"]))
        x = synth.activations(seed + 4, n_pos, c["d_model"], bf16=True)
        t0 = time.perf_counter()
        logits = x.astype(np.float64) @ E.astype(np.float64).T
        dec.cross_entropy_rows(logits, np.zeros(n_pos, np.int64))
        t_head = time.perf_counter() - t0
        fwd = c["n_blocks"] * c["batch"] * t_block + (ntok / n_pos) * (c["vocab"] / vs) * t_head
        wall += t_block * n_seq + t_head
        fwd_sample = (f"1 decoder block x {n_seq} sequence(s) of {c['seq']} tokens scaled "
                      f"x{c['n_blocks']} blocks x{c['batch'] / n_seq:g}; LM head+CE on {n_pos} "
                      f"positions x {vs} vocabulary columns scaled x{ntok / n_pos:g} "
                      f"x{c['vocab'] / vs:g}")
    else:
        fwd_sample = "forward time of the same workload's baseline at the same thread count"
    t_theta, n_th = 0.0, 1 << 20
    if theta_n:
        th = synth.latents(seed + 5, [n_th], bf16=True)
        t0 = time.perf_counter()
        orc.theta_perturbed(th, 0, 1, 1e-3, 1, True)
        orc.theta_perturbed(th, 0, 1, 1e-3, -1, True)
        orc.theta_updated(th, 0, 1, 1e-4, 1.0, True)
        t_theta = (time.perf_counter() - t0) * theta_n / n_th
        wall += t_theta * n_th / theta_n
    # K directions: K perturbation pairs and 2K forwards; ES: es one-sided members
    t_step = K * (2 * fwd + t_latent + t_theta)
    if es:
        t_step = es * (fwd + 0.5 * (t_latent + t_theta))
    return {"value": 1.0 / t_step, "unit": "steps/s",
            "sample": (f"oracle perturb(+/-)+update+shrink on {n_lat_layers} projection(s) ({nsmp} "
                       f"bf16 latents, mask ratio {rho:g}) scaled to {D}; {fwd_sample}; two "
                       f"forwards per step"
                       + (f"; theta perturb(+/-)+update on {n_th} ids scaled to {theta_n}"
                          if theta_n else "")
                       + (f"; all of it x{K} directions" if K > 1 and not es else "")
                       + (f"; ES: {es} members x (one forward + half the perturb/update sample)"
                          if es else "")
                       + f"; sample wall {wall:.1f} s; extrapolated"),
            "extrapolated_step_s": t_step, "_fwd": fwd}


def cpu_full_steps(c, rho, n_steps=8, seed=0, theta=False):
    """The oracle's full decoder step (perturb +/-, two forwards, update) on the same
    workload, for configurations small enough to run whole."""
    import numpy as np
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
    return {"value": 1.0 / dt, "unit": "steps/s",
            "sample": f"{n_steps} full oracle steps of the same workload"}


def cpu_layer_steps(n_steps=200, seed=0):
    """The oracle's full single-layer step (perturb +/-, BitLinear, MSE, update), timed."""
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
    return {"value": 1.0 / dt, "unit": "steps/s",
            "sample": f"{n_steps} full oracle steps of the same workload (C + numpy)"}


# ---------------------------------------------------------------------------
# Kernel sweeps: the perturb/requant and update kernels over a 2.4e9-latent
# tensor at several mask ratios, and the BitLinear forward over small and large
# token counts.
# ---------------------------------------------------------------------------
SWEEP_LAYER = (6912, 2560)           # 136 layers of this shape: 2,406,481,920 latents
SWEEP_LAYERS = 136
SWEEP_RATIOS = (1e-4, 1e-3, 1e-2, 1.0)
SWEEP_GEMM_KN = ((2560, 2560), (2560, 6912), (6912, 2560))
SWEEP_GEMM_M = (1, 16, 128, 2048, 8192)
LATENT_CPU_LAYER = (2560, 2560)


def cpu_latent_point(ratio, seed=0):
    """Oracle perturb(+) and update(+shrink) on one 2560 x 2560 bf16 layer at the
    sweep's mask ratio: perturb GB/s by the sweep's byte count, update time scaled
    to the sweep's 2.4e9 latents."""
    from oracle import termezo_ref as orc
    from paper_2609_33548_amd import synth
    o, i = LATENT_CPU_LAYER
    n = o * i
    w = synth.latents(seed, [n], bf16=True)
    st = orc.TerMeZOOracle([orc.Layer(o, i)], w, bf16=True)
    st.build_mask(ratio)
    k = st.k
    t0 = time.perf_counter()
    st.perturb(1, 1e-3, 1)
    t_p = time.perf_counter() - t0
    t0 = time.perf_counter()
    st.update(1.0, 1e-5)
    t_u = time.perf_counter() - t0
    scale = SWEEP_LAYERS * SWEEP_LAYER[0] * SWEEP_LAYER[1] / n
    return {"perturb": {"value": (n * 2.25 + k * 6) / t_p / 1e9, "unit": "GB/s",
                        "sample": f"one {o}x{i} bf16 layer, perturb(+), same mask ratio"},
            "update": {"value": t_u * scale * 1e6, "unit": "us (scaled to the sweep's latents)",
                       "sample": f"one {o}x{i} bf16 layer, update+shrink, same mask ratio, "
                                 f"time x{scale:g}"}}


def cpu_bitlinear_point(M, K, N, rows=16, seed=0):
    """Oracle BitLinear (activation quantisation + exact integer product, the C
    triple loop) on at most `rows` rows, scaled to M."""
    import numpy as np
    from oracle import termezo_ref as orc
    from paper_2609_33548_amd import synth
    m = min(M, rows)
    rng = np.random.default_rng(seed)
    codes = rng.integers(-1, 2, size=(N, K)).astype(np.int8)
    x = synth.activations(seed, m, K, bf16=True)
    t0 = time.perf_counter()
    xq, s = orc.act_quant(x)
    orc.bitlinear(xq, s, codes, 0.016)
    t = (time.perf_counter() - t0) * M / m
    return {"value": 2.0 * M * K * N / t / 1e12, "unit": "TOP/s",
            "sample": f"{m} rows scaled to {M}"}


# ---------------------------------------------------------------------------
# GPU workloads
# ---------------------------------------------------------------------------
def row_single_layer(torch, termezo, synth, dev, steps=100, warmup=5, cpu=True):
    """Single-layer workload: one BitLinear 256 x 256 with fp32 latents, 8 token rows, MSE
    to a N(0, 1) target, mask ratio 1e-2.  A step is perturb +/-, two forwards with the
    MSE written to device scalars, g and the masked update on the device (no host
    synchronisation)."""
    w = synth.torch_latents(0, LAYER["d_out"] * LAYER["d_in"], torch.float32, dev).view(
        LAYER["d_out"], LAYER["d_in"])
    x = torch.from_numpy(synth.activations(100, LAYER["tokens"], LAYER["d_in"])).to(dev)
    tgt = torch.from_numpy(synth.activations(101, LAYER["tokens"], LAYER["d_out"])).to(dev)
    y = torch.empty((LAYER["tokens"], LAYER["d_out"]), device=dev)
    F = torch.zeros(2, device=dev)
    ctx = termezo.Context([w])
    k0, _ = ctx.build_mask(LAYER["rho"])

    def step(t):
        for j, sign in enumerate((1, -1)):
            ctx.perturb(t, LAYER["eps"], sign)
            ctx.bitlinear_forward(0, x, y)
            ctx.mse_loss_dev(y, tgt, F[j: j + 1])
        ctx.update_from_losses(F[0:1], F[1:2], LAYER["eps"], LAYER["lr"])

    for t in range(warmup):
        step(t)
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for t in range(warmup, warmup + steps):
        step(t)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / steps
    k_final = ctx.active_count()
    ctx.close()
    log(f"single layer: {steps} steps, {ms * 1e3:.1f} us/step")
    out = {"metric": "ZO steps/sec, single BitLinear with MSE loss", "value": 1000.0 / ms,
           "unit": "steps/s", "steps": steps, "warmup": warmup, "ms_per_step": ms,
           "dtype": "int8xternary+f32",
           "config": {"workload": "termezo_zo_step_bitlinear_256x256_mse", **LAYER, "k0": k0,
                      "k_final": k_final},
           "roofline": None,
           "bound": "launch latency: a few dozen microsecond-scale kernels per step on 65,536 "
                    "weights and 8 token rows; reported as an absolute rate"}
    if cpu:
        out["cpu_baseline"] = two_legs(cpu_layer_steps, {"n_steps": 200}, {"n_steps": 200})[0]
    return out


# the two evaluations of a pair run at the same time in the timed pass (--sequential: one
# after the other on the context's stream, as in the per-kernel timing pass)
PAIR_STREAMS = True


def run_decoder(torch, termezo, synth, dev, c, rho, eps, lr, steps, warmup, theta=False, K=1,
                es=0, compact=False, calib_copy=False, keep=False):
    """The decoder step of configuration c: builds the workload, times `steps` steps
    after `warmup` (one event pair on the library's stream), then the same number of
    steps again with per-kernel event timing of the matrix-core kernels and of the
    perturbation / update calls.  Returns the result dict, and the live state when
    keep is set (for a second mask ratio on the same workload)."""
    fp32 = c.get("fp32", False)
    adt = torch.float32 if fp32 else torch.bfloat16
    shapes = layer_shapes(c)
    D = sum(o * i for o, i in shapes)
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
    # the F+ evaluation of each pair: a second model on a stream of its own, reading a
    # snapshot of the + codes while the context computes and evaluates the - side
    pair = None
    if K == 1 and not es and PAIR_STREAMS:
        pair = termezo.Model(ctx, c["n_blocks"], c["d_model"], c["n_heads"], c["n_kv_heads"],
                             c["d_ffn"], c["vocab"], E)
        pair.set_stream(torch.cuda.Stream())
        pair.use_snapshot(True)
    n_theta = 0
    if theta:
        NW = torch.ones((2 * c["n_blocks"] + 1, c["d_model"]), dtype=adt, device=dev)
        model.set_norm_weights(NW)
        if pair is not None:
            pair.set_norm_weights(NW)
        ctx.theta_register([E, NW])
        n_theta = E.numel() + NW.numel()
        log(f"theta: {n_theta} full-precision parameters perturbed and updated")
    st = {"ctx": ctx, "model": model, "pair": pair, "tok": tok, "lat": lat, "layers": layers,
          "E": E, "D": D, "c": c, "n_theta": n_theta}
    res = measure_steps(torch, st, rho, eps, lr, steps, warmup, K=K, es=es, compact=compact)
    if calib_copy:
        calibration_copy(torch, dev)
    if keep:
        return res, st
    close_state(torch, st)
    return res, None


def close_state(torch, st):
    if st.get("pair") is not None:
        st["pair"].close()
    st["model"].close()
    st["ctx"].close()
    st.clear()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def measure_steps(torch, st, rho, eps, lr, steps, warmup, K=1, es=0, compact=False):
    ctx, model, tok, c, D = st["ctx"], st["model"], st["tok"], st["c"], st["D"]
    pair = st.get("pair")
    fp32 = c.get("fp32", False)
    t0 = time.perf_counter()
    k0, xi0 = ctx.build_mask(rho)
    mask_ms = (time.perf_counter() - t0) * 1e3
    log(f"{c['n_blocks']}-block decoder, {D} latents: mask ratio {rho:g}, k0={k0} xi0={xi0:.3e} "
        f"built in {mask_ms:.1f} ms")
    if compact:
        ctx.compact()
        del st["lat"], st["layers"]      # frozen latents live on only as their ternary codes
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    lib_b, lat_b = ctx.memory_footprint()
    bsz = 4 if fp32 else 2
    # eq. memory of the paper for the latent side: every latent as a 2-bit code, the active
    # latents at full width, the mask as an index list or a bitmask (whichever is smaller)
    idx_bits = math.ceil(math.log2(D))
    eq_mem = D * 0.25 + k0 * bsz + min(-(-D // 8), -(-k0 * idx_bits // 8))
    F = torch.zeros(max(2 * K, es, 2), device="cuda")
    stream = torch.cuda.current_stream()
    lat_ev = []                          # event pairs around the perturbation / update calls
    record = [False]

    def timed(fn):
        if not record[0]:
            fn()
            return
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        fn()
        b.record(stream)
        lat_ev.append((a, b))

    def step(t):
        if es:
            seeds = [t * es + n for n in range(es)]
            for n, sd in enumerate(seeds):
                timed(lambda: ctx.perturb(sd, eps, 1))
                model.loss(tok, loss_dev=F[n: n + 1], host=False)
            # the losses are the rewards of the descent: -lr ascends on -loss
            timed(lambda: ctx.es_update_from_rewards(seeds, F[:es], -lr))
            return
        if K == 1 and pair is not None and not record[0]:
            # F+ on the pair model's stream from the snapshot, F- on the context's stream
            ctx.perturb(t, eps, 1)
            ctx.codes_snapshot()
            pair.loss(tok, loss_dev=F[0:1], host=False)
            ctx.perturb(t, eps, -1)
            model.loss(tok, loss_dev=F[1:2], host=False)
            pair.join()
            ctx.update_from_losses(F[0:1], F[1:2], eps, lr)
            return
        if K == 1:
            timed(lambda: ctx.perturb(t, eps, 1))
            model.loss(tok, loss_dev=F[0:1], host=False)
            timed(lambda: ctx.perturb(t, eps, -1))
            model.loss(tok, loss_dev=F[1:2], host=False)
            timed(lambda: ctx.update_from_losses(F[0:1], F[1:2], eps, lr))
            return
        seeds = [t * K + k for k in range(K)]     # seed s_{t,k}
        for k, sd in enumerate(seeds):
            timed(lambda: ctx.perturb(sd, eps, 1))
            model.loss(tok, loss_dev=F[2 * k: 2 * k + 1], host=False)
            timed(lambda: ctx.perturb(sd, eps, -1))
            model.loss(tok, loss_dev=F[2 * k + 1: 2 * k + 2], host=False)
        timed(lambda: ctx.update_multi_from_losses(seeds, F, eps, lr))

    for t in range(warmup):
        step(t)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for t in range(warmup, warmup + steps):
        step(t)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = ev0.elapsed_time(ev1) / steps
    log(f"{steps} steps: {ms_per_step:.2f} ms/step")

    # second pass: per-kernel event timing of the matrix-core kernels and of the calls
    # that perturb and update the latents
    record[0] = True
    model.set_timing(True)
    ev0.record(stream)
    for t in range(warmup + steps, warmup + 2 * steps):
        step(t)
    ev1.record(stream)
    torch.cuda.synchronize()
    timed_ms = ev0.elapsed_time(ev1) / steps
    g_ms, g_n, g_ops = model.timing(model.GEMM)
    a_ms, a_n, a_ops = model.timing(model.ATTENTION)
    h_ms, h_n, h_ops = model.timing(model.LM_HEAD)
    model.set_timing(False)
    latent_ms = sum(a.elapsed_time(b) for a, b in lat_ev) / steps
    k_final = ctx.active_count()
    lib_s, _ = ctx.memory_footprint()   # while stepping: the codes snapshot of the pair included
    gemm_tops = g_ops / (g_ms * 1e-3) / 1e12
    log(f"gemm {g_n} launches, {g_ms / g_n * 1e3:.1f} us avg, {gemm_tops:.1f} TOP/s; attention "
        f"{a_ms / max(1, a_n) * 1e3:.1f} us avg; lm head {h_ms / max(1, h_n) * 1e3:.1f} us avg; "
        f"perturb+update calls {latent_ms:.2f} ms/step")
    return {
        "value": 1000.0 / ms_per_step, "unit": "steps/s", "steps": steps, "warmup": warmup,
        "ms_per_step": ms_per_step,
        "dtype": "int8xternary+f32" if fp32 else "int8xternary+bf16",
        "config": {"theta_params": st["n_theta"], "directions_per_step": es if es else K,
                   "pair_evaluation": "two_streams" if pair is not None else "sequential",
                   "estimator": "es_one_sided" if es else "spsa_two_point",
                   "storage": "compact" if compact else "full_latents",
                   **{k: v for k, v in c.items() if k not in ("rho", "lr", "fp32")},
                   "tokens_per_forward": c["batch"] * c["seq"], "latents": D,
                   "mask_ratio": rho, "k0": k0, "k_final": k_final, "eps": eps, "lr": lr},
        "roofline": {"bound": "mfma",
                     "kernel": "k_gemm_i8_dma + k_gemm_i8_dma_h (BitLinear int8 x ternary "
                               "GEMM, all four projections of a block)",
                     "achieved": gemm_tops, "peak": PEAK_INT8_TOPS, "unit": "TOP/s",
                     "frac": gemm_tops / PEAK_INT8_TOPS,
                     "algorithmic_bytes_per_launch": gemm_algorithmic_bytes(c),
                     "launches": g_n, "avg_launch_us": g_ms / g_n * 1e3,
                     "ops_per_launch": g_ops / g_n},
        "kernels_ms_per_step": {"bitlinear_gemm": g_ms / steps, "attention": a_ms / steps,
                                "lm_head_ce": h_ms / steps,
                                "perturb_update_calls": latent_ms,
                                "event_timed_step_ms": timed_ms},
        "step_roofline": step_roofline(c, g_ops / steps, a_ops / steps, h_ops / steps, k0,
                                       K if not es else es, ms_per_step),
        "attention_tflops": a_ops / (a_ms * 1e-3) / 1e12 if a_ms else None,
        "lm_head_tflops": h_ops / (h_ms * 1e-3) / 1e12 if h_ms else None,
        "mask_build_ms": mask_ms,
        "memory": {"library_bytes": lib_s, "library_bytes_after_mask_build": lib_b,
                   "latent_bytes_needed": lat_b, "method_state_bytes": lib_s + lat_b,
                   "eq_memory_latent_side_bytes": int(eq_mem),
                   "torch_allocated_bytes": int(torch.cuda.memory_allocated())},
    }


def step_roofline(c, gemm_ops, attn_flops, lm_flops, k, dirs, ms_per_step):
    """The whole step against the rooflines: sum over its kernel classes of algorithmic
    work / peak (matrix-core classes at their dense peak, attention at the larger of its
    flop and HBM times, the bandwidth-bound classes at 8 TB/s), over the measured step."""
    el = 4 if c.get("fp32") else 2                       # bytes per stored activation
    peak_mm = PEAK_FP32_TFLOPS if c.get("fp32") else PEAK_BF16_TFLOPS   # attention, LM head
    M = c["batch"] * c["seq"]
    d, F = c["d_model"], c["d_ffn"]
    hd = d // c["n_heads"]
    dkv = c["n_kv_heads"] * hd
    evals = 2 * dirs                                     # forwards per step
    # per forward: quantising row kernels read the activation and write int8 (+ 8 B scale and
    # row sum per token); K rotation and V transposition read and write K and V; the
    # embedding gather and the stored final norm read and write one activation row each
    row_b = c["n_blocks"] * (3 * M * ((el + 1) * d + 8) + M * ((el + 1) * F + 8)
                             + 4 * el * M * dkv) + 4 * el * M * d
    attn_b = c["n_blocks"] * (2 * el * M * d + 2 * el * M * dkv)
    attn_f = attn_flops / max(1, evals)
    attn_ms = evals * max(attn_f / (peak_mm * 1e12),
                          attn_b / (HBM_PEAK_GBS * 1e9)) * 1e3
    # latent side: perturbation pair (index, w' of both signs, code word read and write per
    # active) and update (index, latent read and write, new value)
    lat_b = dirs * 2 * 26 * k + 20 * k
    parts = {"bitlinear_gemm": gemm_ops / (PEAK_INT8_TOPS * 1e12) * 1e3,
             "lm_head_ce": lm_flops / (peak_mm * 1e12) * 1e3,
             "attention": attn_ms,
             "row_kernels": evals * row_b / (HBM_PEAK_GBS * 1e9) * 1e3,
             "latent_side": lat_b / (HBM_PEAK_GBS * 1e9) * 1e3}
    ideal = sum(parts.values())
    return {"ideal_ms": ideal, "measured_ms": ms_per_step, "frac": ideal / ms_per_step,
            "ideal_ms_parts": parts}


def _hbm(gbs):
    return {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": gbs / HBM_PEAK_GBS}


VALU_NOTE = ("generator-bound: every latent draws its Philox word and Box-Muller pair; VALU "
             "busy from SQ counters in profiles/latent_valu_2p4e9_latents.md; the HBM target "
             "does not apply")


def sweep_latent(torch, termezo, synth, dev, cpu, compact_mode=True, reps=10):
    """Returns (perturb points, update points)."""
    o, i = SWEEP_LAYER
    D = SWEEP_LAYERS * o * i
    lat = synth.torch_latents(4321, D, torch.bfloat16, dev)
    layers = [lat[l * o * i:(l + 1) * o * i].view(o, i) for l in range(SWEEP_LAYERS)]
    torch.cuda.synchronize()
    ctx = termezo.Context(layers)
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    pert, upd = [], []
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
        # update + shrink per active: 4 B index, 2 B latent read and written, 4 B z (the pair
        # pass's draws, read instead of drawn again), 2 B new value; the shrink reads the new
        # value and the index and writes the index: 20 B in all
        b_u = 20 * k
        # default path: the same codes; only the actives' codes are rewritten while the
        # threshold-drift guard holds (per active: 4 B index + 2 B latent read, 4 B w' written,
        # index and w' read again, the code word read and, where the code changes, written)
        # (above 1/256 active: the code words of the tiles with actives read and written,
        # 0.5 B per weight, plus 4 B index + 4 B w' + 6 B for the delta per active)
        b_g = k * 26 if k * 256 <= D else D * 0.5 + k * 14
        dense_gbs, guard_gbs, upd_gbs = b_p / t_p / 1e9, b_g / t_g / 1e9, b_u / t_u / 1e9
        valu = {"bound": "alu", "frac": None, "note": VALU_NOTE}
        p = {"ratio": r, "k": k, "latents": D,
             "dense_requant": {"ms": t_p * 1e3, "algorithmic_bytes": b_p, "GB/s": dense_gbs,
                               "roofline": _hbm(dense_gbs) if r < 1 else
                               {**valu, "frac_hbm": dense_gbs / HBM_PEAK_GBS}},
             "guarded": {"ms": t_g * 1e3, "algorithmic_bytes": b_g, "GB/s": guard_gbs,
                         "speedup_vs_dense": t_p / t_g,
                         "roofline": _hbm(guard_gbs) if r < 1 else
                         {**valu, "frac_hbm": guard_gbs / HBM_PEAK_GBS}},
             "protocol": "mean over 5 (+eps, -eps) pairs of one seed each; dense = every latent "
                         "re-quantised (termezo_set_dense_requant), guarded = the default path "
                         "(the same codes)"}
        if r == 1e-2:
            u_roof = _hbm(upd_gbs)
        elif r < 1e-2:
            u_roof = {"bound": "latency", "frac": None, "frac_hbm": upd_gbs / HBM_PEAK_GBS,
                      "note": "microsecond-scale kernels over a few MB; reported in us"}
        else:
            u_roof = {**_hbm(upd_gbs),
                      "note": "the draws come from the pair pass (no generator in the update); "
                              "VALU busy about 65% (SQ counters in "
                              "profiles/latent_valu_2p4e9_latents.md)"}
        u = {"ratio": r, "k": k, "k_after": k_after, "latents": D, "us": t_u * 1e6,
             "algorithmic_bytes": b_u, "GB/s": upd_gbs, "roofline": u_roof}
        if cpu:
            _, cst, cmt = two_legs(cpu_latent_point, {"ratio": r}, {"ratio": r})
            n_all = all_cores()
            p["cpu_baseline"] = combine_legs(cst["perturb"], cmt["perturb"], n_all)
            u["cpu_baseline"] = combine_legs(cst["update"], cmt["update"], n_all)
        pert.append(p)
        upd.append(u)
        log(f"latent sweep ratio {r:g}: dense {t_p * 1e3:.3f} ms ({dense_gbs:.0f} GB/s), guarded "
            f"{t_g * 1e3:.3f} ms, update {t_u * 1e6:.1f} us")
    ctx.close()
    if compact_mode:
        # memory-optimal storage: a fresh context per ratio (the compact form is kept until
        # the context ends); the actives live contiguously in list order
        for j, r in enumerate(SWEEP_RATIOS):
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
            cc.sync()
            cc.close()
            b_g = k * 26 if k * 256 <= D else D * 0.5 + k * 14
            pert[j]["compact"] = {"ms": t_c * 1e3, "GB/s": b_g / t_c / 1e9,
                                  "library_bytes": lib_b}
            upd[j]["compact_us"] = t_uc * 1e6
    del lat, layers
    torch.cuda.empty_cache()
    return pert, upd


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


def sweep_bitlinear(torch, termezo, synth, dev, cpu, vendor=True):
    pts = []
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
            tops, gbs = ops / t / 1e12, byts / t / 1e9
            p = {"M": M, "K": K, "N": N, "us": t * 1e6, "TOP/s": tops,
                 "algorithmic_bytes": byts, "GB/s": gbs,
                 "roofline": _hbm(gbs) if M <= 128 else
                 {"bound": "mfma", "achieved": tops, "peak": PEAK_INT8_TOPS, "unit": "TOP/s",
                  "frac": tops / PEAK_INT8_TOPS},
                 "protocol": (f"graph over {L} code buffers ({L * code_bytes >> 20} MiB), "
                              "activation quantisation included") if M <= 128 else
                             "10 back-to-back calls, activation quantisation included"}
            if vendor and M > 128:
                p["vendor_int8_gemm"] = vendor_int8_gemm(torch, dev, M, K, N)
            if cpu:
                cb = two_legs(cpu_bitlinear_point, {"M": M, "K": K, "N": N},
                              {"M": M, "K": K, "N": N})[0]
                cb.pop("host", None)
                p["cpu_baseline"] = cb
            pts.append(p)
            log(f"bitlinear M={M} K={K} N={N}: {t * 1e6:.1f} us, {tops:.1f} TOP/s, {gbs:.0f} GB/s")
        ctx.close()
        del lat, layers
        torch.cuda.empty_cache()
    return pts


# ---------------------------------------------------------------------------
def build_rows(args, torch, termezo, synth, dev, which, head_state=None, head_fwd=None):
    """The other workloads of the hot path, one entry each (see the module docstring)."""
    cpu = not args.no_cpu_baseline
    rows = {}
    if "d4" in which and head_state is not None:
        c = CONFIGS["2b"]
        res = measure_steps(torch, head_state, 1.0, args.eps, c["lr"], steps=5, warmup=2)
        res["metric"] = "ZO steps/sec at the 2B shape with every latent active (dense MeZO)"
        res["config"]["workload"] = "termezo_zo_step_bitnet_2b_rho1"
        res["bound_note"] = ("the GEMMs as in the headline step; at this ratio the perturbation "
                             "pair is generator-bound and the update (which reads the pair's "
                             "draws) and shrink stream every latent (perturb_update_calls)")
        if cpu:
            fwd_st, fwd_mt = head_fwd if head_fwd else (None, None)
            res["cpu_baseline"] = two_legs(
                cpu_decoder_step, {"c": c, "rho": 1.0, "n_seq": 2, "n_pos": 256, "fwd": fwd_st},
                {"c": c, "rho": 1.0, "n_lat_layers": 2, "n_seq": 16, "n_pos": 2048,
                 "fwd": fwd_mt})[0]
        rows["d4_2b_rho1"] = res
    if head_state is not None:
        close_state(torch, head_state)
    if "d3" in which:
        c = CONFIGS["700m"]
        res, _ = run_decoder(torch, termezo, synth, dev, c, c["rho"], args.eps, c["lr"],
                             steps=10, warmup=3)
        res["metric"] = ("ZO steps/sec at the 700M-class decoder shape (24 blocks, d 1536, "
                         "16 heads of 96)")
        res["config"]["workload"] = "termezo_zo_step_bitnet_700m"
        if cpu:
            res["cpu_baseline"] = two_legs(
                cpu_decoder_step, {"c": c, "rho": c["rho"], "n_seq": 1, "n_pos": 512},
                {"c": c, "rho": c["rho"], "n_lat_layers": 7, "n_seq": 8, "n_pos": 4096})[0]
        rows["d3_700m"] = res
    if "d2" in which:
        c = CONFIGS["tiny"]
        res, _ = run_decoder(torch, termezo, synth, dev, c, c["rho"], args.eps, c["lr"],
                             steps=20, warmup=3)
        res["metric"] = "ZO steps/sec, tiny decoder (2 blocks, d 256, fp32)"
        res["config"]["workload"] = "termezo_zo_step_tiny_decoder"
        res["roofline"] = None
        res["bound"] = ("launch latency: about 60 kernels per forward on 256 tokens; reported "
                        "as an absolute rate")
        if cpu:
            res["cpu_baseline"] = two_legs(cpu_full_steps, {"c": c, "rho": c["rho"], "n_steps": 16},
                                           {"c": c, "rho": c["rho"], "n_steps": 16})[0]
        rows["d2_tiny"] = res
    if "d1" in which:
        rows["d1_single_layer"] = row_single_layer(torch, termezo, synth, dev, cpu=cpu)
    if "d5ab" in which:
        pert, upd = sweep_latent(torch, termezo, synth, dev, cpu, compact_mode=False)
        rows["d5a_perturb_requant"] = pert
        rows["d5b_update"] = upd
    if "d5cd" in which:
        pts = sweep_bitlinear(torch, termezo, synth, dev, cpu)
        rows["d5c_bitlinear_small_m"] = [p for p in pts if p["M"] <= 128]
        rows["d5d_bitlinear_large_m"] = [p for p in pts if p["M"] > 128]
    return rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="2b", choices=sorted(CONFIGS) + ["layer"],
                    help="the headline workload: 2b (default), 700m, tiny, or layer (one "
                         "256 x 256 BitLinear with an MSE loss)")
    ap.add_argument("--rows", default=None,
                    help="comma list of the other workloads to add to the line ("
                         + ",".join(ROWS) + "), 'all' or 'none'; default: all for the plain "
                         "2B run, none otherwise")
    ap.add_argument("--only", choices=ROWS, default=None,
                    help="measure one of the other workloads alone (no headline step)")
    ap.add_argument("--rho", type=float, default=None, help="mask ratio (default: the config's)")
    ap.add_argument("--eps", type=float, default=1e-3)
    ap.add_argument("--lr", type=float, default=None, help="learning rate (default: the config's)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sweep", choices=["latent", "bitlinear", "all"],
                    help="run the kernel sweeps alone, one JSON line per point")
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
    ap.add_argument("--sequential", action="store_true",
                    help="evaluate the two sides of each perturbation pair one after the other "
                         "(default: the + side on a second stream from a snapshot of its codes)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="after the measurement, copy 1 GiB device to device (a kernel of known "
                         "traffic, for scaling hardware byte counters)")
    args = ap.parse_args()
    global PAIR_STREAMS
    PAIR_STREAMS = not args.sequential
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the TerMeZO step "
              "here is measured on a single MI355X", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_33548_amd import synth, termezo

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cpu = not args.no_cpu_baseline
    t_start = time.perf_counter()
    if args.sweep:
        if args.sweep in ("latent", "all"):
            pert, upd = sweep_latent(torch, termezo, synth, dev, cpu)
            for p in pert:
                _emit({"sweep": "perturb_requant", **p})
            for u in upd:
                _emit({"sweep": "update", **u})
        if args.sweep in ("bitlinear", "all"):
            for p in sweep_bitlinear(torch, termezo, synth, dev, cpu):
                _emit({"sweep": "bitlinear_forward", **p})
        return
    if args.only:
        state = fwd = None
        if args.only == "d4":
            c = CONFIGS["2b"]
            _, state = run_decoder(torch, termezo, synth, dev, c, c["rho"], args.eps, c["lr"], 1, 1,
                                   keep=True)
        rows = build_rows(args, torch, termezo, synth, dev, [args.only], head_state=state,
                          head_fwd=fwd)
        if args.calib_copy:
            calibration_copy(torch, dev)
        _emit({"rows": rows, "wall_s": time.perf_counter() - t_start})
        return
    if args.config == "layer":
        out = row_single_layer(torch, termezo, synth, dev, steps=args.steps, warmup=args.warmup,
                               cpu=cpu)
        out.update({"n_gpus": 1, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
                    "data": "synthetic"})
        out["config"]["parallelism"] = "single_gpu"
        _emit(out)
        return

    c = CONFIGS[args.config]
    rho = args.rho if args.rho is not None else c["rho"]
    lr = args.lr if args.lr is not None else c["lr"]
    plain = (args.config == "2b" and args.K == 1 and not args.es and not args.compact
             and not args.theta and args.rho is None)
    if args.rows in (None, "all"):
        which = list(ROWS) if (plain or args.rows == "all") else []
    elif args.rows == "none":
        which = []
    else:
        which = args.rows.split(",")
    keep = "d4" in which and plain
    log(f"config {args.config}: {len(layer_shapes(c))} ternary projections")
    head, state = run_decoder(torch, termezo, synth, dev, c, rho, args.eps, lr, args.steps,
                              args.warmup, theta=args.theta, K=args.K, es=args.es,
                              compact=args.compact, calib_copy=args.calib_copy, keep=keep)
    head_fwd = None
    cpu_head = None
    if cpu:
        if args.config == "tiny":
            cpu_head = two_legs(cpu_full_steps,
                                {"c": c, "rho": rho, "n_steps": 16, "theta": args.theta},
                                {"c": c, "rho": rho, "n_steps": 16, "theta": args.theta})[0]
        else:
            kw = dict(c=c, rho=rho, theta_n=head["config"]["theta_params"], K=args.K, es=args.es)
            cpu_head, st_leg, mt_leg = two_legs(
                cpu_decoder_step, {**kw, "n_seq": 2, "n_pos": 256},
                {**kw, "n_lat_layers": 7, "n_seq": 16, "n_pos": 2048})
            head_fwd = (st_leg["_fwd"], mt_leg["_fwd"])
    rows = (build_rows(args, torch, termezo, synth, dev, which, head_state=state,
                       head_fwd=head_fwd) if which else {})

    workload = (("termezo_zo_step_tiny_decoder" if args.config == "tiny"
                 else f"termezo_zo_step_bitnet_{args.config}")
                + ("_with_theta" if args.theta else "")
                + (f"_K{args.K}" if args.K > 1 and not args.es else "")
                + (f"_es{args.es}" if args.es else "")
                + ("_compact" if args.compact else ""))
    metric = METRIC if args.config == "2b" else {
        "700m": "ZO steps/sec at the 700M-class decoder shape (24 blocks, d 1536, 16 heads of 96)",
        "tiny": "ZO steps/sec, tiny decoder (2 blocks, d 256, fp32)"}[args.config]
    head["roofline"]["traffic"] = measured_traffic() if args.config == "2b" else None
    head["roofline"]["traffic_unit"] = "HBM bytes per launch"
    out = {
        "metric": metric, "value": head["value"], "unit": "steps/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": head["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": head["dtype"], "data": "synthetic",
        "config": {"workload": workload, **head["config"], "parallelism": "single_gpu"},
        "roofline": head["roofline"],
        "kernels_ms_per_step": head["kernels_ms_per_step"],
        "step_roofline": head["step_roofline"],
        "attention_tflops": head["attention_tflops"], "lm_head_tflops": head["lm_head_tflops"],
        "mask_build_ms": head["mask_build_ms"], "memory": head["memory"],
        "cpu_baseline": cpu_head,
    }
    if args.config == "tiny":
        out["note"] = "launch-latency bound; the roofline figures are those of its tiny GEMMs"
    if rows:
        out["rows"] = rows
    out["wall_s"] = time.perf_counter() - t_start
    _emit(out)


if __name__ == "__main__":
    main()
