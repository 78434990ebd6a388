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
    "2b": dict(n_blocks=30, d_model=2560, n_heads=20, n_kv_heads=5, d_ffn=6912, vocab=128256,
               seq=512, batch=16),
    "700m": dict(n_blocks=24, d_model=1536, n_heads=16, n_kv_heads=16, d_ffn=4096, vocab=32000,
                 seq=512, batch=8),
}
PEAK_INT8_TOPS = 5000.0          # MI355X dense int8 MFMA, TOP/s
METRIC = "ZO steps/sec at 2B BitNet shape; perturb+requant GB/s; BitLinear int8 TOPS"


def layer_shapes(c):
    hd = c["d_model"] // c["n_heads"]
    d, F = c["d_model"], c["d_ffn"]
    q, kv = c["n_heads"] * hd, c["n_kv_heads"] * hd
    return [(q, d), (kv, d), (kv, d), (d, q), (F, d), (F, d), (d, F)] * c["n_blocks"]


def cpu_baseline(c, rho, seed=0):
    """The oracle, as it stands, on a bounded sample of the same step; the
    full-step time is extrapolated by operation counts (stated in 'sample')."""
    import numpy as np
    from threadpoolctl import threadpool_info
    from oracle import decoder_ref as dec
    from oracle import termezo_ref as orc
    from paper_2609_33548_amd import synth

    shapes = layer_shapes(c)
    D = sum(o * i for o, i in shapes)
    # (1) perturb / requant / update / shrink on one sample layer (q shape)
    smp = [shapes[0]]
    nsmp = sum(o * i for o, i in smp)
    w = synth.latents(seed, [o * i for o, i in smp], bf16=True)
    st = orc.TerMeZOOracle([orc.Layer(o, i) for o, i in smp], w, bf16=True)
    st.build_mask(rho)
    t0 = time.perf_counter()
    st.perturb(1, 1e-3, 1)
    st.perturb(1, 1e-3, -1)
    st.update(1.0, 1e-4)
    t_latent = (time.perf_counter() - t0) * D / nsmp
    # (2) one decoder block on one sequence (vocab shrunk so the head is negligible)
    cfg1 = dec.DecoderConfig(n_blocks=1, d_model=c["d_model"], n_heads=c["n_heads"],
                             n_kv_heads=c["n_kv_heads"], d_ffn=c["d_ffn"], vocab=64, bf16=True)
    rng = np.random.default_rng(seed)
    codes = [rng.integers(-1, 2, size=s).astype(np.int8) for s in cfg1.layer_shapes()]
    betas = [0.016] * 7
    emb = synth.latents(seed + 1, [64 * c["d_model"]], bf16=True).reshape(64, c["d_model"])
    tok = synth.tokens(seed + 2, 1, c["seq"], 64)
    t0 = time.perf_counter()
    dec.forward_row_losses(cfg1, emb, tok, codes, betas)
    t_block = time.perf_counter() - t0
    # (3) LM head + cross-entropy for 64 positions over the full vocabulary
    E = synth.latents(seed + 3, [c["vocab"] * c["d_model"]], bf16=True).reshape(c["vocab"], c["d_model"])
    x = synth.activations(seed + 4, 64, c["d_model"], bf16=True)
    t0 = time.perf_counter()
    logits = x.astype(np.float64) @ E.astype(np.float64).T
    dec.cross_entropy_rows(logits, np.zeros(64, np.int64))
    t_head = time.perf_counter() - t0
    ntok = c["batch"] * c["seq"]
    t_fwd = c["n_blocks"] * c["batch"] * t_block + (ntok / 64) * t_head
    t_step = 2 * t_fwd + t_latent
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {
        "value": 1.0 / t_step, "unit": "steps/s", "cores": int(threads), "kind": "oracle",
        "sample": (f"oracle perturb(+/-)+update+shrink on 1 layer ({nsmp} bf16 latents) scaled to "
                   f"{D}; 1 decoder block x 1 sequence of {c['seq']} tokens scaled x{c['n_blocks']}"
                   f" blocks x{c['batch']} sequences; LM head+CE on 64 positions scaled "
                   f"x{ntok // 64}; two forwards per step; sample wall {t_latent * nsmp / D + t_block + t_head:.1f}s"),
        "extrapolated_step_s": t_step,
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="2b", choices=sorted(CONFIGS))
    ap.add_argument("--rho", type=float, default=1e-3)
    ap.add_argument("--eps", type=float, default=1e-3)
    ap.add_argument("--lr", type=float, default=1e-5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the TerMeZO step "
              "here is measured on a single MI355X", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_33548_amd import synth, termezo

    c = CONFIGS[args.config]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    shapes = layer_shapes(c)
    D = sum(o * i for o, i in shapes)
    print(f"[bench] config {args.config}: {len(shapes)} ternary projections, {D} latents", flush=True)
    lat = synth.torch_latents(1234, D, torch.bfloat16, dev)
    layers, off = [], 0
    for o, i in shapes:
        layers.append(lat[off: off + o * i].view(o, i))
        off += o * i
    E = synth.torch_normal(1235, (c["vocab"], c["d_model"]), torch.float32, dev)
    E = (E * synth.LATENT_STD).to(torch.bfloat16)
    tok = synth.torch_tokens(1236, c["batch"], c["seq"], c["vocab"], dev)
    torch.cuda.synchronize()

    ctx = termezo.Context(layers)
    model = termezo.Model(ctx, c["n_blocks"], c["d_model"], c["n_heads"], c["n_kv_heads"],
                          c["d_ffn"], c["vocab"], E)
    t0 = time.perf_counter()
    k0, xi0 = ctx.build_mask(args.rho)
    mask_ms = (time.perf_counter() - t0) * 1e3
    print(f"[bench] mask: k0={k0} xi0={xi0:.3e} built in {mask_ms:.1f} ms", flush=True)
    F = torch.zeros(2, device=dev)

    def step(t):
        ctx.perturb(t, args.eps, 1)
        model.loss(tok, loss_dev=F[0:1], host=False)
        ctx.perturb(t, args.eps, -1)
        model.loss(tok, loss_dev=F[1:2], host=False)
        ctx.update_from_losses(F[0:1], F[1:2], args.eps, args.lr)

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

    cpu = None
    if not args.no_cpu_baseline:
        t0 = time.perf_counter()
        cpu = cpu_baseline(c, args.rho)
        print(f"[bench] cpu baseline sample took {time.perf_counter() - t0:.1f} s", flush=True)

    out = {
        "metric": METRIC,
        "value": 1000.0 / ms_per_step,
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8xternary+bf16",
        "data": "synthetic",
        "config": {"workload": f"termezo_zo_step_bitnet_{args.config}", **c,
                   "tokens_per_forward": c["batch"] * c["seq"], "latents": D,
                   "mask_ratio": args.rho, "k0": k0, "k_final": k_final, "eps": args.eps,
                   "lr": args.lr, "parallelism": "single_gpu"},
        "roofline": {"bound": "mfma", "kernel": "k_gemm_i8 (BitLinear int8 GEMM)",
                     "achieved": gemm_tops, "peak": PEAK_INT8_TOPS, "unit": "TOP/s",
                     "frac": gemm_tops / PEAK_INT8_TOPS, "traffic": None,
                     "launches": g_n, "avg_launch_us": g_ms / g_n * 1e3,
                     "ops_per_launch": g_ops / g_n},
        "kernels_ms_per_step": {"bitlinear_gemm": g_ms / args.steps,
                                "attention": a_ms / args.steps,
                                "lm_head_ce": h_ms / args.steps,
                                "event_timed_step_ms": timed_ms_per_step},
        "mask_build_ms": mask_ms,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    model.close()
    ctx.close()


if __name__ == "__main__":
    main()
