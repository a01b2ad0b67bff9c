"""Throughput of the CAT-Q calibration step on one MI355X.

Workload: one decoder block shaped like Qwen3-1.7B (hidden 2048, 16 q / 8 kv
heads of 128, SwiGLU 6144, QK-norm, RoPE) on 4 synthetic calibration samples
of 2048 tokens (Student-t(4) activations, N(0, 0.02^2) bf16 weights, seed 0).

One step = every part of the hot path on one batch:
  group statistics + learnable modulation + softened ternarisation of all
  seven weights (s = 15, SOFT), block forward with the fake-ternary weights,
  reconstruction loss against the cached full-precision output, backward to
  the input and to every group's three factors, then hard ternarisation and
  2-bit packing of all weights.
The full-precision target is computed once before timing (it does not change
during calibration).  Inputs are resident in HBM when the timed region starts.  The step runs on
two streams: each linear's weight-gradient half (G = dY^T X and the factor
gradients) and the hard finalize go to a side stream and overlap the
input-gradient chain (--no-overlap: one stream).

Prints one JSON line.  ``value`` and ``ms_per_step`` come from the timed pass
(the production schedule: two streams, no per-launch instrumentation; --graph
replays the step captured as a HIP graph instead).  A
kernel pass then repeats the same steps on one stream with a HIP event pair
recorded by the library around each of its launches, on the launch stream:
the per-kernel durations behind ``roofline`` come from there, so a kernel's
time is not shared with concurrent work.  The CPU baseline times the float64
oracle on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "calibration block-steps/s + fake-ternary GEMM TFLOP/s and LM+ST kernel HBM GB/s"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 matrix-core peak
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E peak


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-gib", type=float, default=0.0,
                    help="only run a plain device copy of this size (counter calibration)")
    ap.add_argument("--breakdown", action="store_true", help="print the per-kernel table")
    ap.add_argument("--no-overlap", action="store_true",
                    help="run the step on one stream (no side stream for the weight-gradient "
                         "halves and the finalize)")
    ap.add_argument("--graph", action="store_true",
                    help="replay the step captured as a HIP graph in the timed pass (measured "
                         "slower than issuing the launches on this step: it is not launch-bound)")
    ap.add_argument("--ternary", type=int, default=0, metavar="M",
                    help="only time the packed-ternary decode layers of a Qwen3-14B-shaped "
                         "block at M tokens (deployment on the 2-bit storage)")
    ap.add_argument("--a8", action="store_true",
                    help="the W1.58A8 setting: activations fake-quantized to 8 bits in the step")
    ap.add_argument("--block", default="qwen3-1.7b",
                    choices=["qwen3-1.7b", "llama3-8b", "qwen3-14b", "qwen3-235b-moe",
                             "qwen3-235b-moe-skew"],
                    help="block shape of the step (the default is the headline workload; the "
                         "others are reported without a CPU baseline)")
    ap.add_argument("--window", type=int, default=1,
                    help="calibrate this many consecutive blocks jointly (sliding-window "
                         "reconstruction; 1 = the single-block step)")
    return ap.parse_args()


def counted_traffic(kernel_tag):
    """HBM bytes per launch of `kernel_tag` as last counted with rocprofv3
    (FETCH_SIZE and WRITE_SIZE runs, scaled by a plain copy's reading; the
    summary under profiles/ records the figure with a hash of the kernel
    sources).  None when no summary covers this kernel or when the sources
    changed since the count."""
    import glob
    import hashlib
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "traffic_*.md"))):
        fields = {}
        for line in open(path):
            if ":" in line and not line.startswith(("|", "#", " ")):
                k, _, v = line.partition(":")
                fields[k.strip()] = v.strip()
        if fields.get("kernel") != kernel_tag or "traffic_bytes_per_launch" not in fields:
            continue
        h = hashlib.sha256()
        try:
            for src in fields.get("sources", "").split():
                with open(os.path.join(ROOT, src), "rb") as f:
                    h.update(f.read())
        except OSError:
            return None
        if h.hexdigest() != fields.get("source_sha256"):
            return None
        return float(fields["traffic_bytes_per_launch"])
    return None


def workload_config(args, cfg):
    """The JSON `config` object: the workload named by what it is, its sizes."""
    moe = hasattr(cfg, "n_experts")
    shape = {"qwen3-1.7b": "qwen3-1.7b", "llama3-8b": "llama3-8b", "qwen3-14b": "qwen3-14b",
             "qwen3-235b-moe": "qwen3-235b-a22b routed-expert",
             "qwen3-235b-moe-skew": "qwen3-235b-a22b routed-expert (skewed expert loads)"}
    name = shape[args.block] + "-shaped decoder block"
    if args.window > 1:
        name = f"window of {args.window} {name}s"
    name += (f", {cfg.batch} x {cfg.seq} tokens, one CAT-Q calibration step (LM+ST s=15, fwd, "
             "loss, bwd to factors, ternarise+pack)")
    if args.a8:
        name += ", W1.58A8 (8-bit activations)"
    conf = {"workload": name, "hidden": cfg.hidden, "heads": [cfg.n_q, cfg.n_kv, cfg.head_dim],
            "tokens": cfg.tokens, "group_size": 128}
    if moe:
        n_w = sum(a * b for a, b in cfg.attn_shapes().values())
        n_w += sum(e * a * b for e, a, b in cfg.expert_shapes().values())
        conf.update({"experts": cfg.n_experts, "top_k": cfg.top_k, "expert_ffn": cfg.expert_ffn,
                     "weights": n_w})
    else:
        conf.update({"ffn": cfg.ffn, "weights": cfg.n_weights()})
    return conf


def cpu_baseline(cfg, W, xb, row_frac=1, n_samples=None):
    """The float64 oracle on a bounded sample of the same step (by default
    the whole step: about 10 s of host work).
    Weight side (LM+ST forward, factor gradients, final ternarise+pack): the
    first 1/row_frac of the rows of every weight matrix, scaled by row_frac
    (the work is elementwise per group, exactly linear in the weight count).
    Token side (block forward+backward): n_samples of the calibration samples
    (default all), one at a time with all weights; samples are independent in
    the block, so a full step costs t_weights + batch * (mean t_sample)."""
    import dataclasses

    import numpy as np

    import synthgen as sg
    from oracle import block, calib, lmst

    try:
        from threadpoolctl import threadpool_info
        info = threadpool_info()
        cores = max(int(i.get("num_threads", 1)) for i in info) if info else 1
    except Exception:  # pragma: no cover
        cores = 1
    cores = min(cores, len(os.sched_getaffinity(0)))
    Wo = {k: sg.bf16_bits_to_f32(v).astype(np.float64) for k, v in W.items()}
    Ws = {k: v[: v.shape[0] // row_frac] for k, v in Wo.items()}
    fac_s = {k: sg.init_factors(v.size // 128) for k, v in Ws.items()}
    one = dataclasses.replace(cfg, batch=1)
    n_samples = cfg.batch if n_samples is None else n_samples
    # weight side on the row sample
    t0 = time.perf_counter()
    calib.fake_weights(Ws, fac_s, 128, lmst.SOFT, 15.0)
    Gs = {k: np.ones_like(v) for k, v in Ws.items()}
    t1 = time.perf_counter()
    calib.factor_grads_all(Gs, Ws, fac_s, 128, lmst.SOFT, 15.0, 30.0)
    for k, v in Ws.items():
        lmst.pack_ternary(lmst.modulate_ternarize(v, 128, *fac_s[k], lmst.HARD)["codes"])
    t2 = time.perf_counter()
    t_weights = row_frac * ((t1 - t0) + (t2 - t1))
    # token side: one sample through the whole block; the arithmetic does not
    # depend on the weight values, so the bf16 weights stand in for alpha*T
    # and the input for the cached target
    t3 = time.perf_counter()
    for i in range(n_samples):
        x1 = sg.bf16_bits_to_f32(xb[i * cfg.seq:(i + 1) * cfg.seq]).astype(np.float64)
        y_q, cache = block.block_forward(x1, Wo, one)
        loss, dy = block.recon_loss(y_q, x1)
        block.block_backward(dy, cache, Wo, one)
        del cache
    t4 = time.perf_counter()
    t_sample = (t4 - t3) / n_samples
    step = t_weights + cfg.batch * t_sample
    rows = "all rows" if row_frac == 1 else f"1/{row_frac} of the rows"
    return {"value": 1.0 / step, "unit": "block-steps/s", "cores": cores, "kind": "oracle",
            "sample": (f"float64 oracle, {cores} BLAS threads: LM+ST forward, factor gradients "
                       f"and ternarise+pack on {rows} of every weight ({(t2 - t0):.1f} s"
                       f"{'' if row_frac == 1 else f', x{row_frac}'}) plus block "
                       f"forward+backward of {n_samples} of the {cfg.batch} samples of "
                       f"{cfg.seq} tokens, one at a time ({t4 - t3:.1f} s"
                       f"{'' if n_samples == cfg.batch else f', x{cfg.batch / n_samples:g}'}); "
                       "full-precision target excluded"),
            "seconds_per_step": step}


def ternary_bench(args):
    """Deployment side: the four linears of a Qwen3-14B-shaped block (q|k|v
    7168x5120, o 5120x5120, gate|up 34816x5120, down 5120x17408) as packed
    ternary weights, applied to M tokens (decode).  Random codes and scales
    (the product's cost does not depend on their values); inputs resident in
    HBM.  Reports HBM bytes moved per second (2-bit codes + fp32 scales + X +
    Y, each once) against the 8 TB/s peak, with torch's bf16 dense product
    on the same shapes (hipBLASLt) as context."""
    import numpy as np
    import torch

    import paper_2606_26650_amd as cq

    torch.cuda.set_device(0)
    M = args.ternary
    shapes = [("qkv", 7168, 5120), ("o", 5120, 5120), ("gu", 34816, 5120), ("d", 5120, 17408)]
    g = torch.Generator(device="cuda").manual_seed(0)
    layers = []
    for name, n, k in shapes:
        packed = torch.randint(0, 256, (n, k // 4), dtype=torch.uint8, device="cuda", generator=g)
        alpha = torch.rand(n, k // 128, device="cuda", generator=g) * 0.05 + 0.002
        x = torch.randn(M, k, device="cuda", generator=g).to(torch.bfloat16)
        y = torch.empty(M, n, dtype=torch.float32, device="cuda")
        layers.append((name, n, k, packed, alpha, x, y))

    def run():
        for _, _, _, packed, alpha, x, y in layers:
            cq.catq_ternary_linear(x, packed, alpha, y)

    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        run()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    # per-launch durations (HIP events on the launch stream)
    cq.catq_trace_enable(8 * args.steps + 8)
    for _ in range(args.steps):
        run()
    torch.cuda.synchronize()
    recs = cq.trace_records()
    cq.catq_trace_disable()
    per = {}
    for r, (name, n, k, *_rest) in zip(recs, [l for _ in range(args.steps) for l in layers]):
        a = per.setdefault(name, {"ms": 0.0, "bytes": r["bytes"], "tag": r["tag"]})
        a["ms"] += r["ms"] / args.steps
    tot_bytes = sum(v["bytes"] for v in per.values())
    tot_ms = sum(v["ms"] for v in per.values())
    big = per["gu"]
    # context: bf16 dense weights through torch (hipBLASLt), same shapes
    dense = [(torch.randn(n, k, device="cuda", generator=g).to(torch.bfloat16), x)
             for (_, n, k, _, _, x, _) in layers]
    for _ in range(3):
        for w, x in dense:
            torch.nn.functional.linear(x, w)
    torch.cuda.synchronize()
    d0 = time.perf_counter()
    for _ in range(args.steps):
        for w, x in dense:
            torch.nn.functional.linear(x, w)
    torch.cuda.synchronize()
    dense_ms = 1000.0 * (time.perf_counter() - d0) / args.steps
    out = {
        "metric": "packed-ternary decode: HBM GB/s of the 2-bit linear layers",
        "value": tot_bytes / (tot_ms * 1e-3) / 1e9,
        "unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": 1000.0 * elapsed / args.steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"qwen3-14b-shaped block linears (q|k|v, o, gate|up, down) as "
                               f"2-bit ternary + fp32 group scales, {M} token(s)",
                   "tokens": M, "weights": sum(n * k for _, n, k in shapes), "group_size": 128},
        "roofline": {"bound": "hbm", "kernel": big["tag"] + " (gate|up 34816x5120)",
                     "achieved": big["bytes"] / (big["ms"] * 1e-3) / 1e9, "peak": PEAK_HBM_GBS,
                     "unit": "GB/s",
                     "frac": big["bytes"] / (big["ms"] * 1e-3) / 1e9 / PEAK_HBM_GBS,
                     "avg_launch_us": 1000.0 * big["ms"], "bytes_per_launch": big["bytes"],
                     "traffic": None},
        "per_layer": {k: {"us": 1000.0 * v["ms"], "GB/s": v["bytes"] / (v["ms"] * 1e-3) / 1e9}
                      for k, v in per.items()},
        "bf16_dense_torch_ms_per_step": dense_ms,
        "kernel_ms_per_step": tot_ms,
    }
    print(json.dumps(out))


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(the sharding design is described in DESIGN.md); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2606_26650_amd as cq
    import synthgen as sg
    from paper_2606_26650_amd.block import DenseBlock, bf16_tensor

    torch.cuda.set_device(0)
    if args.copy_gib > 0:
        n = int(args.copy_gib * (1 << 30)) // 4
        a = torch.ones(n, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4}))
        return

    if args.ternary > 0:
        ternary_bench(args)
        return

    cfg = {"qwen3-1.7b": sg.QWEN3_1P7B, "llama3-8b": sg.LLAMA3_8B, "qwen3-14b": sg.QWEN3_14B,
           "qwen3-235b-moe": sg.QWEN3_235B_MOE,
           "qwen3-235b-moe-skew": sg.QWEN3_235B_MOE_SKEW}[args.block]
    moe = hasattr(cfg, "n_experts")
    if (moe or args.block != "qwen3-1.7b") and (args.window > 1 or args.a8):
        sys.exit("--window and --a8 run on the qwen3-1.7b-shaped dense block only")
    W = sg.block_weights(cfg, 0)
    xb = sg.activations(cfg, 0)
    if moe:
        from paper_2606_26650_amd.block import MoEBlock
        blk = MoEBlock(cfg, W, sg.router_logits(cfg, 0))
    elif args.window > 1:
        from paper_2606_26650_amd.window import Window
        blk = Window([DenseBlock(cfg, W, a8=args.a8)] +
                     [DenseBlock(cfg, sg.block_weights(cfg, i), a8=args.a8)
                      for i in range(1, args.window)])
    else:
        blk = DenseBlock(cfg, W, a8=args.a8)
    del W
    x = bf16_tensor(xb)
    y_fp = blk.new_output()
    blk.target(x, y_fp)
    # the final ternarisation writes the 2-bit storage directly (no int8 codes)
    fin = blk.finalize_buffers(codes=False)

    def step(overlap):
        blk.step(x, y_fp, mode=cq.SOFT, s=15.0, s_bwd=30.0, recompute_stats=True,
                 overlap=overlap, finalize=fin)

    # timed pass: the production schedule (two streams; optionally the step
    # replayed as a HIP graph), no per-launch instrumentation
    run = lambda: step(not args.no_overlap)
    if args.graph:
        from paper_2606_26650_amd.block import StepGraph
        graph = StepGraph(blk, x, y_fp, mode=cq.SOFT, s=15.0, s_bwd=30.0, recompute_stats=True,
                          overlap=not args.no_overlap, finalize=fin)
        run = graph.replay
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        run()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    elapsed = t1 - t0
    ms_step = 1000.0 * elapsed / args.steps
    loss = float(blk.loss.item())

    # kernel pass: the same steps on one stream with a HIP event pair around
    # every library launch (on its launch stream), so each kernel's duration
    # is its own and not shared with concurrent work
    step(False)
    torch.cuda.synchronize()
    cq.catq_trace_enable(64 * max(args.steps, 1) + 64)
    torch.cuda.synchronize()
    k0 = time.perf_counter()
    for _ in range(args.steps):
        step(False)
    torch.cuda.synchronize()
    k1 = time.perf_counter()
    recs = cq.trace_records()
    cq.catq_trace_disable()
    kernel_pass_ms = 1000.0 * (k1 - k0) / args.steps

    # per-kernel aggregation over the timed steps
    agg = {}
    for r in recs:
        a = agg.setdefault(r["tag"], {"n": 0, "ms": 0.0, "flops": 0.0, "bytes": 0.0})
        a["n"] += 1
        a["ms"] += r["ms"]
        a["flops"] += r["flops"]
        a["bytes"] += r["bytes"]
    gemm = {k: v for k, v in agg.items() if k.startswith("gemm") and v["flops"] > 0}
    # dominant kernel: the GEMM variant with the largest share of step time
    dom_tag, dom = max(gemm.items(), key=lambda kv: kv[1]["ms"])
    dom_tflops = dom["flops"] / (dom["ms"] * 1e-3) / 1e12
    all_gemm_ms = sum(v["ms"] for v in gemm.values())
    all_gemm_flops = sum(v["flops"] for v in gemm.values())
    lm_fwd = {k: v for k, v in agg.items() if k.startswith("lmst_fwd_kernel")}
    lmf_ms = sum(v["ms"] for v in lm_fwd.values())
    lmf_bytes = sum(v["bytes"] for v in lm_fwd.values())
    lmb = agg.get("lmst_bwd_kernel<__bf16>", {"ms": 0.0, "bytes": 0.0})
    step_gemm_flops = all_gemm_flops / args.steps

    out = {
        "metric": METRIC,
        "value": args.steps / elapsed,
        "unit": "block-steps/s" if args.window == 1 else "window-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": workload_config(args, cfg),
        "roofline": {
            "bound": "mfma",
            "kernel": dom_tag,
            "achieved": dom_tflops,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": dom_tflops / PEAK_BF16_TFLOPS,
            "avg_launch_us": 1000.0 * dom["ms"] / dom["n"],
            "flops_per_launch": dom["flops"] / dom["n"],
            "traffic": counted_traffic(dom_tag),
        },
        "schedule": ("two streams" if not args.no_overlap else "one stream") +
                    (", step replayed as a HIP graph" if args.graph else ", launches issued per step"),
        "kernel_pass": {"ms_per_step": kernel_pass_ms, "streams": 1, "steps": args.steps,
                        "instrumented": "HIP event pair per launch"},
        "gemm_tflops_all": all_gemm_flops / (all_gemm_ms * 1e-3) / 1e12,
        "gemm_share_of_step": all_gemm_ms / args.steps / kernel_pass_ms,
        "step_gemm_tflop": step_gemm_flops / 1e12,
        "lmst_fwd_gbs": lmf_bytes / (lmf_ms * 1e-3) / 1e9 if lmf_ms else None,
        "lmst_fwd_frac_hbm": (lmf_bytes / (lmf_ms * 1e-3) / 1e9) / PEAK_HBM_GBS if lmf_ms else None,
        "lmst_bwd_gbs": lmb["bytes"] / (lmb["ms"] * 1e-3) / 1e9 if lmb["ms"] else None,
        "loss": loss,
    }
    if not args.no_cpu_baseline and args.window == 1 and not args.a8 and args.block == "qwen3-1.7b":
        out["cpu_baseline"] = cpu_baseline(cfg, sg.block_weights(cfg, 0), xb)
    if args.breakdown:
        shp = {}
        for r in recs:
            if r["flops"] > 0:
                a = shp.setdefault((r["tag"], r["M"], r["N"], r["K"]), [0, 0.0, 0.0])
                a[0] += 1
                a[1] += r["ms"]
                a[2] += r["flops"]
        for (t, m, n, k), (c, ms, fl) in sorted(shp.items(), key=lambda kv: -kv[1][1]):
            print(f"{ms / args.steps:9.3f} ms/step {c // args.steps:3d}x {fl / (ms * 1e-3) / 1e12:8.1f} TF/s"
                  f"  M={m} N={n} K={k}  {t}", file=sys.stderr)
        for k, v in sorted(agg.items(), key=lambda kv: -kv[1]["ms"]):
            tf = v["flops"] / (v["ms"] * 1e-3) / 1e12 if v["flops"] else 0
            gb = v["bytes"] / (v["ms"] * 1e-3) / 1e9
            print(f"{v['ms'] / args.steps:9.3f} ms/step {v['n'] // args.steps:3d}x "
                  f"{tf:8.1f} TF/s {gb:8.1f} GB/s  {k}", file=sys.stderr)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
