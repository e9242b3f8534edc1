#!/usr/bin/env python3
"""Throughput of the forward pass of one UniF-MoE feed-forward layer on one
MI355X (bf16 expert FFNs, fp32 router), on seeded synthetic tokens.

Workload: the ViT-B/16-shaped layer - 256 images x 197 tokens = 50,432 tokens,
d = 768, K = 16 residual experts plus the shared expert, all upcycled from a
d_ff = 3072 GELU FFN and split into B = 16 blocks of M = 192 channels,
cumulative-mass threshold 0.6.

One step = one unif_moe_layer_forward call (routing, permutation, the
block-sparse expert GEMMs and the weighted merge) with inputs already
resident in HBM. Prints one JSON line. Per-phase kernel durations come from
HIP events recorded by the library itself on the launch stream during a
second pass over the same number of steps (unif_moe_layer_forward_profiled).

    python bench.py [--steps 20] [--warmup 3] [--workload vit_b16] [--no-cpu-baseline]
                    [--no-paper-exact] [--no-block] [--no-backward]

Unless --no-paper-exact, a second, shorter run repeats the workload with the
cumulative target exactly Eq. beta (t = 1) and reports it under
"paper_exact_t1" (whole-step time only). Unless --no-block, a third repeats
it as the pre-LN transformer block around the layer (LayerNorm, FFN biases,
residual add; unif_moe_block_forward) and reports it under "block_pre_ln".
Unless --no-backward, the training step's backward pass (unif_moe_layer_backward,
a first fp32 version on the vector units) is timed on the same workload and
reported under "backward" against the fp32 vector peak.
"""
import argparse
import json
import os
import sys
import time

PEAK_BF16_FLOPS = 2.5e15   # MI355X dense bf16 matrix-core peak
PEAK_HBM_BYTES = 8.0e12    # MI355X HBM3E bandwidth
PEAK_FP32_VECTOR = 157.3e12  # MI355X fp32 vector peak
METRIC = "UniF-MoE layer fwd tokens/s (bf16); MFMA util of activated FLOPs vs peak"


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="vit_b16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-paper-exact", action="store_true",
                    help="skip the second, shorter run at cumulative target t = 1")
    ap.add_argument("--no-block", action="store_true",
                    help="skip the pre-LN block run")
    ap.add_argument("--no-backward", action="store_true",
                    help="skip the backward-pass run")
    ap.add_argument("--cpu-sample", type=int, default=2048)
    ap.add_argument("--cpu-repeats", type=int, default=3)
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="after the timed steps, copy a buffer of this many MiB device to "
                         "device (a known-size reference for HBM byte counters)")
    return ap.parse_args()


def phase_bytes(cfg, st):
    """Algorithmic HBM bytes of the non-GEMM phases (minimum traffic of each
    step as defined, not counter readings)."""
    N, d, K = cfg["n_tokens"], cfg["d_model"], cfg["n_experts"]
    nv, sum_k, sum_cb = st["n_valid"], st["mean_k"] * st["n_valid"], st["activated_blocks"]
    pairs = nv + sum_k
    es = 2 if cfg["dtype"] == "bf16" else 4
    routing = N * d * es + N * (4 + 4 + 8 + 4 + 8 * K)             # read X, write the record
    permute = (N * (8 + 4) + sum_k * 4                               # read mask, k, q_1..q_k
               + pairs * (4 + 8 + 4 + 4)                             # pair token/mask/expert, pair_of
               + pairs * (4 + 8) + sum_cb * 4)                       # slab lists: read pairs, write rows
    combine = pairs * d * 4 + pairs * 8 + N * 4 + N * d * es         # fp32 per-expert rows, weights, Y
    return dict(routing=routing, permute=permute, combine=combine)


COUNTERS_PROFILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles",
                                "gemm_vit_b16_hbm_counters.md")


def library_source_hash():
    """SHA-256 over the library's kernel sources and build flags."""
    import hashlib
    base = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2608_10392_amd")
    csrc = os.path.join(base, "csrc")
    files = sorted(os.path.join("paper_2608_10392_amd", "csrc", f) for f in os.listdir(csrc)
                   if os.path.isfile(os.path.join(csrc, f)) and f.endswith((".hip", ".hpp", ".h", ".py")))
    files.append(os.path.join("paper_2608_10392_amd", "build.py"))
    h = hashlib.sha256()
    root = os.path.dirname(base)
    for f in files:
        h.update(f.encode())
        with open(os.path.join(root, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def committed_traffic(kernel):
    """HBM bytes per launch of `kernel` from the committed counter summary
    (FETCH_SIZE and WRITE_SIZE scaled by a same-run copy of known size), or
    None when the summary is missing or the sources changed since."""
    try:
        with open(COUNTERS_PROFILE) as f:
            line = next(l for l in f if l.startswith("counters-json:"))
        c = json.loads(line.split(":", 1)[1])
        if c.get("source_sha256") != library_source_hash():
            return None
        k = c["kernels"][kernel]
        return int(k["read_bytes_per_launch"] + k["write_bytes_per_launch"])
    except (OSError, StopIteration, ValueError, KeyError):
        return None


def cpu_baseline(g, n_sample, repeats):
    """The CPU oracle timed on a seeded sample of the same workload."""
    import numpy as np
    from threadpoolctl import threadpool_info
    import oracle.unif_moe_oracle as O

    cfg = dict(g["cfg"])
    valid_idx = np.arange(cfg["n_tokens"]) if g["valid"] is None else np.nonzero(g["valid"])[0]
    rng = np.random.default_rng(2024)
    sample = np.sort(rng.choice(valid_idx, size=min(n_sample, valid_idx.size), replace=False))
    sub = dict(cfg, n_tokens=int(sample.size))
    Xs = g["X"][sample]
    weights = O.ExpertWeights(cfg, g["W_up"], g["W_down"])   # one-time weight preparation
    times, cpu = [], []
    for _ in range(repeats):
        w0, c0 = time.perf_counter(), time.process_time()
        O.forward(sub, Xs, None, g["W_router"], g["prototypes"], None, None, weights=weights)
        times.append(time.perf_counter() - w0)
        cpu.append(time.process_time() - c0)
    med = float(np.median(times))
    blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
    threads = int(blas[0]["num_threads"]) if blas else 1
    return {"value": round(sample.size / med, 2), "unit": "tokens/s", "cores": threads,
            "kind": "oracle",
            "sample": f"{sample.size} seeded valid tokens of the same workload, routing + "
                      f"per-token expert evaluation, median of {repeats} runs "
                      f"({med:.2f} s each; numpy BLAS threads {threads}, "
                      f"CPU/wall {float(np.median(cpu)) / med:.2f}; weights converted once, untimed)",
            "host_cpu": _cpu_model(), "nproc": os.cpu_count()}


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the layer forward shards by tokens with no "
              "communication; run it with --gpus 1 (one MI355X).",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2608_10392_amd import _lib
    from paper_2608_10392_amd.layer import DeviceLayer
    from synth import generate, layer_config

    print(f"[bench] generating workload {args.workload}", file=sys.stderr, flush=True)
    g = generate(args.workload)
    cfg = layer_config(g["cfg"])
    dev = DeviceLayer(cfg, g["X"], g["valid"], g["W_router"], g["prototypes"], g["W_up"], g["W_down"])
    stream = torch.cuda.current_stream()

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        dev.forward()
    torch.cuda.synchronize()
    st = dev.stats()

    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        dev.forward()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall / args.steps * 1e3

    # Same steps again through the instrumented entry point: the library
    # records seven events per step on the launch stream.
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(_lib.N_PHASE_EVENTS)]
              for _ in range(args.steps)]
    for evs in events:
        for ev in evs:
            ev.record(stream)          # creates the underlying HIP event
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for evs in events:
        _lib.layer_forward_profiled(cfg, dev.X, dev.valid, dev.W_router, dev.prototypes, dev.W_up,
                                    dev.W_down, dev.Y, dev.ws_forward, evs, routing=dev.routing,
                                    stream=stream)
    torch.cuda.synchronize()
    wall_prof = time.perf_counter() - t0
    names = ["wdown_f16", "routing", "permute", "up_gemm", "down_gemm", "combine"]
    phase_ms = {n: float(np.mean([evs[i].elapsed_time(evs[i + 1]) for evs in events]))
                for i, n in enumerate(names)}

    nv = st["n_valid"]
    value = nv / (ms_per_step / 1e3)
    act = st["activated_gemm_flops"]
    gemm_ms = phase_ms["up_gemm"] + phase_ms["down_gemm"]
    dom = "up_gemm" if phase_ms["up_gemm"] >= phase_ms["down_gemm"] else "down_gemm"
    dom_flops = act / 2.0                       # each projection is half of 4 d M C_B
    achieved = dom_flops / (phase_ms[dom] / 1e3)
    pb = phase_bytes(cfg, st)
    hbm = {n: pb[n] / (phase_ms[n] / 1e3) / PEAK_HBM_BYTES for n in pb}
    hbm_all = sum(pb.values()) / ((phase_ms["routing"] + phase_ms["permute"] + phase_ms["combine"]) / 1e3)

    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {cfg['n_tokens']} tokens x d={cfg['d_model']}, "
                               f"K={cfg['n_experts']} residual + 1 shared expert, B={cfg['n_blocks']} "
                               f"blocks of M={cfg['block_width']}, threshold {cfg['mass_threshold']}",
                   "n_tokens": cfg["n_tokens"], "n_valid": nv, "d_model": cfg["d_model"],
                   "n_experts": cfg["n_experts"], "n_blocks": cfg["n_blocks"],
                   "block_width": cfg["block_width"], "mass_threshold": cfg["mass_threshold"]},
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": round(achieved / 1e12, 2),
                     "peak": PEAK_BF16_FLOPS / 1e12, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_FLOPS, 4), "traffic": committed_traffic(dom)},
        "mfma_util_activated": round(act / (gemm_ms / 1e3) / PEAK_BF16_FLOPS, 4),
        "hbm_frac": {n: round(v, 4) for n, v in hbm.items()},
        "hbm_frac_routing_permute_combine": round(hbm_all / PEAK_HBM_BYTES, 4),
        "phases_ms": {n: round(v, 4) for n, v in phase_ms.items()},
        "profiled_ms_per_step": round(wall_prof / args.steps * 1e3, 4),
        "routing_stats": {"mean_b": round(st["mean_b"], 3), "mean_k": round(st["mean_k"], 3),
                          "mean_cb": round(st["mean_cb"], 3),
                          "activated_gemm_tflop": round(act / 1e12, 4)},
    }
    if not args.no_paper_exact and cfg["mass_threshold"] != 1.0:
        # The same tokens and weights with the target exactly Eq. beta
        # (t = 1): more residual experts per token, so more activated work.
        cfg1 = dict(cfg, mass_threshold=1.0)
        dev1 = DeviceLayer(cfg1, g["X"], g["valid"], g["W_router"], g["prototypes"], g["W_up"], g["W_down"])
        steps1 = max(1, args.steps // 2)
        for _ in range(args.warmup):
            dev1.forward()
        torch.cuda.synchronize()
        st1 = dev1.stats()
        t0 = time.perf_counter()
        for _ in range(steps1):
            dev1.forward()
        torch.cuda.synchronize()
        ms1 = (time.perf_counter() - t0) / steps1 * 1e3
        out["paper_exact_t1"] = {
            "ms_per_step": round(ms1, 4), "tokens_per_s": round(st1["n_valid"] / (ms1 / 1e3), 1),
            "steps": steps1, "mean_k": round(st1["mean_k"], 3), "mean_cb": round(st1["mean_cb"], 3),
            "activated_gemm_tflop": round(st1["activated_gemm_flops"] / 1e12, 4),
            "activated_tflops_per_s": round(st1["activated_gemm_flops"] / (ms1 / 1e3) / 1e12, 1)}
        del dev1
    if not args.no_block:
        # The pre-LN block (as in DeiT) around the same layer: LN(x) feeds
        # routing and experts, b1 and b2 are added, and x is added back.
        from synth import block_inputs
        blk, Xb = block_inputs(g, "pre", residual=True, eps=1e-6)
        dev.X = None
        torch.cuda.empty_cache()
        Xd = torch.from_numpy(Xb.view(np.int16)).view(torch.bfloat16).to(dev.device)
        bd = dict(norm="pre", residual=True, ln_eps=float(blk["ln_eps"]))
        for k in ("ln_gamma", "ln_beta", "b_up", "b_down"):
            bd[k] = torch.from_numpy(blk[k]).to(dev.device)
        wsb = _lib.alloc_workspace(_lib.block_forward_workspace_size(cfg, bd), dev.device)
        dev.ws_forward = None
        torch.cuda.empty_cache()
        stepsb = max(1, args.steps // 2)

        def block_step():
            _lib.block_forward(cfg, bd, Xd, dev.valid, dev.W_router, dev.prototypes, dev.W_up,
                               dev.W_down, dev.Y, wsb, routing=dev.routing, stream=stream)
        for _ in range(args.warmup):
            block_step()
        torch.cuda.synchronize()
        stb = dev.stats()
        t0 = time.perf_counter()
        for _ in range(stepsb):
            block_step()
        torch.cuda.synchronize()
        msb = (time.perf_counter() - t0) / stepsb * 1e3
        out["block_pre_ln"] = {
            "ms_per_step": round(msb, 4), "tokens_per_s": round(stb["n_valid"] / (msb / 1e3), 1),
            "steps": stepsb, "mean_cb": round(stb["mean_cb"], 3),
            "over_layer_ms": round(msb - ms_per_step, 4)}
        del Xd, wsb, bd
    if not args.no_backward:
        # Gradients of sum(dY * Y) for the layer (forward recomputed inside).
        # Algorithmic work: four products of 2 d M per activated block (dh,
        # dx, dW_up, dW_down), i.e. 8 d M sum(C_B).
        from synth import upstream_grad
        if dev.X is None:
            dev.X = torch.from_numpy(g["X"].view(np.int16)).view(torch.bfloat16).to(dev.device)
        dY = upstream_grad(g)
        dYd = torch.from_numpy(dY.view(np.int16)).view(torch.bfloat16).to(dev.device)
        N, d, K = cfg["n_tokens"], cfg["d_model"], cfg["n_experts"]
        H = cfg["n_blocks"] * cfg["block_width"]
        f32 = dict(dtype=torch.float32, device=dev.device)
        gr = dict(dX=torch.empty((N, d), **f32), dW_up=torch.empty((K + 1, H, d), **f32),
                  dW_down=torch.empty((K + 1, d, H), **f32), dW_router=torch.empty((K + 1, d), **f32))
        wsg = _lib.alloc_workspace(_lib.layer_backward_workspace_size(cfg), dev.device)

        def bwd_step():
            _lib.layer_backward(cfg, dev.X, dev.valid, dev.W_router, dev.prototypes, dev.W_up,
                                dev.W_down, dYd, gr["dX"], gr["dW_up"], gr["dW_down"],
                                gr["dW_router"], wsg, stream=stream)
        print("[bench] backward", file=sys.stderr, flush=True)
        bwd_step()
        torch.cuda.synchronize()
        stepsg = 2
        t0 = time.perf_counter()
        for _ in range(stepsg):
            bwd_step()
        torch.cuda.synchronize()
        msg = (time.perf_counter() - t0) / stepsg * 1e3
        bflops = 8.0 * cfg["d_model"] * cfg["block_width"] * st["activated_blocks"]
        out["backward"] = {
            "ms_per_step": round(msg, 3), "steps": stepsg, "dtype": "f32 (bf16 inputs)",
            "algorithmic_tflop": round(bflops / 1e12, 4),
            "roofline": {"bound": "alu", "achieved": round(bflops / (msg / 1e3) / 1e12, 2),
                         "peak": PEAK_FP32_VECTOR / 1e12, "unit": "TFLOP/s",
                         "frac": round(bflops / (msg / 1e3) / PEAK_FP32_VECTOR, 4)}}
        del wsg, gr, dYd
        torch.cuda.empty_cache()
    if args.copy_calibration_mb > 0:
        nbytes = args.copy_calibration_mb << 20
        src = torch.ones(nbytes, dtype=torch.uint8, device=dev.device)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_calibration_bytes"] = nbytes
        del src, dst
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(g, args.cpu_sample, args.cpu_repeats)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
