#!/usr/bin/env python3
"""Throughput of the forward pass of one UniF-MoE feed-forward layer on one
MI355X (bf16 expert FFNs, fp32 router), on seeded synthetic tokens.

Headline workload: the ViT-B/16-shaped layer - 256 images x 197 tokens =
50,432 tokens, d = 768, K = 16 residual experts plus the shared expert, all
upcycled from a d_ff = 3072 GELU FFN and split into B = 16 blocks of M = 192
channels, cumulative-mass threshold 0.6.

One step = one unif_moe_layer_forward call (routing, permutation, the
block-sparse expert GEMMs and the weighted merge) with inputs already
resident in HBM. `value` is valid tokens / wall-clock seconds over exactly
`steps` synchronized steps; the median of per-step HIP events on the launch
stream is reported beside it. Per-phase kernel durations come from HIP events
the library records on the launch stream (unif_moe_layer_forward_profiled),
medians over the steps. Prints one JSON line.

    python bench.py [--steps 50] [--warmup 3] [--workload vit_b16] [--no-cpu-baseline]
                    [--no-configs] [--no-paper-exact] [--no-block] [--no-backward]
                    [--no-ablations] [--vendor-reference]

Also, unless switched off: "configs" - the other workloads (ViT-S/16, BERT-base
with padding, the skewed 131k-token layer, the paper's DeiT-S and BERT-large
operating points), each with tokens/s, phases, MFMA utilisation and roofline;
"paper_exact_t1" - the headline tokens with the cumulative target exactly
Eq. beta (t = 1); "ablations" - the headline tokens under the ablation
table's routing variants (fixed alpha, top-2 residual, prefix blocks);
"block_pre_ln" - the DeiT-style pre-LN block around the layer;
"block_post_ln" - the BERT-style post-LN block on the paper's BERT-large
shape; "backward" - the training step's backward pass and the Gram
diversity loss; "cpu_baseline" - the CPU oracle timed on a sample of the
headline workload, with the GPU output on the same sample checked against it
("parity_on_sample").
"""
import argparse
import json
import os
import sys
import threading
import time

PEAK_BF16_FLOPS = 2.5e15   # MI355X dense bf16/fp16 matrix-core peak
PEAK_HBM_BYTES = 8.0e12    # MI355X HBM3E bandwidth
METRIC = "UniF-MoE layer fwd tokens/s (bf16); MFMA util of activated FLOPs vs peak"
# Intervals between the profiled entry point's 7 events; the first is empty
# (the fp16 copy of W_down runs inside the routing launches) and not reported.
PHASES = ["(empty)", "routing", "permute", "up_gemm", "down_gemm", "combine"]
OTHER_CONFIGS = ["vit_s16", "bert_base_padded", "zipf_stress", "paper_vision", "paper_language"]


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="vit_b16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true", help="skip the other workloads")
    ap.add_argument("--no-paper-exact", action="store_true",
                    help="skip the second, shorter run at cumulative target t = 1")
    ap.add_argument("--no-block", action="store_true", help="skip the pre-LN block run")
    ap.add_argument("--no-backward", action="store_true", help="skip the backward-pass run")
    ap.add_argument("--no-ablations", action="store_true",
                    help="skip the routing ablation modes and the post-LN block")
    ap.add_argument("--cpu-sample", type=int, default=2048)
    ap.add_argument("--cpu-repeats", type=int, default=3)
    ap.add_argument("--vendor-reference", action="store_true",
                    help="also time dense bf16 GEMMs of the workload's FFN shapes and one expert slab "
                         "through torch.matmul (hipBLASLt), and a device copy, as a vendor reference")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="after the timed steps, copy a buffer of this many MiB device to "
                         "device (a known-size reference for HBM byte counters)")
    return ap.parse_args()


def phase_bytes(cfg, st):
    """Algorithmic HBM bytes of the non-GEMM phases (minimum traffic of each
    step as defined, not counter readings). The fp16 copy of W_down (bf16
    layers) is made by extra workgroups of the routing decisions' launch, so
    its bytes belong to the routing phase."""
    N, d, K, H = cfg["n_tokens"], cfg["d_model"], cfg["n_experts"], cfg["n_blocks"] * cfg["block_width"]
    nv, sum_k, sum_cb = st["n_valid"], st["mean_k"] * st["n_valid"], st["activated_blocks"]
    pairs = nv + sum_k
    es = 2 if cfg["dtype"] == "bf16" else 4
    wdown = (K + 1) * d * H * (2 + 2) if cfg["dtype"] == "bf16" else 0   # read bf16, write fp16
    routing = N * d * es + N * (4 + 4 + 8 + 4 + 8 * K) + wdown       # read X, write the record; the copy
    permute = (N * (8 + 4) + sum_k * 4                               # read mask, k, q_1..q_k
               + pairs * (4 + 8 + 4 + 4)                             # pair token/mask/expert, pair_of
               + sum_cb * 8)                                         # slab lists: pair and token per row
    combine = pairs * d * 4 + pairs * 8 + N * 4 + N * d * es         # fp32 per-expert rows, weights, Y
    return dict(routing=routing, permute=permute, combine=combine)


COUNTERS_PROFILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles",
                                "vit_b16_forward_hbm_counters.md")


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


def committed_phase_bytes():
    """HBM bytes per forward of each phase (sum over its kernels) from the
    committed counter summary of the headline workload (FETCH_SIZE and
    WRITE_SIZE scaled by a same-run copy of known size), or None when the
    summary is missing or the sources changed since."""
    try:
        with open(COUNTERS_PROFILE) as f:
            line = next(l for l in f if l.startswith("counters-json:"))
        c = json.loads(line.split(":", 1)[1])
        if c.get("source_sha256") != library_source_hash():
            return None
        out = {}
        for k in c["kernels"].values():
            out[k["phase"]] = out.get(k["phase"], 0) + int(k["read_bytes_per_launch"] + k["write_bytes_per_launch"])
        return out
    except (OSError, StopIteration, ValueError, KeyError):
        return None


def median(v):
    v = sorted(v)
    n = len(v)
    return v[n // 2] if n % 2 else 0.5 * (v[n // 2 - 1] + v[n // 2])


class ClockSampler:
    """Shader- and memory-clock samples read from sysfs while the GPU runs
    (the current levels of pp_dpm_sclk and pp_dpm_mclk; the shader clock
    falls back to the hwmon frequency); best effort, no child processes."""

    def __init__(self):
        import glob
        self.samples = {"sclk": [], "mclk": []}
        self._stop = threading.Event()
        self._t = None
        self._dpm = {k: sorted(glob.glob(f"/sys/class/drm/card*/device/pp_dpm_{k}")) for k in self.samples}
        self._hwmon = sorted(glob.glob("/sys/class/drm/card*/device/hwmon/hwmon*/freq1_input"))

    def _read(self, kind):
        for path in self._dpm[kind]:
            try:
                with open(path) as f:
                    for line in f:
                        if line.rstrip().endswith("*"):
                            return int("".join(ch for ch in line.split(":", 1)[1] if ch.isdigit()))
            except (OSError, ValueError, IndexError):
                pass
        if kind == "sclk":
            for path in self._hwmon:
                try:
                    with open(path) as f:
                        return int(f.read().strip()) // 1000000
                except (OSError, ValueError):
                    pass
        return None

    def _run(self):
        while not self._stop.is_set():
            for kind, v in self.samples.items():
                x = self._read(kind)
                if x:
                    v.append(x)
            self._stop.wait(0.05)

    def start(self):
        self._t = threading.Thread(target=self._run, daemon=True)
        self._t.start()

    def stop(self):
        self._stop.set()
        if self._t is not None:
            self._t.join(timeout=5)
        out = {}
        for kind, v in self.samples.items():
            s = sorted(v)
            out[kind] = {"samples": len(s), "max_mhz": s[-1] if s else None,
                         "median_mhz": s[len(s) // 2] if s else None}
        out["note"] = ("sysfs current DPM levels every 50 ms from the headline run to the end of the other "
                       "workloads (idle gaps included); the shader clock under each kernel, from SQ counters, "
                       "is in the committed SQ profile")
        return out


def measure(torch, _lib, dev, cfg, steps, warmup, stream):
    """Wall-clock and event timing of `steps` forwards, then the same steps
    through the profiled entry point (phase events)."""
    for _ in range(warmup):
        dev.forward(stream=stream)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for a, b in ev:
        a.record(stream)
        dev.forward(stream=stream)
        b.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_ms = [a.elapsed_time(b) for a, b in ev]
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(_lib.N_PHASE_EVENTS)] for _ in range(steps)]
    for evs in events:
        for e in evs:
            e.record(stream)          # creates the underlying HIP event
    torch.cuda.synchronize()
    for evs in events:
        _lib.layer_forward_profiled(cfg, dev.X, dev.valid, dev.W_router, dev.prototypes, dev.W_up,
                                    dev.W_down, dev.Y, dev.ws_forward, evs, routing=dev.routing,
                                    stream=stream)
    torch.cuda.synchronize()
    phase_ms = {n: median([evs[i].elapsed_time(evs[i + 1]) for evs in events]) for i, n in enumerate(PHASES)
                if n != "(empty)"}
    return wall / steps * 1e3, median(step_ms), phase_ms


def summarize(cfg, st, work, ms_event, phase_ms):
    """Throughput, MFMA utilisation, roofline of the dominant GEMM and HBM
    fractions of the other phases."""
    nv = st["n_valid"]
    act = st["activated_gemm_flops"]
    gemm_ms = phase_ms["up_gemm"] + phase_ms["down_gemm"]
    dom = "up_gemm" if phase_ms["up_gemm"] >= phase_ms["down_gemm"] else "down_gemm"
    achieved = act / 2.0 / (phase_ms[dom] / 1e3)       # each projection is half of 4 d M C_B
    pb = phase_bytes(cfg, st)
    rpc = ["routing", "permute", "combine"]
    out = {
        "tokens_per_s": round(nv / (ms_event / 1e3), 1), "ms_per_step_event_median": round(ms_event, 4),
        "n_valid": nv, "mean_b": round(st["mean_b"], 3), "mean_k": round(st["mean_k"], 3),
        "mean_cb": round(st["mean_cb"], 3), "activated_gemm_tflop": round(act / 1e12, 4),
        "phases_ms": {n: round(v, 4) for n, v in phase_ms.items()},
        "mfma_util_activated": round(act / (gemm_ms / 1e3) / PEAK_BF16_FLOPS, 4),
        "roofline_dominant_gemm": {"bound": "mfma", "kernel": dom, "achieved": round(achieved / 1e12, 2),
                                   "peak": PEAK_BF16_FLOPS / 1e12, "unit": "TFLOP/s",
                                   "frac": round(achieved / PEAK_BF16_FLOPS, 4)},
        "hbm_frac": {n: round(pb[n] / (phase_ms[n] / 1e3) / PEAK_HBM_BYTES, 4) for n in pb if phase_ms[n] > 0},
        "hbm_frac_routing_permute_combine": round(
            sum(pb[n] for n in rpc) / (sum(phase_ms[n] for n in rpc) / 1e3) / PEAK_HBM_BYTES, 4),
    }
    if work is not None:
        out["executed_vs_activated"] = {
            "up": round(work["up_mfma_flops"] / (act / 2.0), 4),
            "down": round(work["down_mfma_flops"] / (act / 2.0), 4),
            "mfma_util_executed": round((work["up_mfma_flops"] + work["down_mfma_flops"]) / (gemm_ms / 1e3)
                                        / PEAK_BF16_FLOPS, 4)}
    return out


def vendor_reference(torch, cfg, st):
    """Dense bf16 GEMMs of the layer's FFN shapes (all N tokens through all H
    channels: [N, d] x [d, H] and [N, H] x [H, d]) and of one expert-block
    slab's shape (its mean row count x d x M) through torch.matmul, which
    dispatches to hipBLASLt; medians of 20 HIP-event timings after 3 warmups,
    against the 2.5 PFLOP/s bf16 peak. Also a device-to-device copy of 1 GiB
    (bytes read + written per second)."""
    N, d, H, M = cfg["n_tokens"], cfg["d_model"], cfg["n_blocks"] * cfg["block_width"], cfg["block_width"]
    g = torch.Generator(device="cuda")
    g.manual_seed(0)
    out = {}

    def timed(fn, reps=20):
        for _ in range(3):
            fn()
        ts = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        return median(ts)

    def gemm(name, m, k, n):
        A = torch.randn(m, k, device="cuda", dtype=torch.bfloat16, generator=g)
        B = torch.randn(k, n, device="cuda", dtype=torch.bfloat16, generator=g)
        ms = timed(lambda: A @ B)
        fl = 2.0 * m * k * n
        out[name] = {"shape": f"{m}x{k}x{n}", "ms": round(ms, 4), "tflops": round(fl / ms / 1e9, 1),
                     "frac": round(fl / ms / 1e9 / (PEAK_BF16_FLOPS / 1e12), 4)}

    gemm("dense_up", N, d, H)
    gemm("dense_down", N, H, d)
    rows = max(1, int(round(st["activated_blocks"] / ((cfg["n_experts"] + 1) * cfg["n_blocks"]))))
    gemm("slab_up", rows, d, M)
    src = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    ms = timed(lambda: dst.copy_(src), reps=10)
    out["copy_1gib"] = {"ms": round(ms, 4), "TBps": round(2 * src.numel() * 4 / ms / 1e9, 2)}
    out["note"] = "torch.matmul (hipBLASLt) and torch copy, HIP-event medians"
    return out


def cpu_baseline_and_sample_check(g, Y_gpu, rec_gpu, n_sample, repeats):
    """The CPU oracle timed on a seeded sample of the same workload; the GPU
    output on the sample checked against it (raw and beyond-half-ulp error
    x RMS over the tokens whose decisions the two agree on and whose margins
    are at least 1e-4; near-tie tokens counted)."""
    import numpy as np
    from threadpoolctl import threadpool_info
    import oracle.unif_moe_oracle as O
    from synth.generate import bf16_bits_to_f32

    cfg = dict(g["cfg"])
    valid_idx = np.arange(cfg["n_tokens"]) if g["valid"] is None else np.nonzero(g["valid"])[0]
    rng = np.random.default_rng(2024)
    sample = np.sort(rng.choice(valid_idx, size=min(n_sample, valid_idx.size), replace=False))
    sub = dict(cfg, n_tokens=int(sample.size))
    Xs = g["X"][sample]
    weights = O.ExpertWeights(cfg, g["W_up"], g["W_down"])   # one-time weight preparation
    times, cpu = [], []
    Yref = rec = None
    for _ in range(repeats):
        w0, c0 = time.perf_counter(), time.process_time()
        Yref, rec = O.forward(sub, Xs, None, g["W_router"], g["prototypes"], None, None, weights=weights)
        times.append(time.perf_counter() - w0)
        cpu.append(time.process_time() - c0)
    med = float(np.median(times))
    blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
    threads = int(blas[0]["num_threads"]) if blas else 1
    base = {"value": round(sample.size / med, 2), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{sample.size} seeded valid tokens of the same workload, routing + "
                      f"per-token expert evaluation, median of {repeats} runs "
                      f"({med:.2f} s each; numpy BLAS threads {threads}, "
                      f"CPU/wall {float(np.median(cpu)) / med:.2f}; weights converted once, untimed)",
            "host_cpu": _cpu_model(), "nproc": os.cpu_count()}
    m, _ = O.margins(sub, rec)
    same = np.ones(sample.size, bool)
    for key in ("n_shared", "shared_mask", "n_res"):
        same &= rec_gpu[key][sample] == rec[key]
    sure = (m >= 1e-4) & same
    yg = bf16_bits_to_f32(Y_gpu[sample][sure]).astype(np.float64)
    ref = Yref[sure]
    rms = float(np.sqrt(np.mean(ref ** 2))) if ref.size else 1.0
    err = np.abs(yg - ref)
    half = np.where(ref == 0, 0.0, 2.0 ** (np.floor(np.log2(np.maximum(np.abs(ref), 1e-300))) - 8))
    check = {"tokens": int(sample.size), "near_ties": int(np.sum(m < 1e-4)),
             "decisions_differ_beyond_margin": int(np.sum((m >= 1e-4) & ~same)),
             "max_raw_error_x_rms": round(float(err.max() / rms), 5) if err.size else 0.0,
             "max_error_beyond_half_ulp_x_rms": round(float(np.maximum(err - half, 0).max() / rms), 5)
             if err.size else 0.0}
    return base, check


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

    print(f"[bench] warmup {args.warmup}, timing {args.steps} steps", file=sys.stderr, flush=True)
    clock = ClockSampler()
    clock.start()
    ms_per_step, ms_event, phase_ms = measure(torch, _lib, dev, cfg, args.steps, args.warmup, stream)
    st = dev.stats()
    work = _lib.forward_work(cfg, dev.ws_forward) if cfg["dtype"] == "bf16" else None
    Y_head = dev.output_numpy()
    rec_head = dev.routing_numpy()
    head = summarize(cfg, st, work, ms_event, phase_ms)
    nv = st["n_valid"]
    rf = head["roofline_dominant_gemm"]
    out = {
        "metric": METRIC, "value": round(nv / (ms_per_step / 1e3), 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "ms_per_step_event_median": head["ms_per_step_event_median"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {cfg['n_tokens']} tokens x d={cfg['d_model']}, "
                               f"K={cfg['n_experts']} residual + 1 shared expert, B={cfg['n_blocks']} "
                               f"blocks of M={cfg['block_width']}, threshold {cfg['mass_threshold']}",
                   "n_tokens": cfg["n_tokens"], "n_valid": nv, "d_model": cfg["d_model"],
                   "n_experts": cfg["n_experts"], "n_blocks": cfg["n_blocks"],
                   "block_width": cfg["block_width"], "mass_threshold": cfg["mass_threshold"]},
        "roofline": {"bound": "mfma", "kernel": rf["kernel"], "achieved": rf["achieved"], "peak": rf["peak"],
                     "unit": "TFLOP/s", "frac": rf["frac"], "traffic": None},
    }
    counted = committed_phase_bytes() if args.workload == "vit_b16" else None
    if counted is not None:
        out["roofline"]["traffic"] = counted.get(rf["kernel"])
        rpc = [n for n in ("routing", "permute", "combine") if n in counted]
        out["hbm_frac_counters"] = {n: round(counted[n] / (phase_ms[n] / 1e3) / PEAK_HBM_BYTES, 4) for n in rpc}
        out["hbm_frac_counters"]["routing_permute_combine"] = round(
            sum(counted[n] for n in rpc) / (sum(phase_ms[n] for n in rpc) / 1e3) / PEAK_HBM_BYTES, 4)
        out["counted_bytes"] = counted
    for k in ("mfma_util_activated", "executed_vs_activated", "hbm_frac", "hbm_frac_routing_permute_combine",
              "phases_ms"):
        if k in head:
            out[k] = head[k]
    out["routing_stats"] = {k: head[k] for k in ("mean_b", "mean_k", "mean_cb", "activated_gemm_tflop")}
    # Workspace of the timed forward (sized for the worst case, every token on
    # all K experts) against one sized by the pair capacity cfg max_pairs for
    # the pairs this routing produced (what a caller that knows its routing
    # statistics allocates; unif_moe_forward_status reports an overflow).
    _, pairs = _lib.forward_status(cfg, dev.ws_forward)
    out["workspace_gb"] = {
        "worst_case": round(_lib.layer_forward_workspace_size(cfg) / 1e9, 3),
        "at_capacity": round(_lib.layer_forward_workspace_size(dict(cfg, max_pairs=pairs)) / 1e9, 3),
        "pairs": pairs, "worst_case_pairs": cfg["n_tokens"] * (cfg["n_experts"] + 1)}

    if not args.no_paper_exact and cfg["mass_threshold"] != 1.0:
        # The same tokens and weights with the target exactly Eq. beta
        # (t = 1): more residual experts per token, so more activated work.
        print("[bench] paper-exact target t = 1", file=sys.stderr, flush=True)
        cfg1 = dict(cfg, mass_threshold=1.0)
        dev1 = DeviceLayer(cfg1, g["X"], g["valid"], g["W_router"], g["prototypes"], g["W_up"], g["W_down"])
        steps1 = max(2, args.steps // 2)
        ms1, ev1, ph1 = measure(torch, _lib, dev1, cfg1, steps1, args.warmup, stream)
        st1 = dev1.stats()
        s1 = summarize(cfg1, st1, _lib.forward_work(cfg1, dev1.ws_forward), ev1, ph1)
        out["paper_exact_t1"] = dict(s1, steps=steps1, ms_per_step=round(ms1, 4))
        del dev1
        torch.cuda.empty_cache()
    if not args.no_configs:
        out["configs"] = {}
        for name in OTHER_CONFIGS:
            print(f"[bench] workload {name}", file=sys.stderr, flush=True)
            gc = generate(name)
            cc = layer_config(gc["cfg"])
            dc = DeviceLayer(cc, gc["X"], gc["valid"], gc["W_router"], gc["prototypes"], gc["W_up"], gc["W_down"])
            sc = max(2, args.steps // 2) if cc["n_tokens"] > 100000 else args.steps
            msc, evc, phc = measure(torch, _lib, dc, cc, sc, args.warmup, stream)
            stc = dc.stats()
            entry = summarize(cc, stc, _lib.forward_work(cc, dc.ws_forward), evc, phc)
            entry.update(steps=sc, ms_per_step=round(msc, 4),
                         shape=f"{cc['n_tokens']} tokens x d={cc['d_model']}, K={cc['n_experts']}, "
                               f"B={cc['n_blocks']} x M={cc['block_width']}, t={cc['mass_threshold']}")
            out["configs"][name] = entry
            del dc, gc
            torch.cuda.empty_cache()
    if not args.no_ablations and args.workload == "vit_b16":
        # The routing variants of the ablation table on the same tokens and
        # weights: a fixed shared demand alpha = 0.4, top-2 residual experts,
        # prefix instead of prototype block selection.
        out["ablations"] = {}
        for name, over in (("fixed_alpha_0.4", dict(alpha_mode="fixed", alpha_fixed=0.4)),
                           ("top2_residual", dict(mass_mode="topk", fixed_k=2)),
                           ("prefix_selection", dict(select_mode="prefix"))):
            print(f"[bench] ablation {name}", file=sys.stderr, flush=True)
            ca = dict(cfg, **over)
            da = DeviceLayer(ca, g["X"], g["valid"], g["W_router"], g["prototypes"], g["W_up"], g["W_down"])
            sa = max(2, args.steps // 2)
            msa, eva, pha = measure(torch, _lib, da, ca, sa, args.warmup, stream)
            sta = da.stats()
            ea = summarize(ca, sta, _lib.forward_work(ca, da.ws_forward), eva, pha)
            out["ablations"][name] = {k: ea[k] for k in ("tokens_per_s", "ms_per_step_event_median", "mean_b",
                                                         "mean_k", "mean_cb", "activated_gemm_tflop",
                                                         "mfma_util_activated", "executed_vs_activated",
                                                         "phases_ms")}
            del da
            torch.cuda.empty_cache()
        # The post-LN block (as in BERT) on the paper's BERT-large shape:
        # the FFN input is the previous LayerNorm's output; LN(x + F(x)).
        print("[bench] post-LN block (paper_language)", file=sys.stderr, flush=True)
        from synth import block_inputs
        gl = generate("paper_language")
        cl = layer_config(gl["cfg"])
        dl = DeviceLayer(cl, gl["X"], gl["valid"], gl["W_router"], gl["prototypes"], gl["W_up"], gl["W_down"])
        msl, evl, _ = measure(torch, _lib, dl, cl, args.steps, args.warmup, stream)
        blkl, Xl = block_inputs(gl, "post", residual=True, eps=1e-12)
        bl = dict(norm="post", residual=True, ln_eps=float(blkl["ln_eps"]))
        for k in ("ln_gamma", "ln_beta", "b_up", "b_down"):
            bl[k] = torch.from_numpy(blkl[k]).to(dl.device)
        Xld = torch.from_numpy(Xl.view(np.int16)).view(torch.bfloat16).to(dl.device)
        wsl = _lib.alloc_workspace(_lib.block_forward_workspace_size(cl, bl), dl.device)

        def post_step():
            _lib.block_forward(cl, bl, Xld, dl.valid, dl.W_router, dl.prototypes, dl.W_up, dl.W_down, dl.Y, wsl,
                               routing=dl.routing, stream=stream)
        for _ in range(args.warmup):
            post_step()
        torch.cuda.synchronize()
        evp = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        for a, b in evp:
            a.record(stream)
            post_step()
            b.record(stream)
        torch.cuda.synchronize()
        msp = median([a.elapsed_time(b) for a, b in evp])
        stl = dl.stats()
        out["block_post_ln"] = {"workload": "paper_language (4096 slots, d=1024, K=16, B=16 x M=256, t=1)",
                                "ms_per_step_event_median": round(msp, 4),
                                "tokens_per_s": round(stl["n_valid"] / (msp / 1e3), 1),
                                "layer_ms_event_median": round(evl, 4), "over_layer_ms": round(msp - evl, 4)}
        del dl, gl, wsl, Xld, bl
        torch.cuda.empty_cache()
    out["clocks"] = clock.stop()
    if not args.no_block:
        # The pre-LN block (as in DeiT) around the same layer: LN(x) feeds
        # routing and experts, b1 and b2 are added, and x is added back.
        print("[bench] pre-LN block", file=sys.stderr, flush=True)
        from synth import block_inputs
        blk, Xb = block_inputs(g, "pre", residual=True, eps=1e-6)
        Xd = torch.from_numpy(Xb.view(np.int16)).view(torch.bfloat16).to(dev.device)
        bd = dict(norm="pre", residual=True, ln_eps=float(blk["ln_eps"]))
        for k in ("ln_gamma", "ln_beta", "b_up", "b_down"):
            bd[k] = torch.from_numpy(blk[k]).to(dev.device)
        dev.ws_forward = None
        torch.cuda.empty_cache()
        wsb = _lib.alloc_workspace(_lib.block_forward_workspace_size(cfg, bd), dev.device)
        stepsb = max(2, args.steps // 2)

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
        torch.cuda.empty_cache()
    if not args.no_backward:
        # Gradients of sum(dY * Y) for the layer (forward recomputed inside).
        # Algorithmic work: four products of 2 d M per activated block (dh,
        # dx, dW_up, dW_down), i.e. 8 d M sum(C_B).
        print("[bench] backward", file=sys.stderr, flush=True)
        from synth import upstream_grad
        dev.ws_forward = None
        torch.cuda.empty_cache()
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
        bwd_step()
        torch.cuda.synchronize()
        stepsg = 3
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(stepsg)]
        for a, b in ev:
            a.record(stream)
            bwd_step()
            b.record(stream)
        torch.cuda.synchronize()
        msg = median([a.elapsed_time(b) for a, b in ev])
        bflops = 8.0 * cfg["d_model"] * cfg["block_width"] * st["activated_blocks"]
        # The Gram diversity loss of the router (Eq. diversity-loss) and its
        # gradient added to dW_router, as in a training step.
        wsd = _lib.alloc_workspace(_lib.diversity_loss_workspace_size(cfg), dev.device)
        lossd = torch.zeros(1, dtype=torch.float32, device=dev.device)
        _lib.diversity_loss(cfg, dev.W_router, 0.01, lossd, gr["dW_router"], wsd, stream=stream)
        evd = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(5)]
        for a, b in evd:
            a.record(stream)
            _lib.diversity_loss(cfg, dev.W_router, 0.01, lossd, gr["dW_router"], wsd, stream=stream)
            b.record(stream)
        torch.cuda.synchronize()
        msd = median([a.elapsed_time(b) for a, b in evd])
        out["backward"] = {
            "ms_per_step": round(msg, 3), "steps": stepsg, "over_forward": round(msg / ms_event, 2),
            "diversity_loss_ms": round(msd, 4), "diversity_loss": round(float(lossd.item()), 6),
            "algorithmic_tflop": round(bflops / 1e12, 4),
            "achieved_tflops": round(bflops / (msg / 1e3) / 1e12, 2),
            "workspace_gb": round(wsg.numel() / 1e9, 2)}
        del wsg, gr, dYd, wsd
        torch.cuda.empty_cache()
    if args.vendor_reference:
        print("[bench] vendor reference GEMMs", file=sys.stderr, flush=True)
        out["vendor_reference"] = vendor_reference(torch, cfg, st)
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
        base, check = cpu_baseline_and_sample_check(g, Y_head, rec_head, args.cpu_sample, args.cpu_repeats)
        out["cpu_baseline"] = base
        out["parity_on_sample"] = check
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
