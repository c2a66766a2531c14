"""Throughput of MM-ShiftKV prefill-stage KV selection on one MI355X.

A step is the whole hot path for every layer of one batch of synthetic
inputs: proxies -> row log-sum-exp pass -> mass pass -> tau-sets / votes /
top-k -> K/V gather, through the C ABI, inputs resident in HBM.  Default
workload: 28 layers, batch 4, 28 query / 4 KV heads, d=128, T=16384 prompt
keys (16128 visual + 256 text), W=64 window queries, budget 256 per KV
head, the paper's method settings (P=512, G=32, gamma=10, tau=0.95,
lambda=1, vote mode).

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--streams N]

The layers of a step are independent, so the throughput steps spread them
over N HIP streams (layer l on stream l % N, default 4: one per hardware queue): the latency-bound
selection kernels and the tails of one layer's score passes then overlap
another layer's work.  The score-pass durations for the roofline come from
K further steps on one stream, where no other kernel shares the GPU.

Prints one JSON line: keys scored+selected per second (B*L*T / step time),
the roofline of the dominant kernel (algorithmic MFMA flops per launch /
launch time, events on the launch stream) and the CPU oracle timed on a
bounded sample of the same workload.

Other modes, one JSON line each: --decode-check N_DEC (the decode-time
coverage check), --selectors N_DEC (the method beside the baseline
selectors on the same kernels), --hidden (the hidden-state form of the
proxies in front of the same scoring and selection).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
SPIN_CYCLES = 20_000_000      # GPU spin ahead of the stage timings (several ms)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_score_qwen7b_16k_b4.json")
SCORE_SRC = os.path.join(ROOT, "paper_2607_22586_amd", "csrc", "score.hip")


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def measured_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` (score_lse, score_mass, ...) from the
    committed rocprofv3 counter summary, or None when it is missing, for
    another workload or kernel, or older than the current kernel source."""
    import hashlib
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
        with open(SCORE_SRC, "rb") as f:
            src = hashlib.sha256(f.read()).hexdigest()
    except (OSError, ValueError):
        return None
    if t.get("workload") != workload or t.get("score_hip_sha256") != src:
        return None
    k = t.get("kernels", {}).get(kernel)
    if k is None or k.get("hbm_bytes_per_launch") is None:
        return None
    return k["hbm_bytes_per_launch"]


def measured_mfma_util(workload):
    """MFMA busy fraction (and clock) of the two score kernels from the committed
    counter summary, or None under the same conditions as measured_traffic."""
    import hashlib
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
        with open(SCORE_SRC, "rb") as f:
            src = hashlib.sha256(f.read()).hexdigest()
    except (OSError, ValueError):
        return None
    if t.get("workload") != workload or t.get("score_hip_sha256") != src:
        return None
    k = t.get("kernels", {})
    try:
        return {p: {"mfma_busy": k[p]["mfma_busy"], "valu_busy": k[p]["valu_busy"], "clock_ghz": k[p]["clock_ghz"]}
                for p in ("score_lse", "score_mass")} | {"source": "profiles/counters_score_qwen7b_16k_b4.md"}
    except KeyError:
        return None


def calibrate_copy(nbytes=1 << 30, reps=5):
    """A plain device copy of known size, profiled with the FETCH_SIZE /
    WRITE_SIZE counters to scale them to bytes."""
    import torch
    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda:0").fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": nbytes, "copy_bytes_written": nbytes, "reps": reps}), flush=True)


def cpu_baseline(w, cfg, layer_inputs, heads=1):
    """The fp64 CPU oracle on `heads` (batch row, KV head) pairs of layer 0."""
    import oracle
    from paper_2607_22586_amd import workloads as wl
    oracle.build()
    Gh = w.Gh
    t0 = time.perf_counter()
    for i in range(heads):
        b, c = i % w.B, (i // w.B) % w.Hkv
        q1 = wl.to_numpy_bits(layer_inputs["q_win"][b:b + 1, c * Gh:(c + 1) * Gh].contiguous())
        k1 = wl.to_numpy_bits(layer_inputs["k"][b:b + 1, c:c + 1].contiguous())
        v1 = wl.to_numpy_bits(layer_inputs["v"][b:b + 1, c:c + 1].contiguous())
        prox, ql, _ = oracle.build_proxies(q1, cfg.P, cfg.gamma, cfg.seed, 0, b0=b, h0=c * Gh)
        gm, mass, an = oracle.score(prox, ql, k1, 1, cfg.G)
        sel = oracle.select(gm, mass, an, w.budget, cfg.tau, cfg.lam, mode=cfg.mode)
        oracle.gather(k1, sel.idx, sel.counts)
        oracle.gather(v1, sel.idx, sel.counts)
    dt = time.perf_counter() - t0
    keys = heads / w.Hkv * w.T          # one KV head covers 1/Hkv of a sequence-layer's keys
    return {"value": keys / dt, "unit": "prompt keys/s", "cores": oracle.num_threads(), "kind": "oracle",
            "nproc": os.cpu_count(), "cpu_model": cpu_model(),
            "sample": "%d (batch row, KV head) pair(s) of layer 0, T=%d, all steps; %.1f s"
                      % (heads, w.T, dt)}


def cpu_model():
    """The host CPU's model name (first entry of /proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def decode_check_bench(args):
    """The decode-time check (Fig. 1b's attention-mass coverage of decode
    queries on the kept prompt keys, and decode attention over the compacted
    cache): the selection path runs once per layer, then K steps time the
    check over all layers on one stream.  One JSON line."""
    import torch
    from paper_2607_22586_amd import binding as bd
    from paper_2607_22586_amd import workloads as wl
    bd.load_library()
    dev = torch.device("cuda:0")
    w = wl.WORKLOADS[args.workload]
    L = args.layers or w.L
    n = args.decode_check
    B, Hq, Hkv, T, W, d = w.B, w.Hq, w.Hkv, w.T, w.W, w.d
    log("generating %d layers of %s with %d decode queries per head" % (L, w.name, n))
    layers = [wl.make_layer(w, l, device=dev, n_dec=n) for l in range(L)]
    sels = []
    for l, x in enumerate(layers):
        cfg = bd.SelectionConfig(seed=w.wid, layer=l)
        out = bd.select_layer(x["q_win"], x["k"], x["v"], w.budget, cfg)
        sels.append(out)
    ws = torch.empty(bd.decode_workspace(B, Hq, Hkv, T, d, n), dtype=torch.uint8, device=dev)
    res = [(torch.empty((B, Hq, n), dtype=torch.float32, device=dev),
            torch.empty((B, Hq, n, d), dtype=torch.float32, device=dev)) for _ in range(L)]

    def step(ev=None):
        for l in range(L):
            if ev is not None:
                ev[l][0].record()
            bd.decode_check(layers[l]["q_dec"], layers[l]["k"], sels[l].sel, sels[l].k_out, sels[l].v_out,
                            workspace=ws, out=res[l])
            if ev is not None:
                ev[l][1].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ev = [[[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(L)] for _ in range(args.steps)]
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for s_ in range(args.steps):
        step(ev[s_])
    t1.record()
    torch.cuda.synchronize()
    ms_step = t0.elapsed_time(t1) / args.steps
    call_ms = sum(ev[s_][l][0].elapsed_time(ev[s_][l][1]) for s_ in range(args.steps) for l in range(L)) / (args.steps * L)
    eb = layers[0]["k"].element_size()
    c_max = sels[0].sel.idx.shape[2]
    # algorithmic bytes of one call: K once, the decode queries, the compacted
    # K'/V' and indices, the outputs
    nbytes = (B * Hkv * T * d * eb + B * Hq * n * d * 2 + 2 * B * Hkv * c_max * d * eb + B * Hkv * c_max * 4
              + B * Hq * n * (d + 1) * 4)
    achieved = nbytes / (call_ms * 1e-3) / 1e9
    cov = torch.stack([r[0] for r in res]).double()
    out = {
        "metric": "decode queries checked/sec",
        "value": B * Hq * n * L / (ms_step * 1e-3),
        "unit": "queries/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "us_per_layer": ms_step * 1e3 / L, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "layers": L, "batch": B, "T": T, "Hq": Hq, "Hkv": Hkv, "d": d,
                   "budget": w.budget, "n_dec": n, "decode_var_scale": wl.DECODE_VAR_SCALE},
        "coverage": {"mean": float(cov.mean()), "min": float(cov.min()), "max": float(cov.max())},
        "roofline": {"kernel": "decode check call (decode_scale_kernel + decode_cover_kernel + decode_attend_mfma_kernel)",
                     "bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBS, "traffic": None,
                     "bytes_per_call": nbytes, "us_per_call": call_ms * 1e3},
    }
    print(json.dumps(out), flush=True)


def selectors_bench(args):
    """The method and the baseline selectors (LastAttn = tau 1, SnapKV,
    StreamingLLM, ExpectedAttn) on the same kernels: per selector, K timed
    steps of its whole selection path over all layers on one stream, and the
    mean decode-time coverage of its kept keys (the synthetic analogue of
    Fig. 1b) for N_DEC decode queries per head.  One JSON line."""
    import torch
    from paper_2607_22586_amd import binding as bd
    from paper_2607_22586_amd import workloads as wl
    bd.load_library()
    dev = torch.device("cuda:0")
    w = wl.WORKLOADS[args.workload]
    L = args.layers or w.L
    n_dec = args.selectors
    B, Hq, Hkv, T, W, d = w.B, w.Hq, w.Hkv, w.T, w.W, w.d
    log("generating %d layers of %s" % (L, w.name))
    layers = [wl.make_layer(w, l, device=dev, n_dec=n_dec) for l in range(L)]

    def run(name, l):
        x = layers[l]
        if name in ("mm-shiftkv", "lastattn"):
            cfg = bd.SelectionConfig(seed=w.wid, layer=l, tau=1.0 if name == "lastattn" else 0.95)
            o = bd.select_layer(x["q_win"], x["k"], x["v"], w.budget, cfg)
            return o.sel, o.k_out, o.v_out
        sel, _, _, ko, vo = bd.baseline_select(name, x["q_win"], x["k"], x["v"], w.budget, seed=w.wid, layer=l)
        return sel, ko, vo

    res = {}
    for name in ("mm-shiftkv", "lastattn", "snapkv", "expected", "streaming"):
        for _ in range(args.warmup):
            for l in range(L):
                run(name, l)
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record()
        for _ in range(args.steps):
            for l in range(L):
                run(name, l)
        t1.record()
        torch.cuda.synchronize()
        ms = t0.elapsed_time(t1) / args.steps
        covs = []
        for l in range(L):
            sel, ko, vo = run(name, l)
            cov, _ = bd.decode_check(layers[l]["q_dec"], layers[l]["k"], sel, ko, vo)
            covs.append(cov.double())
        cov = torch.stack(covs)
        res[name] = {"us_per_layer": ms * 1e3 / L, "keys_per_s": B * L * T / (ms * 1e-3),
                     "coverage_mean": float(cov.mean()), "coverage_p10": float(torch.quantile(cov.flatten().float(), 0.1))}
        log("%s: %.1f us/layer, coverage %.4f" % (name, ms * 1e3 / L, res[name]["coverage_mean"]))
    out = {
        "metric": "selectors on the same kernels: throughput and decode-time coverage",
        "value": res["mm-shiftkv"]["coverage_mean"], "unit": "mean coverage (mm-shiftkv)",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "higher_is_better": True,
        "data": "synthetic", "dtype": "bf16",
        "config": {"workload": w.name, "layers": L, "batch": B, "T": T, "Hq": Hq, "Hkv": Hkv, "d": d,
                   "budget": w.budget, "n_dec": n_dec, "decode_var_scale": wl.DECODE_VAR_SCALE,
                   "snapkv": {"window": 32, "pool": 5}, "streaming": {"sinks": 4},
                   "expected": {"samples": 512, "gamma": 1.0, "sinks": 4}, "lastattn": {"tau": 1.0}},
        "selectors": res,
    }
    print(json.dumps(out), flush=True)


def hidden_bench(args):
    """The hidden-state form of the proxies (Sec. 3.2.1 Eqs. 4-6, Algorithm 1)
    in front of the same scoring, selection and gather: per layer, the
    statistics of the T prefill hidden states, the hidden-space samples and
    their projection by every head's W_Q replace the query-space proxy call.
    K steps over all layers on one stream, events around every call; the
    roofline is taken for the slowest of the three hidden-path calls.  The
    hidden states of HIDDEN_LAYERS distinct layers (470 MiB each at the 16k
    batch-4 shape, more than the last-level cache) are reused cyclically.
    One JSON line."""
    import torch
    from paper_2607_22586_amd import binding as bd
    from paper_2607_22586_amd import workloads as wl
    bd.load_library()
    dev = torch.device("cuda:0")
    w = wl.WORKLOADS[args.workload]
    L = args.layers or w.L
    nh = max(1, min(L, args.hidden_layers))
    B, Hq, Hkv, T, W, d = w.B, w.Hq, w.Hkv, w.T, w.W, w.d
    D = Hq * d
    cfgs = [bd.SelectionConfig(seed=w.wid, layer=l) for l in range(L)]
    cfg = cfgs[0]
    log("generating %d layers of %s and %d hidden-state layers" % (L, w.name, nh))
    layers = [wl.make_layer(w, l, device=dev) for l in range(L)]
    hid = [wl.make_hidden(w, l, device=dev) for l in range(nh)]
    torch.cuda.synchronize()
    st = torch.empty((B, 2, D), dtype=torch.float64, device=dev)
    ws_st = torch.empty(bd.hidden_stats_workspace(B, T, D), dtype=torch.uint8, device=dev)
    hp = torch.empty((B, cfg.P, D), dtype=torch.bfloat16, device=dev)
    prox = torch.empty((B, Hq, cfg.P, d), dtype=torch.bfloat16, device=dev)
    sc = bd.ScoreOut(torch.empty((B, Hkv, cfg.G, T), dtype=torch.float32, device=dev),
                     torch.empty((B, Hkv, T), dtype=torch.float32, device=dev),
                     torch.empty((B, Hkv, T), dtype=torch.float32, device=dev))
    ws_score = torch.empty(bd.score_workspace(B, Hq, Hkv, T, W, d, cfg), dtype=torch.uint8, device=dev)
    ws_sel = torch.empty(bd.select_workspace(B, Hq, Hkv, T, W, d, cfg), dtype=torch.uint8, device=dev)
    sel = bd.Selected(torch.empty((B, Hkv, w.budget), dtype=torch.int32, device=dev),
                      torch.empty((B, Hkv), dtype=torch.int32, device=dev), None)
    kv_out = (torch.empty((B, Hkv, w.budget, d), dtype=layers[0]["k"].dtype, device=dev),
              torch.empty((B, Hkv, w.budget, d), dtype=layers[0]["k"].dtype, device=dev))
    names = ("hidden_stats", "hidden_proxies", "project_proxies", "score_select_gather")

    def step(ev=None):
        for l in range(L):
            x, hx, c = layers[l], hid[l % nh], cfgs[l]
            if ev is not None:
                ev[l][0].record()
            bd.hidden_stats(hx["hidden"], out=st, workspace=ws_st)
            if ev is not None:
                ev[l][1].record()
            bd.hidden_proxies(st, c, T, out=hp)
            if ev is not None:
                ev[l][2].record()
            bd.project_proxies(hp, hx["wq"], Hq, out=prox)
            if ev is not None:
                ev[l][3].record()
            bd.score_lse(prox, hx["q_last"], x["k"], c, ws_score, W)
            bd.score_mass(prox, hx["q_last"], x["k"], c, ws_score, W, out=sc)
            bd.select_topk(sc, c, w.budget, w.budget, None, Hq, W, out=sel, workspace=ws_sel)
            bd.gather_kv(x["k"], x["v"], sel, out=kv_out)
            if ev is not None:
                ev[l][4].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(args.steps):
        step()
    t1.record()
    torch.cuda.synchronize()
    ms_step = t0.elapsed_time(t1) / args.steps
    ev = [[[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(L)] for _ in range(args.steps)]
    for s_ in range(args.steps):
        step(ev[s_])
    torch.cuda.synchronize()
    us = {n: 1e3 * sum(ev[s_][l][i].elapsed_time(ev[s_][l][i + 1]) for s_ in range(args.steps) for l in range(L))
          / (args.steps * L) for i, n in enumerate(names)}
    # algorithmic work per call: the statistics read the hidden states once
    # and write mean / std; the projection is a (B*P) x D by D x (Hq*d)
    # product.  The samples (the generator, as in the query-space proxy
    # call) are ALU work and are reported by time only.
    hb = hid[0]["hidden"].element_size()
    rl = {
        "hidden_stats": {"bound": "hbm", "work": B * T * D * hb + B * 2 * D * 8, "peak": PEAK_HBM_GBS,
                         "unit": "GB/s"},
        "project_proxies": {"bound": "mfma", "work": 2.0 * B * cfg.P * D * Hq * d, "peak": PEAK_BF16_TFLOPS,
                            "unit": "TFLOP/s"},
    }
    for n, r in rl.items():
        scale = 1e9 if r["unit"] == "GB/s" else 1e12
        r["achieved"] = r["work"] / (us[n] * 1e-6) / scale
        r["frac"] = r["achieved"] / r["peak"]
        r["us_per_call"] = us[n]
    dom = max(rl, key=lambda n: us[n])
    r = rl[dom]
    out = {
        "metric": "prompt keys scored+selected/sec (hidden-state proxies)",
        "value": B * L * T / (ms_step * 1e-3), "unit": "keys/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "us_per_layer": ms_step * 1e3 / L, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "layers": L, "hidden_layers": nh, "batch": B, "T": T, "D": D,
                   "Hq": Hq, "Hkv": Hkv, "d": d, "P": cfg.P, "G": cfg.G, "budget": w.budget,
                   "proxies": "hidden-state (Eqs. 4-6)", "streams": 1},
        "stages_us_per_layer": us,
        "roofline": {"kernel": dom, "bound": r["bound"], "achieved": r["achieved"], "peak": r["peak"],
                     "unit": r["unit"], "frac": r["frac"], "traffic": None},
        "hidden_rooflines": rl,
    }
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="qwen7b_16k_b4")
    ap.add_argument("--layers", type=int, default=0, help="override the layer count (0 = workload's)")
    ap.add_argument("--mode", choices=["vote", "mass"], default="vote")
    ap.add_argument("--cpu-heads", type=int, default=12)
    ap.add_argument("--streams", type=int, default=4,
                    help="HIP streams the layers are spread over in the throughput steps "
                         "(layer l on stream l %% n); the kernel-timing steps use one")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--decode-check", type=int, default=0, metavar="N_DEC",
                    help="time the decode-time coverage check with N_DEC decode queries per head instead")
    ap.add_argument("--selectors", type=int, default=0, metavar="N_DEC",
                    help="compare the method with the baseline selectors (throughput and decode-time "
                         "coverage with N_DEC decode queries per head) instead")
    ap.add_argument("--hidden", action="store_true",
                    help="time the hidden-state form of the proxies (statistics, samples, W_Q projection) "
                         "in front of the same scoring, selection and gather")
    ap.add_argument("--hidden-layers", type=int, default=4,
                    help="distinct hidden-state layers generated for --hidden (reused cyclically)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a 1 GiB device copy (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the selection path is independent per (layer, KV head) and "
              "needs no collectives; --gpus %d is not supported" % args.gpus, file=sys.stderr)
        sys.exit(2)

    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.decode_check > 0:
        decode_check_bench(args)
        return
    if args.selectors > 0:
        selectors_bench(args)
        return
    if args.hidden:
        hidden_bench(args)
        return

    import torch

    from paper_2607_22586_amd import binding as bd
    from paper_2607_22586_amd import workloads as wl

    if not os.path.exists(bd.LIB_PATH):
        from paper_2607_22586_amd import build
        build.build()
    bd.load_library()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = wl.WORKLOADS[args.workload]
    L = args.layers or w.L
    B, Hq, Hkv, T, W, d = w.B, w.Hq, w.Hkv, w.T, w.W, w.d
    mode = bd.MMSKV_VOTE if args.mode == "vote" else bd.MMSKV_MASS
    cfgs = [bd.SelectionConfig(seed=w.wid, layer=l, mode=mode) for l in range(L)]
    cfg = cfgs[0]

    log("generating %d layers of %s on the device" % (L, w.name))
    layers = [wl.make_layer(w, l, device=dev) for l in range(L)]
    torch.cuda.synchronize()
    log("inputs ready: %.2f GiB" % (sum(x["k"].numel() * 2 * x["k"].element_size() for x in layers) / 2**30))

    # preallocated outputs and workspaces, one set per stream (reused by the
    # layers of that stream)
    def buffers():
        return dict(
            prox=torch.empty((B, Hq, cfg.P, d), dtype=torch.bfloat16, device=dev),
            qlast=torch.empty((B, Hq, d), dtype=torch.bfloat16, device=dev),
            sc=bd.ScoreOut(torch.empty((B, Hkv, cfg.G, T), dtype=torch.float32, device=dev) if mode == 0 else None,
                           torch.empty((B, Hkv, T), dtype=torch.float32, device=dev),
                           torch.empty((B, Hkv, T), dtype=torch.float32, device=dev)),
            ws_score=torch.empty(bd.score_workspace(B, Hq, Hkv, T, W, d, cfg), dtype=torch.uint8, device=dev),
            ws_sel=torch.empty(bd.select_workspace(B, Hq, Hkv, T, W, d, cfg), dtype=torch.uint8, device=dev),
            sel=bd.Selected(torch.empty((B, Hkv, w.budget), dtype=torch.int32, device=dev),
                            torch.empty((B, Hkv), dtype=torch.int32, device=dev), None))
    n_streams = max(1, args.streams)
    bufs = [buffers() for _ in range(n_streams)]
    kv_out = [(torch.empty((B, Hkv, w.budget, d), dtype=layers[0]["k"].dtype, device=dev),
               torch.empty((B, Hkv, w.budget, d), dtype=layers[0]["k"].dtype, device=dev)) for _ in range(L)]
    stream = torch.cuda.current_stream(dev)
    # extra streams at the default priority
    streams = [stream] + [torch.cuda.Stream(dev) for _ in range(n_streams - 1)]

    def step(events=None, n=n_streams):
        for s in streams[1:n]:
            s.wait_stream(stream)
        for l in range(L):
            x = layers[l]
            c = cfgs[l]
            s = streams[l % n]
            bf = bufs[l % n]
            with torch.cuda.stream(s):
                bd.build_proxies(x["q_win"], c, T, Hkv, out=(bf["prox"], bf["qlast"]))
                if events is None:
                    bd.score_lse(bf["prox"], bf["qlast"], x["k"], c, bf["ws_score"], W)
                else:
                    # the log-sum-exp pass as its two calls, so that the events
                    # bracket score_lse_kernel alone, then the merge kernel
                    events[l][0].record(s)
                    bd.score_lse(bf["prox"], bf["qlast"], x["k"], c, bf["ws_score"], W, stage="blocks")
                    events[l][1].record(s)
                    bd.score_lse(bf["prox"], bf["qlast"], x["k"], c, bf["ws_score"], W, stage="merge")
                    events[l][2].record(s)
                bd.score_mass(bf["prox"], bf["qlast"], x["k"], c, bf["ws_score"], W, out=bf["sc"])
                if events is not None:
                    events[l][3].record(s)
                bd.select_topk(bf["sc"], c, w.budget, w.budget, None, Hq, W, out=bf["sel"], workspace=bf["ws_sel"])
                bd.gather_kv(x["k"], x["v"], bf["sel"], out=kv_out[l])
        for s in streams[1:n]:
            stream.wait_stream(s)

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        log("warmup step %d done" % (i + 1))

    # throughput: K whole steps, layers spread over the streams
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(stream)
    for s in range(args.steps):
        step()
    t_end.record(stream)
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    ms_step = total_ms / args.steps
    log("timed %d steps on %d stream(s): %.3f ms/step" % (args.steps, n_streams, ms_step))

    # kernel timing: one more warmup and K steps on one stream, with events
    # around score_lse_kernel (mmshiftkv_score_lse_blocks), the merge of its
    # partials (mmshiftkv_score_lse_merge) and score_mass_kernel
    # (mmshiftkv_score_mass) of every layer (un-overlapped durations)
    step(n=1)
    ev = [[[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(L)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    for s in range(args.steps):
        step(ev[s], n=1)
    torch.cuda.synchronize()

    def ev_ms(i, j):
        return sum(ev[s][l][i].elapsed_time(ev[s][l][j]) for s in range(args.steps) for l in range(L)) / (args.steps * L)
    lse_ms, merge_ms, mass_ms = ev_ms(0, 1), ev_ms(1, 2), ev_ms(2, 3)
    log("kernel timing on one stream: score_lse_kernel %.1f us, merge %.1f us, score_mass_kernel %.1f us per layer"
        % (lse_ms * 1e3, merge_ms * 1e3, mass_ms * 1e3))

    # the other stages: each C-ABI call repeated back to back on one stream
    # (layer 0's inputs, the buffers of stream 0) behind a GPU-side spin long
    # enough for the host to queue all of them, so the time per call is its
    # kernels plus the launch gaps between them (not the host's call cost)
    x, c, bf = layers[0], cfgs[0], bufs[0]
    sel_args = (bf["sc"], c, w.budget, w.budget, None, Hq, W)
    calls = {
        "build_proxies": lambda: bd.build_proxies(x["q_win"], c, T, Hkv, out=(bf["prox"], bf["qlast"])),
        "select_tau": lambda: bd.select_topk(*sel_args, out=bf["sel"], workspace=bf["ws_sel"], stage="tau"),
        "select_vote": lambda: bd.select_topk(*sel_args, out=bf["sel"], workspace=bf["ws_sel"], stage="vote"),
        "select_pick": lambda: bd.select_topk(*sel_args, out=bf["sel"], workspace=bf["ws_sel"], stage="pick"),
        "gather": lambda: bd.gather_kv(x["k"], x["v"], bf["sel"], out=kv_out[0]),
    }
    reps = 20
    stage_ms = {}
    with torch.cuda.stream(stream):
        for name, fn in calls.items():
            if name == "select_pick":
                # the vote repetitions added to the first-digit counts: one
                # tau + vote pair restores the state the pick reads
                calls["select_tau"]()
                calls["select_vote"]()
            fn()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            es = torch.cuda.Event(enable_timing=True)
            es.record(stream)
            torch.cuda._sleep(SPIN_CYCLES)
            e0.record(stream)
            h0 = time.perf_counter()
            for _ in range(reps):
                fn()
            host_ms = (time.perf_counter() - h0) * 1e3
            e1.record(stream)
            torch.cuda.synchronize()
            spin_ms = es.elapsed_time(e0)
            if host_ms > spin_ms:
                log("warning: queuing %s took %.2f ms, longer than the %.2f ms spin: its time includes host "
                    "call cost" % (name, host_ms, spin_ms))
            stage_ms[name] = e0.elapsed_time(e1) / reps
        # leave layer 0's selection as a whole call made it
        bd.select_topk(*sel_args, out=bf["sel"], workspace=bf["ws_sel"])
        torch.cuda.synchronize()
    stage_ms = {"build_proxies": stage_ms["build_proxies"], "score_lse": lse_ms, "score_lse_merge": merge_ms,
                "score_mass": mass_ms, **{k: v for k, v in stage_ms.items() if k != "build_proxies"}}
    log("per call (us): " + ", ".join("%s %.1f" % (k, v * 1e3) for k, v in stage_ms.items()))

    # algorithmic MFMA work of one scoring launch: 2*Gh*P*d flops per prompt
    # key per KV head (one proxy-by-key contraction), times B*Hkv*T keys
    flops = 2.0 * w.Gh * cfg.P * d * B * Hkv * T
    # one launch = one kernel: score_lse = score_lse_kernel (mmshiftkv_score_lse_blocks),
    # score_mass = score_mass_kernel (mmshiftkv_score_mass)
    # algorithmic HBM bytes of the memory-bound stages, per layer (all heads)
    heads = B * Hkv
    eb = layers[0]["k"].element_size()
    words = (T + 31) // 32
    vote_mode = mode == bd.MMSKV_VOTE
    stage_bytes = {
        # masses read, membership planes written
        "select_tau": heads * (cfg.G * T * 4 + cfg.G * words * 4) if vote_mode else 0,
        # planes and anchor (or masses) read, fp64 score keys written
        "select_vote": heads * ((cfg.G * words * 4 + T * 4) if vote_mode else T * 4) + heads * T * 8,
        # score keys and first-digit counts read, indices written
        "select_pick": heads * (T * 8 + 2048 * 4 + w.budget * 4 + 4),
        # selected K and V rows read and written
        "gather": heads * w.budget * d * eb * 4,
    }
    stage_bytes = {k: v for k, v in stage_bytes.items() if v > 0}
    dom = "score_mass" if mass_ms >= lse_ms else "score_lse"
    dom_ms = max(mass_ms, lse_ms)
    achieved = flops / (dom_ms * 1e-3) / 1e12
    keys_per_s = B * L * T / (ms_step * 1e-3)
    out = {
        "metric": "prompt keys scored+selected/sec",
        "value": keys_per_s,
        "unit": "keys/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "us_per_layer": ms_step * 1e3 / L,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "layers": L, "batch": B, "T": T, "Hq": Hq, "Hkv": Hkv, "d": d, "W": W,
                   "budget": w.budget, "P": cfg.P, "G": cfg.G, "gamma": cfg.gamma, "tau": cfg.tau,
                   "lambda": cfg.lam, "mode": args.mode, "streams": n_streams},
        "stages_us_per_layer": {k: v * 1e3 for k, v in stage_ms.items()},
        "stages_timing": "score_lse (score_lse_kernel), score_lse_merge (lse_combine_kernel) and score_mass "
                         "(score_mass_kernel): events around each call in %d steps on one stream; the rest: %d "
                         "back-to-back calls of one stage on one stream, queued behind a GPU spin (kernels + launch "
                         "gaps)" % (args.steps, reps),
        "non_score_us_per_layer": sum(v for k, v in stage_ms.items()
                                      if k not in ("score_lse", "score_lse_merge", "score_mass")) * 1e3,
        "stage_hbm_frac": {k: stage_bytes[k] / (stage_ms[k] * 1e-3) / 1e9 / PEAK_HBM_GBS for k in stage_bytes},
        "roofline": {"kernel": dom + "_kernel", "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                     "traffic": measured_traffic(w.name, dom),
                     "timing": "%d steps on one stream after the throughput steps" % args.steps},
        "mfma_util_counter": measured_mfma_util(w.name),
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on %d head(s)" % args.cpu_heads)
        x0 = {k: (v.cpu() if torch.is_tensor(v) else v) for k, v in layers[0].items()}
        out["cpu_baseline"] = cpu_baseline(w, cfg, x0, args.cpu_heads)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
