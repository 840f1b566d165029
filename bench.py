#!/usr/bin/env python3
"""Throughput of the fused RL log-prob step on one MI355X.

One step = mc_logprob_fwd_cached (LM-head GEMM + online log-sum-exp +
target gather, keeping the softmax cache) -> mc_rl_loss (ratios, MirrorPop
filter, group advantages, clipped surrogate, dlogp) ->
mc_logprob_bwd_cached (dHidden and dW from the cache), on one stream, over
one packed batch of synthetic inputs already resident in HBM.  With
--recompute the step uses mc_logprob_fwd / mc_logprob_bwd instead (the
backward recomputes the logits).

Default workload: T = 16384 packed tokens (256 sequences in 32 groups of 8,
lengths 8-2048, 70% of tokens masked, 10% of sequences drifted), d = 4096,
V = 151936, bf16 operands with fp32 accumulation.

Prints one JSON line.  `value` is tokens/s; counted FLOPs are 2TdV forward
plus 4TdV backward; `mfma_frac` is counted FLOP/s over the dense bf16 peak.
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "fused logprob fwd+bwd tokens/s @ d=4096,V=151936; % bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2516.6     # 256 CUs x 4096 FLOP/clk x 2.4 GHz, dense bf16
PEAK_FP32_TFLOPS = 157.3

# HBM traffic per launch of the step's kernels from rocprofv3 FETCH_SIZE /
# WRITE_SIZE passes (scaled by the 1 GiB copy calibration), valid only for
# the kernel sources with this digest (else null).
TRAFFIC = {
    "sources_sha256":
        "4fd5ae0e70ff241c11156f6c4cd0eff374332b9ecf5b799e931b940bfc0eb1ae",
    "bytes_per_launch": {
        "logprob_fwd_gemm": 35759080788,
        "logprob_fwd_merge": 78294580,
        "rl_loss": 91896,
        "logprob_bwd_bucket": 1338976,
        "logprob_bwd_cache_probs": 6307710964,
        "logprob_bwd_transpose": 1378916044,
        "logprob_bwd_dhidden": 30274365503,
        "logprob_bwd_dweight": 32536170929,
        "logprob_bwd_onehot_dw": 176654837,
    },
}


def sources_digest() -> str:
    h = hashlib.sha256()
    for p in sorted(glob.glob(os.path.join(ROOT, "paper_2606_04847_amd", "csrc", "*"))):
        with open(p, "rb") as f:
            h.update(os.path.basename(p).encode())
            h.update(f.read())
    return h.hexdigest()


def workload_name(cfg, s):
    return (f"{cfg['name']}: T={s.T} packed tokens ({s.B} sequences, {s.NG} groups of "
            f"{cfg['group_size']}), d={cfg['d']}, V={cfg['V']}, {cfg['dtype']}")


def build_inputs(cid, dev):
    import torch
    import paper_2606_04847_amd as mc
    from workloads import CONFIGS, make_structure, make_tensors_torch, sample_targets_torch
    cfg = CONFIGS[cid]
    s = make_structure(cid)
    H, W = make_tensors_torch(cfg, s.T, dev)
    y = sample_targets_torch(cfg, H, W)
    logp, _ = mc.logprob_fwd(H, W, y)
    # rollout log-probs: the trainer's plus the workload's per-token offset
    lr = (logp.double() + torch.from_numpy(s.rollout_delta).to(dev).double()).float()
    st = dict(mask=torch.from_numpy(s.loss_mask).to(dev),
              cu=torch.from_numpy(s.cu_seqlens).to(dev),
              cg=torch.from_numpy(s.cu_groups).to(dev),
              rewards=torch.from_numpy(s.rewards).to(dev))
    torch.cuda.synchronize()
    return cfg, s, H, W, y, lr, st


def cpu_baseline(cid, H, W, y, s, target_s):
    """The fp64 oracle on a bounded leading sample of whole groups."""
    import numpy as np
    import oracle
    try:
        import threadpoolctl
        info = threadpoolctl.threadpool_info()
        cores = max([i.get("num_threads", 1) for i in info] + [1])
    except Exception:
        cores = len(os.sched_getaffinity(0))
    Wh = W.float().cpu().numpy()
    cu, cg = s.cu_seqlens, s.cu_groups

    def run(n_groups):
        nseq = int(cg[n_groups])
        n = int(cu[nseq])
        Hs = H[:n].float().cpu().numpy()
        ys = y[:n].cpu().numpy()
        t0 = time.perf_counter()
        logp, lse = oracle.logprob_fwd(Hs, Wh, ys)
        lr = logp + s.rollout_delta[:n].astype(np.float64)
        out = oracle.rl_loss(logp, lr, s.loss_mask[:n], cu[:nseq + 1], cg[:n_groups + 1],
                             s.rewards[:nseq], oracle.RLParams())
        oracle.logprob_bwd(Hs, Wh, ys, lse, out["dlogp"])
        return n, time.perf_counter() - t0

    n1, t1 = run(1)
    per_tok = t1 / n1
    groups = 1
    while groups < s.NG and int(cu[int(cg[groups + 1])]) * per_tok <= target_s:
        groups += 1
    n, t = (n1, t1) if groups == 1 else run(groups)
    return {"value": n / t, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": (f"first {groups} groups ({n} tokens) of the workload: fp64 oracle "
                       f"logprob_fwd + rl_loss + logprob_bwd (full dH rows and dW), "
                       f"{t:.1f} s wall")}


def main():
    ap = argparse.ArgumentParser(description=__doc__,
                                 formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=4, choices=[3, 4, 5])
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="target duration of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--recompute", action="store_true",
                    help="time the recompute path (mc_logprob_fwd / mc_logprob_bwd) instead "
                         "of the softmax-cache path")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a plain 1 GiB device copy three times (calibrates the "
                         "FETCH_SIZE / WRITE_SIZE counters against a known byte count)")
    args = ap.parse_args()
    if args.copy_probe:
        import torch
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_per_launch": src.numel() * 4}), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported by this "
              "single-GPU build (the multi-GPU sharding is a design note only).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2606_04847_amd as mc
    mc.load_library()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg, s, H, W, y, lr, st = build_inputs(args.config, dev)
    T, d, V = s.T, cfg["d"], cfg["V"]

    lib = mc.load_library()
    ws_f = torch.empty(lib.mc_logprob_fwd_workspace_size(T, d, V, 1), dtype=torch.uint8,
                       device=dev)
    if args.recompute:
        ws_b = torch.empty(lib.mc_logprob_bwd_workspace_size(T, d, V, 1), dtype=torch.uint8,
                           device=dev)
        cache = None
    else:
        ws_b = torch.empty(lib.mc_logprob_bwd_cached_workspace_size(T, d, V, 1),
                           dtype=torch.uint8, device=dev)
        cache = mc.softmax_cache(H, W)
    logp = torch.empty(T, dtype=torch.float32, device=dev)
    lse = torch.empty(T, dtype=torch.float32, device=dev)
    dH = torch.empty(T, d, dtype=torch.float32, device=dev)
    dW = torch.empty(V, d, dtype=torch.float32, device=dev)
    params = mc.RLParams()

    def step():
        if cache is None:
            mc.logprob_fwd(H, W, y, logp=logp, lse=lse, workspace=ws_f)
        else:
            mc.logprob_fwd_cached(H, W, y, cache, logp=logp, lse=lse, workspace=ws_f)
        out = mc.rl_loss(logp, lr, st["mask"], st["cu"], st["cg"], st["rewards"], params)
        if cache is None:
            mc.logprob_bwd(H, W, y, lse, out["dlogp"], dhidden=dH, dweight=dW, workspace=ws_b)
        else:
            mc.logprob_bwd_cached(H, W, y, lse, out["dlogp"], cache, dhidden=dH, dweight=dW,
                                  workspace=ws_b)
        return out

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print(f"[bench] warmup done ({args.warmup} steps), timing {args.steps}", file=sys.stderr,
          flush=True)

    mc.profiler_reset()
    mc.profiler_enable(True)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(args.steps):
        out = step()
    e1.record()
    torch.cuda.synchronize()
    mc.profiler_enable(False)
    kernels = mc.profiler_read()
    ms = e0.elapsed_time(e1) / args.steps
    n_valid = int(out["n_valid"].item())
    loss = float(out["loss"].item())

    counted = 6.0 * T * d * V
    tflops = counted / (ms * 1e-3) / 1e12
    dom_name, dom = max(kernels.items(), key=lambda kv: kv[1]["ms"])
    dom_ms = dom["ms"] / dom["launches"]
    achieved = dom["flops"] / (dom["ms"] * 1e-3) / 1e12
    traffic = None
    if TRAFFIC["sources_sha256"] == sources_digest():
        traffic = TRAFFIC["bytes_per_launch"].get(dom_name)
    roofline = {"bound": "mfma", "kernel": dom_name, "achieved": achieved,
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                "traffic": traffic, "avg_launch_ms": dom_ms,
                "algorithmic_flops_per_launch": dom["flops"] / dom["launches"]}
    phases = {k: {"ms_per_launch": v["ms"] / v["launches"], "launches": v["launches"],
                  "tflops": (v["flops"] / (v["ms"] * 1e-3) / 1e12) if v["flops"] else None,
                  "GBps_algorithmic": v["bytes"] / (v["ms"] * 1e-3) / 1e9}
              for k, v in sorted(kernels.items(), key=lambda kv: -kv[1]["ms"])}
    print(f"[bench] {ms:.3f} ms/step, {tflops:.1f} TFLOP/s counted", file=sys.stderr, flush=True)

    base = None
    if not args.no_cpu_baseline:
        print("[bench] timing the fp64 oracle baseline sample", file=sys.stderr, flush=True)
        base = cpu_baseline(args.config, H, W, y, s, args.cpu_seconds)

    line = {
        "metric": METRIC,
        "value": T / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": workload_name(cfg, s), "T": T, "d": d, "V": V,
                   "sequences": s.B, "groups": s.NG, "parallelism": "none (1 GPU)",
                   "backward": "recompute logits" if args.recompute else "softmax cache"},
        "mfma_frac": tflops / PEAK_BF16_TFLOPS,
        "counted_tflops": tflops,
        "roofline": roofline,
        "cpu_baseline": base,
        "kernels": phases,
        "loss": loss,
        "n_valid": n_valid,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
