#!/usr/bin/env python3
"""Throughput of the fused RL log-prob step on one MI355X.

One step = forward (LM-head GEMM + online log-sum-exp + target gather) ->
mc_rl_loss (ratios, MirrorPop filter, group advantages, clipped surrogate,
dlogp) -> backward (dHidden and dW), on one stream, over one packed batch of
synthetic inputs already resident in HBM.  Two steps are timed on the same
inputs in one process:

  recompute  mc_logprob_fwd / mc_logprob_bwd: the forward writes no [T, V]
             tensor (the logits live only in registers), the backward
             recomputes them.  This is the headline figure.
  cached     mc_logprob_fwd_cached / mc_logprob_bwd_cached: the forward also
             writes a [T, V] bf16 softmax cache that the backward reads
             instead of recomputing the logits (reported under "cached").

Default workload: T = 16384 packed tokens (256 sequences in 32 groups of 8,
lengths 8-2048, 70% of tokens masked, 10% of sequences drifted), d = 4096,
V = 151936, bf16 operands with fp32 accumulation.  Other modes:
  --config 2   forward only, T = 8192 (the 9B-class forward workload)
  --config 3|5 the 27B-class (d = 5120, T = 32768) and large-vocabulary
               (V = 248320, T = 65536) workloads
  --shard      one GPU's vocabulary shard (V / 8 entries) of the headline
               shape: shard forward (partials) and shard backward
  --targets zipf  Zipf-like targets (one bucket holds a fifth of the tokens)

Prints one JSON line.  `value` is tokens/s; counted FLOPs are 2TdV forward
plus 4TdV backward; `mfma_frac` is counted FLOP/s over the dense bf16 peak.
`python bench.py --summarize DIR` prints the per-kernel summary of a
rocprofv3 output directory (kernel trace or counters) instead.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import statistics
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "fused logprob fwd+bwd tokens/s @ d=4096,V=151936; % bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2516.6     # 256 CUs x 4096 FLOP/clk x 2.4 GHz, dense bf16
FLOP_PER_CLK = 256 * 4096     # dense bf16 FLOP per clock over the chip
PEAK_HBM_GBPS = 8000.0
FLUSH_BYTES = 1 << 30         # scratch write between flushed reps (> L2 + 256 MB MALL)

# Memory-side traffic per launch of the recompute step's kernels at the
# headline workload: rocprofv3 TCC_EA0_RDREQ_DRAM_32B_sum (reads) and
# TCC_EA0_WRREQ_WRITE_DRAM_32B_sum (writes), x 32 bytes; a 1 GiB device copy
# reads and writes exactly 1 GiB by these counters.  They count L2 misses
# that go to the memory side, so reads served by the 256 MB Infinity Cache
# are included: an upper bound on HBM bytes.  Valid only for kernel sources
# with this digest (else null).
TRAFFIC = {
    "sources_sha256":
        "820083f7ed703dc9d45c95f71e34b4faf478f0fbbaa2986bf6e5b92012caadf3",
    "read_bytes_per_launch": {
        "logprob_fwd_gemm": 37786938368,
        "logprob_fwd_merge": 78110848,
        "logprob_bwd_live_order": 436224,
        "logprob_bwd_live_rows": 37179776,
        "logprob_bwd_bounds": 76928,
        "logprob_bwd_bucket": 5807040,
        "logprob_bwd_probs": 11528877824,
        "logprob_bwd_transpose": 689524640,
        "logprob_bwd_dhidden": 23638051072,
        "logprob_bwd_dweight": 9204613184,
        "logprob_bwd_onehot_dw": 107669504,
        "rl_loss": 340480,
    },
    "write_bytes_per_launch": {
        "logprob_fwd_gemm": 78367680,
        "logprob_fwd_merge": 131072,
        "logprob_bwd_live_order": 66912,
        "logprob_bwd_live_rows": 134217728,
        "logprob_bwd_bounds": 32,
        "logprob_bwd_bucket": 2647584,
        "logprob_bwd_probs": 1322502784,
        "logprob_bwd_transpose": 689438720,
        "logprob_bwd_dhidden": 268435456,
        "logprob_bwd_dweight": 2556428288,
        "logprob_bwd_onehot_dw": 69888768,
        "rl_loss": 80896,
    },
}


def sources_digest() -> str:
    h = hashlib.sha256()
    for p in sorted(glob.glob(os.path.join(ROOT, "paper_2606_04847_amd", "csrc", "*"))):
        with open(p, "rb") as f:
            h.update(os.path.basename(p).encode())
            h.update(f.read())
    return h.hexdigest()


def traffic_of(name):
    if TRAFFIC["sources_sha256"] != sources_digest():
        return None
    r = TRAFFIC["read_bytes_per_launch"].get(name)
    w = TRAFFIC["write_bytes_per_launch"].get(name)
    if r is None or w is None:
        return None
    return r + w


def workload_name(cfg, s, extra=""):
    return (f"{cfg['name']}: T={s.T} packed tokens ({s.B} sequences, {s.NG} groups of "
            f"{cfg['group_size']}), d={cfg['d']}, V={cfg['V']}, {cfg['dtype']}{extra}")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# ---------------------------------------------------------------------------
# inputs
# ---------------------------------------------------------------------------
def build_inputs(cid, dev, targets="model"):
    import torch
    import paper_2606_04847_amd as mc
    from workloads import (CONFIGS, make_structure, make_tensors_torch, sample_targets_torch,
                           zipf_targets)
    cfg = CONFIGS[cid]
    s = make_structure(cid)
    H, W = make_tensors_torch(cfg, s.T, dev)
    if targets == "zipf":
        y = torch.from_numpy(zipf_targets(s.T, cfg["V"], seed=cfg["seed"])).to(dev)
    else:
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


# ---------------------------------------------------------------------------
# clock and power, sampled live through amdsmi while the timed region runs
# ---------------------------------------------------------------------------
class ClockSampler:
    def __init__(self, period_s=0.004):
        self.period = period_s
        self.ok = False
        self.samples = []
        try:
            import amdsmi
            amdsmi.amdsmi_init()
            self.smi = amdsmi
            self.h = amdsmi.amdsmi_get_processor_handles()[0]
            self._metrics()
            self.ok = True
        except Exception as e:   # no amdsmi, no permission: report null
            self.err = str(e)

    def _metrics(self):
        return self.smi.amdsmi_get_gpu_metrics_info(self.h)

    def _run(self):
        while not self.stop.is_set():
            try:
                m = self._metrics()
                clks = [c for c in m.get("current_gfxclks", []) if isinstance(c, (int, float))]
                if clks:
                    self.samples.append((sum(clks) / len(clks), m.get("current_socket_power")))
            except Exception:
                pass
            time.sleep(self.period)

    def start(self):
        if not self.ok:
            return
        self.samples = []
        self.m0 = self._metrics()
        self.stop = threading.Event()
        self.th = threading.Thread(target=self._run, daemon=True)
        self.th.start()

    def finish(self):
        if not self.ok:
            return None
        self.stop.set()
        self.th.join()
        m1 = self._metrics()
        if not self.samples:
            return None
        clk = [c for c, _ in self.samples]
        pw = [p for _, p in self.samples if isinstance(p, (int, float))]
        out = {"gfxclk_mhz_mean": statistics.fmean(clk), "gfxclk_mhz_min": min(clk),
               "gfxclk_mhz_max": max(clk), "samples": len(clk),
               "socket_power_w_mean": statistics.fmean(pw) if pw else None,
               "source": "amdsmi gpu_metrics current_gfxclks (mean over the 8 XCDs), "
                         "sampled every ~4 ms during the timed region"}
        d_acc = None
        try:
            d_acc = m1["accumulation_counter"] - self.m0["accumulation_counter"]
            d_ppt = m1["ppt_residency_acc"] - self.m0["ppt_residency_acc"]
            if d_acc > 0:
                out["power_limited_frac"] = d_ppt / d_acc
        except Exception:
            pass
        # the metrics table did not refresh during the region (seen on some
        # boxes: every sample identical, the accumulation counter still):
        # the reading is not a measurement of this region
        if (d_acc is not None and d_acc <= 0) or (len(clk) > 10 and min(clk) == max(clk)):
            out["stale"] = True
        return out


# ---------------------------------------------------------------------------
# timing
# ---------------------------------------------------------------------------
def time_steps(step, steps, warmup, sampler=None, flush=None, flush_reps=0):
    """Warm-up, then exactly `steps` steps in one region bracketed by
    synchronisation (per-step events inside for the median), with the
    library's per-kernel profiler on; then `flush_reps` more steps, each
    after a write of FLUSH_BYTES of scratch, timed one by one."""
    import torch
    import paper_2606_04847_amd as mc
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    mc.profiler_reset()
    mc.profiler_enable(True)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    if sampler:
        sampler.start()
    torch.cuda.synchronize()
    ev[0].record()
    out = None
    for k in range(steps):
        out = step()
        ev[k + 1].record()
    torch.cuda.synchronize()
    clock = sampler.finish() if sampler else None
    mc.profiler_enable(False)
    kernels = mc.profiler_read()
    per = [ev[k].elapsed_time(ev[k + 1]) for k in range(steps)]
    res = {"ms_per_step": ev[0].elapsed_time(ev[steps]) / steps,
           "median_ms": statistics.median(per), "min_ms": min(per), "max_ms": max(per),
           "kernels": kernels, "clock": clock, "out": out}
    if flush is not None and flush_reps > 0:
        fl = []
        for k in range(flush_reps):
            flush.fill_(float(k))
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            step()
            b.record()
            fl.append((a, b))
        torch.cuda.synchronize()
        res["median_ms_flushed"] = statistics.median(a.elapsed_time(b) for a, b in fl)
    return res


def kernel_table(kernels):
    return {k: {"ms_per_launch": v["ms"] / v["launches"], "launches": v["launches"],
                "tflops": (v["flops"] / (v["ms"] * 1e-3) / 1e12) if v["flops"] else None,
                "GBps_algorithmic": v["bytes"] / (v["ms"] * 1e-3) / 1e9}
            for k, v in sorted(kernels.items(), key=lambda kv: -kv[1]["ms"])}


def roofline_of(kernels):
    """Roofline object of the kernel with the largest time in the region."""
    name, k = max(kernels.items(), key=lambda kv: kv[1]["ms"])
    ms = k["ms"] / k["launches"]
    if k["flops"]:
        achieved = k["flops"] / (k["ms"] * 1e-3) / 1e12
        return {"bound": "mfma", "kernel": name, "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                "traffic": traffic_of(name), "avg_launch_ms": ms,
                "algorithmic_flops_per_launch": k["flops"] / k["launches"]}
    achieved = k["bytes"] / (k["ms"] * 1e-3) / 1e9
    return {"bound": "hbm", "kernel": name, "achieved": achieved, "peak": PEAK_HBM_GBPS,
            "unit": "GB/s", "frac": achieved / PEAK_HBM_GBPS, "traffic": traffic_of(name),
            "avg_launch_ms": ms}


def recompute_cols(y, dlogp, V):
    """Token columns that the recompute backward's softmax contraction runs
    its MFMAs on: the live tokens (nonzero dlogp, target in [0, V)) come first
    in its token order, and a 256-token tile with none of them only writes its
    zero rows."""
    n = int(((dlogp != 0) & (y >= 0) & (y < V)).sum().item())
    return min(int(y.numel()), -(-n // 256) * 256)


def count_recompute(res, cols, T, name="logprob_bwd_probs"):
    """Scale the library's dense figure for a contraction over the tokens
    (2 T d width per launch, one launch per vocabulary chunk) to the FLOPs it
    executes: cols of the T token columns (the softmax contraction always;
    dH and dW with MC_BWD_SKIP_DEAD_TOKENS)."""
    k = res["kernels"].get(name)
    if k:
        k["flops"] *= cols / T


def summary(res, T, counted, executed):
    ms = res["ms_per_step"]
    out = {"value": T / (ms * 1e-3), "ms_per_step": ms, "median_ms_per_step": res["median_ms"],
           "min_ms_per_step": res["min_ms"], "max_ms_per_step": res["max_ms"],
           "median_ms_per_step_flushed": res.get("median_ms_flushed"),
           "counted_tflops": counted / (ms * 1e-3) / 1e12,
           "mfma_frac": counted / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
           "executed_mfma_frac": executed / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
           "clock": res["clock"]}
    clk = res["clock"]
    if clk and clk.get("gfxclk_mhz_mean") and not clk.get("stale"):
        peak_at = FLOP_PER_CLK * clk["gfxclk_mhz_mean"] * 1e6
        out["executed_mfma_frac_at_measured_clock"] = executed / (ms * 1e-3) / peak_at
        out["mfma_frac_at_measured_clock"] = counted / (ms * 1e-3) / peak_at
    out["roofline"] = roofline_of(res["kernels"])
    out["kernels"] = kernel_table(res["kernels"])
    return out


# ---------------------------------------------------------------------------
# the fp64 oracle on the host cores
# ---------------------------------------------------------------------------
def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def oracle_threads():
    try:
        import threadpoolctl
        info = threadpoolctl.threadpool_info()
        return max([i.get("num_threads", 1) for i in info] + [1])
    except Exception:
        return len(os.sched_getaffinity(0))


def cpu_baseline(H, W, y, s, target_s, fwd_only=False):
    """The fp64 oracle on a bounded leading sample of whole groups."""
    import numpy as np
    import oracle
    Wh = W.float().cpu().numpy()
    cu, cg = s.cu_seqlens, s.cu_groups
    d, V = Wh.shape[1], Wh.shape[0]

    def run(n_groups):
        nseq = int(cg[n_groups])
        n = int(cu[nseq])
        Hs = H[:n].float().cpu().numpy()
        ys = y[:n].cpu().numpy()
        t0 = time.perf_counter()
        logp, lse = oracle.logprob_fwd(Hs, Wh, ys)
        if not fwd_only:
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
    # fp64 work the oracle executes: logits 2ndV; backward: logits again,
    # G W and G^T H, 6ndV
    flops = (2.0 if fwd_only else 8.0) * n * d * V
    what = "logprob_fwd" if fwd_only else "logprob_fwd + rl_loss + logprob_bwd (full dH rows and dW)"
    return {"value": n / t, "unit": "tokens/s", "cores": int(oracle_threads()), "kind": "oracle",
            "cpu_model": cpu_model(), "fp64_gflops": flops / t / 1e9,
            "sample": (f"first {groups} groups ({n} tokens) of the workload: fp64 oracle "
                       f"{what}, {t:.1f} s wall")}


# ---------------------------------------------------------------------------
# rocprofv3 summaries (measurement aid)
# ---------------------------------------------------------------------------
def summarize(path, only=None):
    """Per-kernel summary of a rocprofv3 output directory: average kernel
    durations from a kernel trace, or per-dispatch counter values with the
    figures derived from them (clock, MFMA utilisation, memory-side bytes).
    `only`: kernel roles to print (all when None)."""
    rows_t, rows_c = [], []
    for f in glob.glob(os.path.join(path, "**", "*kernel_trace.csv"), recursive=True):
        rows_t += list(csv.DictReader(open(f)))
    for f in glob.glob(os.path.join(path, "**", "*counter_collection.csv"), recursive=True):
        rows_c += list(csv.DictReader(open(f)))

    def role(name):
        for key in ("k_fwd_logits_lse", "k_bwd_probs", "k_bwd_dhidden", "k_bwd_dweight",
                    "k_cache_gather", "k_transpose", "k_onehot_seg", "k_onehot_join", "k_lse_merge",
                    "k_shard_partial", "k_dh_tail_reduce", "k_tail_reduce", "k_surrogate", "k_seq_stats",
                    "k_bucket_rank", "k_bucket_fill", "k_hist", "k_scan", "k_fill_i32", "k_bound_abs",
                    "k_live_rows", "k_live_count", "k_live_perm",
                    "k_count", "k_finish", "k_loss_init", "copyBuffer"):
            if key in name:
                return key
        return "other"

    if rows_t:
        agg = {}
        for r in rows_t:
            dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-6
            agg.setdefault(role(r["Kernel_Name"]), []).append(dur)
        print(f"{'kernel':24s} {'calls':>6s} {'avg_ms':>9s} {'min_ms':>9s} {'max_ms':>9s}")
        for k, v in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
            print(f"{k:24s} {len(v):6d} {statistics.fmean(v):9.3f} {min(v):9.3f} {max(v):9.3f}")
    if rows_c:
        disp = {}
        for r in rows_c:
            d = disp.setdefault(r["Dispatch_Id"], {"role": role(r["Kernel_Name"]), "c": {},
                                                   "ns": int(r["End_Timestamp"]) -
                                                   int(r["Start_Timestamp"])})
            d["c"][r["Counter_Name"]] = d["c"].get(r["Counter_Name"], 0.0) + float(
                r["Counter_Value"])
        by_role = {}
        for d in disp.values():
            if only is None or d["role"] in only:
                by_role.setdefault(d["role"], []).append(d)
        for k, ds in sorted(by_role.items()):
            names = sorted({c for d in ds for c in d["c"]})
            mean = {c: statistics.fmean(d["c"].get(c, 0.0) for d in ds) for c in names}
            ns = statistics.fmean(d["ns"] for d in ds)
            print(f"{k}  ({len(ds)} dispatches, {ns * 1e-6:.3f} ms each under counters)")
            long = ns >= 1e6      # per-dispatch clocks are meaningful for long dispatches only
            for c in names:
                if c != "GRBM_COUNT" and (long or c.startswith("TCC_EA0") or
                                          c == "SQ_LDS_BANK_CONFLICT"):
                    print(f"    {c:40s} {mean[c]:20.1f}")
            g = mean.get("GRBM_GUI_ACTIVE")
            if g and long:
                per_xcd = g / 8.0                       # the counter sums the 8 XCDs
                print(f"    {'clock (GRBM_GUI_ACTIVE / 8 / duration)':40s} "
                      f"{per_xcd / ns:17.3f} GHz")
                if "SQ_VALU_MFMA_BUSY_CYCLES" in mean:
                    util = mean["SQ_VALU_MFMA_BUSY_CYCLES"] / (4 * 256 * per_xcd)
                    print(f"    {'MFMA utilisation (busy / 1024 SIMDs)':40s} {100 * util:18.1f} %")
            if "TCC_EA0_RDREQ_DRAM_32B_sum" in mean:
                rb = 32.0 * mean["TCC_EA0_RDREQ_DRAM_32B_sum"]
                print(f"    {'memory-side read bytes':40s} {rb:20.0f}  ({rb / ns:.1f} GB/s)")
            if "TCC_EA0_WRREQ_WRITE_DRAM_32B_sum" in mean:
                wb = 32.0 * mean["TCC_EA0_WRREQ_WRITE_DRAM_32B_sum"]
                print(f"    {'memory-side write bytes':40s} {wb:20.0f}  ({wb / ns:.1f} GB/s)")


# ---------------------------------------------------------------------------
def main():
    ap = argparse.ArgumentParser(description=__doc__,
                                 formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=4, choices=[2, 3, 4, 5])
    ap.add_argument("--step", default="both", choices=["both", "recompute", "cached", "skip"],
                    help="which step(s) to time (default both; the headline is recompute)")
    ap.add_argument("--shard", action="store_true",
                    help="time one GPU's vocabulary shard (V/8 entries) of the workload")
    ap.add_argument("--targets", default="model", choices=["model", "zipf"])
    ap.add_argument("--flush-reps", type=int, default=10,
                    help="extra steps timed one by one after a 1 GiB scratch write each")
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="target duration of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-clock", action="store_true", help="do not sample the clock")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a plain 1 GiB device copy three times (calibrates the "
                         "memory-traffic counters against a known byte count)")
    ap.add_argument("--summarize", metavar="DIR",
                    help="print the per-kernel summary of a rocprofv3 output directory")
    ap.add_argument("--only", metavar="K1,K2", help="with --summarize: kernels to print")
    args = ap.parse_args()
    if args.summarize:
        summarize(args.summarize, args.only.split(",") if args.only else None)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported by this "
              "single-GPU build (the multi-GPU sharding is a design note only).",
              file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        import torch
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_per_launch": src.numel() * 4}), flush=True)
        return

    import torch
    import paper_2606_04847_amd as mc
    lib = mc.load_library()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg, s, H, W, y, lr, st = build_inputs(args.config, dev, args.targets)
    T, d, V = s.T, cfg["d"], cfg["V"]
    params = mc.RLParams()
    sampler = None if args.no_clock else ClockSampler()
    flush = torch.empty(FLUSH_BYTES // 4, dtype=torch.float32, device=dev)
    logp = torch.empty(T, dtype=torch.float32, device=dev)
    lse = torch.empty(T, dtype=torch.float32, device=dev)
    extra = ", Zipf-like targets (exponent 1.2)" if args.targets == "zipf" else ""
    config = {"workload": workload_name(cfg, s, extra), "T": T, "d": d, "V": V,
              "sequences": s.B, "groups": s.NG, "parallelism": "none (1 GPU)",
              "targets": args.targets}
    line = {"metric": METRIC, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "bf16", "data": "synthetic"}
    fwd_only = cfg["fwd_only"]

    if args.shard:
        # one GPU's part of a vocabulary-parallel LM head: V/8 rows of W; the
        # merge of the 8 shards' partials (a collective) is not part of it
        Vs = -(-V // 8)
        Ws = W[:Vs].contiguous()
        mc.logprob_fwd(H, W, y, logp=logp, lse=lse)
        out = mc.rl_loss(logp, lr, st["mask"], st["cu"], st["cg"], st["rewards"], params)
        dlogp = out["dlogp"]
        ws_f = torch.empty(lib.mc_logprob_fwd_workspace_size(T, d, Vs, 1), dtype=torch.uint8,
                           device=dev)
        ws_b = torch.empty(lib.mc_logprob_bwd_workspace_size(T, d, Vs, 1), dtype=torch.uint8,
                           device=dev)
        part = torch.empty(4, T, dtype=torch.float32, device=dev)
        dH = torch.empty(T, d, dtype=torch.float32, device=dev)
        dWs = torch.empty(Vs, d, dtype=torch.float32, device=dev)

        def step():
            mc.logprob_fwd_shard(H, Ws, y, 0, V, partial=part, workspace=ws_f)
            mc.logprob_bwd_shard(H, Ws, y, lse, dlogp, 0, V, dhidden=dH, dweight=dWs,
                                 workspace=ws_b)
        res = time_steps(step, args.steps, args.warmup, sampler, flush, args.flush_reps)
        cols = recompute_cols(y, dlogp, V)
        count_recompute(res, cols, T)
        summ = summary(res, T, 6.0 * T * d * Vs, 6.0 * T * d * Vs + 2.0 * cols * d * Vs)
        summ["recompute_token_cols"] = cols
        config.update(workload=config["workload"] + f"; vocabulary shard of {Vs} rows (V/8)",
                      V_shard=Vs, backward="recompute logits (shard)")
        line.update(summ)
        line["config"] = config
        line["metric"] = METRIC + " (one GPU's V/8 shard)"
    elif fwd_only:
        ws_f = torch.empty(lib.mc_logprob_fwd_workspace_size(T, d, V, 1), dtype=torch.uint8,
                           device=dev)

        def step():
            mc.logprob_fwd(H, W, y, logp=logp, lse=lse, workspace=ws_f)
        res = time_steps(step, args.steps, args.warmup, sampler, flush, args.flush_reps)
        summ = summary(res, T, 2.0 * T * d * V, 2.0 * T * d * V)
        config.update(backward="none (forward-only workload)")
        line.update(summ)
        line["config"] = config
        line["metric"] = "fused logprob fwd tokens/s (forward-only workload); % bf16 MFMA peak"
    else:
        ws_f = torch.empty(lib.mc_logprob_fwd_workspace_size(T, d, V, 1), dtype=torch.uint8,
                           device=dev)
        dH = torch.empty(T, d, dtype=torch.float32, device=dev)
        dW = torch.empty(V, d, dtype=torch.float32, device=dev)
        results = {}
        if args.step in ("both", "recompute"):
            ws_b = torch.empty(lib.mc_logprob_bwd_workspace_size(T, d, V, 1), dtype=torch.uint8,
                               device=dev)

            def step():
                mc.logprob_fwd(H, W, y, logp=logp, lse=lse, workspace=ws_f)
                out = mc.rl_loss(logp, lr, st["mask"], st["cu"], st["cg"], st["rewards"], params)
                mc.logprob_bwd(H, W, y, lse, out["dlogp"], dhidden=dH, dweight=dW,
                               workspace=ws_b)
                return out
            log("timing the recompute step")
            results["recompute"] = time_steps(step, args.steps, args.warmup, sampler, flush,
                                              args.flush_reps)
        if args.step in ("both", "skip"):
            # the same step with MC_BWD_SKIP_DEAD_TOKENS: dH and dW leave out
            # the dead tokens' zero products (reported beside the headline,
            # which counts the dense backward)
            if args.step == "skip":
                ws_b = torch.empty(lib.mc_logprob_bwd_workspace_size(T, d, V, 1),
                                   dtype=torch.uint8, device=dev)

            def step():
                mc.logprob_fwd(H, W, y, logp=logp, lse=lse, workspace=ws_f)
                out = mc.rl_loss(logp, lr, st["mask"], st["cu"], st["cg"], st["rewards"], params)
                mc.logprob_bwd(H, W, y, lse, out["dlogp"], dhidden=dH, dweight=dW,
                               skip_dead_tokens=True, workspace=ws_b)
                return out
            log("timing the recompute step with dead tokens skipped")
            results["skip_dead"] = time_steps(step, args.steps, args.warmup, sampler, flush,
                                              args.flush_reps)
        if args.step in ("both", "recompute", "skip"):
            del ws_b
            torch.cuda.empty_cache()
        if args.step in ("both", "cached"):
            ws_c = torch.empty(lib.mc_logprob_bwd_cached_workspace_size(T, d, V, 1),
                               dtype=torch.uint8, device=dev)
            cache = mc.softmax_cache(H, W)

            def step():
                mc.logprob_fwd_cached(H, W, y, cache, logp=logp, lse=lse, workspace=ws_f)
                out = mc.rl_loss(logp, lr, st["mask"], st["cu"], st["cg"], st["rewards"], params)
                mc.logprob_bwd_cached(H, W, y, lse, out["dlogp"], cache, dhidden=dH, dweight=dW,
                                      workspace=ws_c)
                return out
            log("timing the cached step")
            results["cached"] = time_steps(step, args.steps, args.warmup, sampler, flush,
                                           args.flush_reps)
            del ws_c, cache
        head = ("recompute" if "recompute" in results else
                "cached" if "cached" in results else "skip_dead")
        for name, res in results.items():
            out = res["out"]
            executed = 6.0 * T * d * V
            if name in ("recompute", "skip_dead"):
                cols = recompute_cols(y, out["dlogp"], V)
                count_recompute(res, cols, T)
                executed += 2.0 * cols * d * V
            if name == "skip_dead":
                for k in ("logprob_bwd_dhidden", "logprob_bwd_dweight"):
                    count_recompute(res, cols, T, k)
                executed = 2.0 * T * d * V + 6.0 * cols * d * V
            summ = summary(res, T, 6.0 * T * d * V, executed)
            if name in ("recompute", "skip_dead"):
                summ["recompute_token_cols"] = cols
            if name == "skip_dead":
                # not the counted step: the backward leaves out dead tokens'
                # products, so only the executed figure is meaningful
                for k in ("mfma_frac", "counted_tflops", "mfma_frac_at_measured_clock"):
                    summ.pop(k, None)
                summ["note"] = ("MC_BWD_SKIP_DEAD_TOKENS: dH and dW leave out the zero products "
                                "of tokens with zero dlogp; same results; executed FLOPs "
                                "2TdV + 6 T_c d V")
            summ["loss"] = float(out["loss"].item())
            summ["n_valid"] = int(out["n_valid"].item())
            results[name] = summ
        line.update(results[head])
        config["backward"] = {
            "recompute": "recompute logits: the forward writes no [T,V] tensor",
            "cached": "softmax cache: the forward writes a [T,V] fp16 cache",
            "skip_dead": "recompute logits, MC_BWD_SKIP_DEAD_TOKENS (not the counted step)"}[head]
        line["config"] = config
        if head == "recompute" and "cached" in results:
            line["cached"] = results["cached"]
        if head == "recompute" and "skip_dead" in results:
            line["skip_dead"] = results["skip_dead"]
        for name, r in results.items():
            frac = (f"{100 * r['mfma_frac']:.1f}% of peak counted" if "mfma_frac" in r else
                    f"{100 * r['executed_mfma_frac']:.1f}% of peak executed")
            log(f"{name}: {r['ms_per_step']:.3f} ms/step ({frac})")

    if not args.no_cpu_baseline:
        log("timing the fp64 oracle baseline sample")
        line["cpu_baseline"] = cpu_baseline(H, W, y, s, args.cpu_seconds, fwd_only=fwd_only)
    else:
        line["cpu_baseline"] = None
    order = ["metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
             "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
             "mfma_frac", "roofline", "cpu_baseline"]
    print(json.dumps({**{k: line[k] for k in order if k in line},
                      **{k: v for k, v in line.items() if k not in order}}), flush=True)


if __name__ == "__main__":
    main()
