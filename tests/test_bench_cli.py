"""bench.py's host-side contract that needs no GPU: it measures one GPU and
refuses a multi-GPU request with a message instead of reporting a figure, and
its stored counter traffic is keyed to the kernel sources (any edit of a
kernel source changes the key, so the figure is reported as null)."""
import os
import shutil
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_multi_gpu_request_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""          # no JSON line


def test_traffic_key_changes_with_any_kernel_source(tmp_path, monkeypatch):
    sys.path.insert(0, ROOT)
    import bench
    csrc = os.path.join(ROOT, "paper_2606_04847_amd", "csrc")
    copy = tmp_path / "paper_2606_04847_amd" / "csrc"
    shutil.copytree(csrc, copy, ignore=shutil.ignore_patterns("__pycache__"))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    d0 = bench.sources_digest()
    assert d0 == bench.sources_digest()
    for name in sorted(os.listdir(copy)):
        p = copy / name
        text = p.read_bytes()
        p.write_bytes(text + b"\n")
        assert bench.sources_digest() != d0, name
        p.write_bytes(text)
    assert bench.sources_digest() == d0


def test_recompute_flops_follow_the_live_tiles():
    # the softmax contraction runs its MFMAs on the live tokens' 256-token
    # tiles only; the executed figure scales the library's dense one (one
    # launch per vocabulary chunk) by the share of token columns it covers
    sys.path.insert(0, ROOT)
    import bench
    import torch
    T, d, V = 1000, 64, 3000
    y = torch.arange(T) % V
    dl = torch.zeros(T)
    dl[[3, 300, 700]] = 1.0
    y[700] = -1                                    # ignored target: dead
    assert bench.recompute_cols(y, dl, V) == 256   # 2 live tokens -> one tile
    dl[:] = 1.0
    assert bench.recompute_cols(y, dl, V) == T     # capped at T
    dense = 2.0 * T * d * 1500                     # two chunks of 1500 rows
    res = {"kernels": {"logprob_bwd_probs": {"flops": 4 * dense, "launches": 4}}}
    bench.count_recompute(res, 256, T)
    assert res["kernels"]["logprob_bwd_probs"]["flops"] == 4 * 2.0 * 256 * d * 1500
