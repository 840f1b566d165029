"""The fused step under HIP graph capture, and the empty batch.

Every entry point enqueues kernels only (no memsets, no allocations, no host
synchronisation), so the whole step — forward, RL loss, backward, through
either pair (recompute, or the softmax cache held outside the graph), with
or without MC_BWD_SKIP_DEAD_TOKENS, whose tile plans come from the live
count on the device — can
be captured once and replayed.  The test replays the captured step
several times with eager work and synchronisations in between, checks every
replay bit for bit against the eager step on the same inputs, then changes
the inputs in place and checks that a replay follows them.  The empty batch
(T = 0) zeroes dW with a kernel, the path that used to be a memset."""
import ctypes

import numpy as np
import pytest

import oracle
from _cases import assert_step_parity, device_tensors, oracle_step, small_case, structure_tensors
from _cases import to_params
from workloads import scaled_config

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_04847_amd as mc
    mc.load_library()


def _case():
    cfg = scaled_config(4, T=1500, n_groups=4, group_size=8, d=256, V=3000, hi=400, seed=61,
                        drift=dict(kind="frac_normal", count=3, mean=0.3, std=0.1))
    return small_case(cfg)


def _step(mc, H, W, y, lr, st, params, cache=None, skip=False):
    if cache is None:
        logp, lse = mc.logprob_fwd(H, W, y)
    else:
        logp, lse = mc.logprob_fwd_cached(H, W, y, cache)
    out = mc.rl_loss(logp, lr, st["mask"], st["cu"], st["cg"], st["rewards"], params)
    if cache is None:
        dH, dW = mc.logprob_bwd(H, W, y, lse, out["dlogp"], skip_dead_tokens=skip)
    else:
        dH, dW = mc.logprob_bwd_cached(H, W, y, lse, out["dlogp"], cache, skip_dead_tokens=skip)
    return dict(logp=logp, lse=lse, loss=out["loss"], dlogp=out["dlogp"],
                seq_mask=out["seq_mask"], seq_len=out["seq_len"], n_valid=out["n_valid"],
                error_flag=out["error_flag"], dH=dH, dW=dW)


def _host(res):
    return {k: v.detach().cpu().numpy().copy() for k, v in res.items()}


def _same(a, b):
    for k in a:
        assert np.array_equal(a[k], b[k], equal_nan=True), k


@pytest.mark.parametrize("pair", ["recompute", "cached", "skip", "cached-skip"])
def test_step_graph_replays(pair):
    import paper_2606_04847_amd as mc
    case = _case()
    p = oracle.RLParams()
    o = oracle_step(case, p)
    H, W, y = device_tensors(case)
    st = structure_tensors(case["s"])
    lr = torch.from_numpy(o["lr"]).cuda()
    params = to_params(p)
    cache = mc.softmax_cache(H, W) if pair.startswith("cached") else None

    eager = _host(_step(mc, H, W, y, lr, st, params, cache, pair.endswith("skip")))
    assert_step_parity(eager, o)   # the eager step itself matches the oracle

    # warm up on a side stream, then capture
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        _step(mc, H, W, y, lr, st, params, cache, pair.endswith("skip"))
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        static = _step(mc, H, W, y, lr, st, params, cache, pair.endswith("skip"))
    torch.cuda.synchronize()

    for rep in range(3):
        # eager work of the program's own between replays
        scratch = torch.randn(1 << 20, device="cuda")
        scratch.mul_(2.0).sum().item()
        graph.replay()
        torch.cuda.synchronize()
        _same(_host(static), eager)
        print(f"replay {rep}: identical to the eager step", flush=True)

    # the graph reads its inputs at replay time
    H.mul_(0.5)
    eager2 = _host(_step(mc, H, W, y, lr, st, params, cache, pair.endswith("skip")))
    assert not np.array_equal(eager2["dW"], eager["dW"])
    graph.replay()
    torch.cuda.synchronize()
    _same(_host(static), eager2)


def test_empty_batch_zeroes_dweight():
    import paper_2606_04847_amd as mc
    lib = mc.load_library()
    d, V = 64, 100
    H = torch.zeros(8, d, dtype=torch.bfloat16, device="cuda")   # any valid pointer: T = 0
    W = torch.randn(V, d, device="cuda").to(torch.bfloat16)
    dW = torch.full((V, d), float("nan"), device="cuda")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    vp = ctypes.c_void_p
    for name in ("mc_logprob_bwd", "mc_logprob_bwd_cached"):
        dW.fill_(float("nan"))
        if name == "mc_logprob_bwd":
            st = lib.mc_logprob_bwd(vp(H.data_ptr()), vp(W.data_ptr()), None, None, None, 0, d, V,
                                    1, None, vp(dW.data_ptr()), 0, None, 0, stream)
        else:
            st = lib.mc_logprob_bwd_cached(vp(H.data_ptr()), vp(W.data_ptr()), None, None, None,
                                           0, d, V, 1, None, 0, None, vp(dW.data_ptr()), 0,
                                           None, 0, stream)
        torch.cuda.synchronize()
        assert st == 0, (name, st)
        assert torch.count_nonzero(dW).item() == 0 and not torch.isnan(dW).any().item(), name
        # accumulate: left as it is
        dW.fill_(1.5)
        flags = 2   # MC_BWD_ACCUMULATE_DWEIGHT
        if name == "mc_logprob_bwd":
            st = lib.mc_logprob_bwd(vp(H.data_ptr()), vp(W.data_ptr()), None, None, None, 0, d, V,
                                    1, None, vp(dW.data_ptr()), flags, None, 0, stream)
        else:
            st = lib.mc_logprob_bwd_cached(vp(H.data_ptr()), vp(W.data_ptr()), None, None, None,
                                           0, d, V, 1, None, 0, None, vp(dW.data_ptr()), flags,
                                           None, 0, stream)
        torch.cuda.synchronize()
        assert st == 0 and bool((dW == 1.5).all().item()), name
