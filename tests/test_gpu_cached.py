"""GPU parity of the softmax-cache path (mc_logprob_fwd_cached /
mc_logprob_bwd_cached): the forward keeps exp(z - block max) and the block
maxima, the backward gathers the live tokens' rows of them into its operand
instead of recomputing the logits, leaving the cache as it was.  Compared
with the fp64 oracle element by element at small and mid sizes, on sampled
rows at full size, and with the recompute path; several backward calls on
one cache; MC_BWD_SKIP_DEAD_TOKENS against the call without it."""
import numpy as np
import pytest

import oracle
from _cases import (GRAD_RTOL, LOGP_ATOL, PTERM_RTOL, assert_step_parity, device_tensors,
                    fullsize_inputs, oracle_step, rel_fro, sample_rows, small_case,
                    structure_tensors, to_params)
from workloads import CONFIGS, make_tensors_numpy, scaled_config

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_04847_amd as mc
    mc.load_library()


def _mc():
    import paper_2606_04847_amd as mc
    return mc


def _drift(B):
    return dict(kind="frac_normal", count=max(1, B // 10), mean=0.3, std=0.1)


def cached_step(case, params, lr, dev="cuda"):
    mc = _mc()
    H, W, y = device_tensors(case, dev)
    st = structure_tensors(case["s"], dev)
    cache = mc.softmax_cache(H, W)
    logp, lse = mc.logprob_fwd_cached(H, W, y, cache)
    out = mc.rl_loss(logp, torch.from_numpy(lr).to(dev), st["mask"], st["cu"], st["cg"],
                     st["rewards"], to_params(params))
    dH, dW = mc.logprob_bwd_cached(H, W, y, lse, out["dlogp"], cache)
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy() for k, v in out.items()}
    res.update(logp=logp.cpu().numpy(), lse=lse.cpu().numpy(), dH=dH.cpu().numpy(),
               dW=dW.cpu().numpy())
    return res


def test_cached_config1_fp32_end_to_end():
    case = small_case(1)
    p = oracle.RLParams()
    o = oracle_step(case, p)
    g = cached_step(case, p, o["lr"])
    assert_step_parity(g, o, grad_rtol=1e-4, logp_atol=1e-4)


@pytest.mark.parametrize("T,d,V", [(1500, 256, 3000), (700, 136, 1000), (2100, 512, 777)])
def test_cached_midsize_bf16_end_to_end(T, d, V):
    cfg = scaled_config(4, T=T, n_groups=2, group_size=8, d=d, V=V, hi=max(100, T // 10),
                        seed=T + V, drift=_drift(16))
    case = small_case(cfg)
    p = oracle.RLParams()
    o = oracle_step(case, p)
    g = cached_step(case, p, o["lr"])
    assert_step_parity(g, o)


def test_cached_forward_equals_plain_forward():
    # the cache is an extra output: lse, logp and entropy are bit-identical
    cfg = scaled_config(4, T=900, n_groups=2, group_size=8, d=256, V=1300, hi=120, seed=71,
                        drift=_drift(16))
    case = small_case(cfg)
    mc = _mc()
    H, W, y = device_tensors(case)
    a = mc.logprob_fwd(H, W, y, with_entropy=True)
    b = mc.logprob_fwd_cached(H, W, y, mc.softmax_cache(H, W), with_entropy=True)
    torch.cuda.synchronize()
    for u, v in zip(a, b):
        assert torch.equal(u, v)


def test_cached_peaked_softmax_pterm():
    # the softmax part alone: two roundings to fp16 (the cached exp and the
    # operand), each within 2^-11 relative, stay inside the 2^-10 bar
    cfg = scaled_config(4, T=600, n_groups=2, group_size=8, d=512, V=2000, hi=200, seed=13,
                        w_std=0.1, drift=_drift(16))
    case = small_case(cfg)
    p = oracle.RLParams(filter="none")
    o = oracle_step(case, p)
    g = cached_step(case, p, o["lr"])
    assert_step_parity(g, o)
    y = case["y"]
    W = case["W"].astype(np.float64)
    H = case["H"].astype(np.float64)
    onehot_o = o["dlogp"][:, None] * W[y]
    onehot_g = g["dlogp"].astype(np.float64)[:, None] * W[y]
    assert rel_fro(g["dH"] - onehot_g, o["dH"] - onehot_o) <= PTERM_RTOL
    Wo = np.zeros_like(o["dW"])
    Wg = np.zeros_like(o["dW"])
    np.add.at(Wo, y, o["dlogp"][:, None] * H)
    np.add.at(Wg, y, g["dlogp"].astype(np.float64)[:, None] * H)
    assert rel_fro(g["dW"] - Wg, o["dW"] - Wo) <= PTERM_RTOL


def test_large_logits_both_paths():
    # W std 10: logits of std ~80, every softmax effectively one-hot and the
    # per-block maxima hundreds of nats apart (the cache's exp(c_b - lse)
    # underflows to 0 for most blocks); targets uniform so that the gradient
    # (dlogp (onehot_y - onehot_argmax)) is far from zero
    cfg = scaled_config(4, d=64, V=2000, seed=77, w_std=10.0)
    T = 300
    H, W, hb, wb = make_tensors_numpy(cfg, T)
    rng = np.random.default_rng(78)
    y = rng.integers(0, 2000, size=T)
    case = dict(H=H, W=W, hb=hb, wb=wb, y=y)
    logp_o, lse_o = oracle.logprob_fwd(H, W, y)
    dlogp = rng.standard_normal(T) * 1e-2
    dH_o, dW_o = oracle.logprob_bwd(H, W, y, lse_o, dlogp)
    mc = _mc()
    Hd, Wd, yd = device_tensors(case)
    dl = torch.from_numpy(dlogp.astype(np.float32)).cuda()
    logp_p, lse_p = mc.logprob_fwd(Hd, Wd, yd)
    dH_p, dW_p = mc.logprob_bwd(Hd, Wd, yd, lse_p, dl)
    cache = mc.softmax_cache(Hd, Wd)
    logp_c, lse_c = mc.logprob_fwd_cached(Hd, Wd, yd, cache)
    dH_c, dW_c = mc.logprob_bwd_cached(Hd, Wd, yd, lse_c, dl, cache)
    torch.cuda.synchronize()
    assert np.abs(lse_o).max() > 100.0
    # here the softmax part carries about half of the gradient, and its fp16
    # operand bounds it at 2^-10 relative with the cache's two roundings (not
    # the near-uniform 1e-3 bar): the one-hot part is exact, so the whole
    # gradient is held to that bound too
    Wf, Hf = W.astype(np.float64), H.astype(np.float64)
    onehot_dH = dlogp[:, None] * Wf[y]
    onehot_dW = np.zeros_like(dW_o)
    np.add.at(onehot_dW, y, dlogp[:, None] * Hf)
    for logp, lse, dH, dW in ((logp_p, lse_p, dH_p, dW_p), (logp_c, lse_c, dH_c, dW_c)):
        assert np.max(np.abs(logp.cpu().numpy() - logp_o)) <= LOGP_ATOL
        assert np.max(np.abs(lse.cpu().numpy() - lse_o)) <= LOGP_ATOL
        g_dH, g_dW = dH.cpu().numpy().astype(np.float64), dW.cpu().numpy().astype(np.float64)
        assert np.isfinite(g_dH).all() and np.isfinite(g_dW).all()
        assert rel_fro(g_dH - onehot_dH, dH_o - onehot_dH) <= PTERM_RTOL
        assert rel_fro(g_dW - onehot_dW, dW_o - onehot_dW) <= PTERM_RTOL
        assert rel_fro(g_dH, dH_o) <= PTERM_RTOL and rel_fro(g_dW, dW_o) <= PTERM_RTOL


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("T,d,V", [(1, 8, 1), (1, 64, 7), (300, 136, 257), (257, 8, 513),
                                   (513, 64, 256)])
def test_cached_edge_shapes(dtype, T, d, V):
    cfg = scaled_config(1, d=d, V=V, dtype=dtype, seed=20 + T + V)
    H, W, hb, wb = make_tensors_numpy(cfg, T)
    rng = np.random.default_rng(T * 7 + V)
    y = rng.integers(0, V, size=T)
    if T > 4:
        y[1] = -1
        y[3] = V
        y[5:9] = y[4]
    case = dict(H=H, W=W, hb=hb, wb=wb, y=y)
    logp_o, lse_o = oracle.logprob_fwd(H, W, y)
    dlogp = rng.standard_normal(T) * 1e-2
    dH_o, dW_o = oracle.logprob_bwd(H, W, y, lse_o, dlogp)
    mc = _mc()
    Hd, Wd, yd = device_tensors(case)
    cache = mc.softmax_cache(Hd, Wd)
    logp, lse = mc.logprob_fwd_cached(Hd, Wd, yd, cache)
    dl = torch.from_numpy(dlogp.astype(np.float32)).cuda()
    dH, dW = mc.logprob_bwd_cached(Hd, Wd, yd, lse, dl, cache)
    torch.cuda.synchronize()
    assert np.max(np.abs(logp.cpu().numpy() - logp_o)) <= LOGP_ATOL
    assert np.max(np.abs(lse.cpu().numpy() - lse_o)) <= LOGP_ATOL
    assert rel_fro(dH.cpu().numpy(), dH_o) <= GRAD_RTOL
    assert rel_fro(dW.cpu().numpy(), dW_o) <= GRAD_RTOL
    if T > 4:
        assert np.all(dH[1].cpu().numpy() == 0.0) and np.all(dH[3].cpu().numpy() == 0.0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_cached_contents_of_cache_and_workspace_do_not_matter(dtype):
    # 0xFF bytes (NaN in both dtypes) in the cache and both workspaces before
    # the calls give results bit-identical to zeroed ones; ragged T and V
    mc = _mc()
    lib = mc.load_library()
    d, V = 136, 1003
    case = small_case(scaled_config(1, d=d, V=V, dtype=dtype, seed=61))   # T = 613
    H, W, y = device_tensors(case)
    T = H.shape[0]
    code = 1 if dtype == "bf16" else 0
    dl = torch.from_numpy((np.random.default_rng(62).standard_normal(T) * 1e-2)
                          .astype(np.float32)).cuda()

    def buf(nbytes, fill):
        return torch.full((max(int(nbytes), 1),), fill, dtype=torch.uint8, device="cuda")

    outs = []
    for fill in (0, 255):
        cache = buf(lib.mc_logprob_cache_size(T, d, V, code), fill)
        logp, lse = mc.logprob_fwd_cached(
            H, W, y, cache, workspace=buf(lib.mc_logprob_fwd_workspace_size(T, d, V, code), fill))
        dH, dW = mc.logprob_bwd_cached(
            H, W, y, lse, dl, cache,
            workspace=buf(lib.mc_logprob_bwd_cached_workspace_size(T, d, V, code), fill))
        torch.cuda.synchronize()
        outs.append((logp, lse, dH, dW))
    for a, b in zip(*outs):
        assert torch.isfinite(b).all()
        assert torch.equal(a, b)


def test_cached_accumulate_flags_and_partial_outputs():
    cfg = scaled_config(4, T=400, n_groups=2, group_size=8, d=128, V=600, hi=100, seed=14,
                        drift=_drift(16))
    case = small_case(cfg)
    mc = _mc()
    H, W, y = device_tensors(case)
    dl = torch.randn(len(case["y"]), device="cuda") * 1e-3

    def run(**kw):
        cache = mc.softmax_cache(H, W)
        _, lse = mc.logprob_fwd_cached(H, W, y, cache)
        return mc.logprob_bwd_cached(H, W, y, lse, dl, cache, **kw)

    dH, dW = run()
    dH2, dW2 = torch.ones_like(dH), torch.ones_like(dW)
    run(dhidden=dH2, dweight=dW2, accumulate_dhidden=True, accumulate_dweight=True)
    only_h, none_w = run(need_dweight=False)
    none_h, only_w = run(need_dhidden=False)
    torch.cuda.synchronize()
    assert none_w is None and none_h is None
    assert torch.allclose(dH2, dH + 1, atol=1e-6, rtol=0)
    assert torch.allclose(dW2, dW + 1, atol=1e-6, rtol=0)
    assert torch.equal(only_h, dH) and torch.equal(only_w, dW)


@pytest.mark.parametrize("cid", [4, 3, 5])
def test_cached_fullsize_sampled(cid):
    # the headline step's configuration (workload 4) and the two larger ones,
    # in the launch configuration the benchmark times
    mc = _mc()
    s, H, W, y = fullsize_inputs(cid)
    T, V = s.T, W.shape[0]
    cache = mc.softmax_cache(H, W)
    logp, lse = mc.logprob_fwd_cached(H, W, y, cache)
    torch.cuda.synchronize()
    rows = sample_rows(T, 40, cid, extra=(T - 2, 8191, 8192))
    Hs = H[rows].float().cpu().numpy()
    Wh = W.float().cpu().numpy()
    ys = y[rows].cpu().numpy()
    lo, so = oracle.logprob_fwd(Hs, Wh, ys)
    assert np.max(np.abs(logp[rows].cpu().numpy() - lo)) <= LOGP_ATOL
    assert np.max(np.abs(lse[rows].cpu().numpy() - so)) <= LOGP_ATOL
    rng = np.random.default_rng(cid)
    dl = np.zeros(T, np.float32)
    dl[rows] = (rng.standard_normal(len(rows)) / T).astype(np.float32)
    dH, dW = mc.logprob_bwd_cached(H, W, y, lse, torch.from_numpy(dl).cuda(), cache)
    torch.cuda.synchronize()
    dH_o = oracle.dhidden_rows(Hs, Wh, ys, so, dl[rows].astype(np.float64))
    assert rel_fro(dH[rows].cpu().numpy(), dH_o) <= GRAD_RTOL
    others = torch.ones(T, dtype=torch.bool, device="cuda")
    others[torch.from_numpy(rows).cuda()] = False
    assert torch.count_nonzero(dH[others]).item() == 0
    vrows = np.unique(np.concatenate([ys[:16], rng.choice(V, 24, replace=False), [0, V - 1]]))
    dW_o = oracle.dweight_rows(Hs, Wh, ys, so, dl[rows].astype(np.float64), vrows)
    assert rel_fro(dW[torch.from_numpy(vrows).cuda()].cpu().numpy(), dW_o) <= GRAD_RTOL
    del dH, dW, cache
    torch.cuda.empty_cache()


@pytest.mark.parametrize("path", ["cached", "recompute"])
@pytest.mark.parametrize("accumulate", [False, True])
def test_zero_dlogp_rows_and_shared_targets(path, accumulate):
    # Tokens outside the loss mask reach the backward with dlogp exactly 0:
    # their softmax rows are written as zeros without being read, they are
    # skipped in dW's one-hot scatter, and a target whose tokens all have
    # zero dlogp leaves its dW row to the contraction alone.  Few distinct
    # targets so that buckets mix zero and nonzero tokens and some hold
    # only zero ones.
    cfg = scaled_config(4, T=700, n_groups=2, group_size=8, d=136, V=300, hi=100, seed=23,
                        drift=_drift(16))
    case = small_case(cfg)
    T = len(case["y"])
    rng = np.random.default_rng(7)
    y = rng.integers(0, 40, T).astype(np.int64)
    dl = rng.normal(0.0, 1e-3, T).astype(np.float32)
    dl[rng.random(T) < 0.6] = 0.0
    dl[y < 8] = 0.0                                  # buckets of only zero-dlogp tokens
    assert (dl == 0).any() and (dl != 0).any()
    _, lse_o = oracle.logprob_fwd(case["H"], case["W"], y)
    dH_o, dW_o = oracle.logprob_bwd(case["H"], case["W"], y, lse_o, dl.astype(np.float64))

    mc = _mc()
    H, W, _ = device_tensors(case)
    yd = torch.from_numpy(y).cuda()
    dld = torch.from_numpy(dl).cuda()
    base_h = torch.full((T, H.shape[1]), 0.5, device="cuda") if accumulate else None
    base_w = torch.full((W.shape[0], W.shape[1]), -0.25, device="cuda") if accumulate else None
    kw = dict(dhidden=base_h, dweight=base_w, accumulate_dhidden=accumulate,
              accumulate_dweight=accumulate)
    if path == "cached":
        cache = mc.softmax_cache(H, W)
        _, lse = mc.logprob_fwd_cached(H, W, yd, cache)
        dH, dW = mc.logprob_bwd_cached(H, W, yd, lse, dld, cache, **kw)
    else:
        _, lse = mc.logprob_fwd(H, W, yd)
        dH, dW = mc.logprob_bwd(H, W, yd, lse, dld, **kw)
    torch.cuda.synchronize()
    dH, dW = dH.cpu().numpy().astype(np.float64), dW.cpu().numpy().astype(np.float64)
    if accumulate:
        dH -= 0.5
        dW += 0.25
    assert np.isfinite(dH).all() and np.isfinite(dW).all()
    assert rel_fro(dH, dH_o) <= GRAD_RTOL
    assert rel_fro(dW, dW_o) <= GRAD_RTOL
    # a token with zero dlogp has a zero gradient row exactly
    assert (dH[dl == 0] == 0).all()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_cache_serves_several_backward_calls(dtype):
    # the backward only reads the cache: two upstream gradients (a third of
    # the tokens dead in the second) from one forward, each against the
    # oracle, the first repeated bit for bit after the second; and each with
    # MC_BWD_SKIP_DEAD_TOKENS (dW bit for bit, dH up to the order of sums)
    mc = _mc()
    d, V = 136, 1003
    case = small_case(scaled_config(1, d=d, V=V, dtype=dtype, seed=91))
    H, W, y = device_tensors(case)
    T = H.shape[0]
    rng = np.random.default_rng(92)
    dls = [(rng.standard_normal(T) * 1e-2).astype(np.float32) for _ in range(2)]
    dls[1][rng.random(T) < 0.33] = 0.0
    cache = mc.softmax_cache(H, W)
    _, lse = mc.logprob_fwd_cached(H, W, y, cache)
    before = cache.clone()
    outs = [mc.logprob_bwd_cached(H, W, y, lse, torch.from_numpy(dl).cuda(), cache)
            for dl in dls]
    again = mc.logprob_bwd_cached(H, W, y, lse, torch.from_numpy(dls[0]).cuda(), cache)
    skips = [mc.logprob_bwd_cached(H, W, y, lse, torch.from_numpy(dl).cuda(), cache,
                                   skip_dead_tokens=True) for dl in dls]
    torch.cuda.synchronize()
    assert torch.equal(cache, before)
    assert torch.equal(outs[0][0], again[0]) and torch.equal(outs[0][1], again[1])
    _, lse_o = oracle.logprob_fwd(case["H"], case["W"], case["y"])
    for dl, (dH, dW), (dHs, dWs) in zip(dls, outs, skips):
        dH_o, dW_o = oracle.logprob_bwd(case["H"], case["W"], case["y"], lse_o,
                                        dl.astype(np.float64))
        assert rel_fro(dH.double().cpu().numpy(), dH_o) <= GRAD_RTOL
        assert rel_fro(dW.double().cpu().numpy(), dW_o) <= GRAD_RTOL
        assert torch.equal(dW, dWs)
        assert rel_fro(dHs.double().cpu().numpy(), dH.double().cpu().numpy()) <= 1e-6
        dead = torch.from_numpy(dl == 0.0).cuda()
        assert not dH[dead].any() and not dHs[dead].any()
