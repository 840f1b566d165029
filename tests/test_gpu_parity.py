"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Small and mid sizes are compared element by element on every output.  The
full-size workloads are compared on sampled rows the oracle evaluates one
by one, in the same launch configuration the benchmark times.
"""
import numpy as np
import pytest

import oracle
from _cases import (GRAD_RTOL, LOGP_ATOL, LOSS_RTOL, PTERM_RTOL_F16, assert_step_parity,
                    device_tensors, fullsize_inputs, gpu_step, oracle_step, rel_fro,
                    sample_rows, small_case, structure_tensors, to_params)
from workloads import CONFIGS, make_structure, scaled_config

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


def test_config1_end_to_end_fp32():
    case = small_case(1)
    p = oracle.RLParams()
    o = oracle_step(case, p)
    g = gpu_step(case, p, o["lr"])
    assert_step_parity(g, o)
    assert np.max(np.abs(g["logp"] - o["logp"])) < 1e-4    # fp32 operands: much tighter
    assert o["seq_mask"].sum() == case["s"].B - 1           # the drifted sequence is dropped


def _drift(B):
    return dict(kind="frac_normal", count=max(1, B // 10), mean=0.3, std=0.1)


@pytest.mark.parametrize("T,d,V,groups,G", [
    (1500, 256, 3000, 4, 8),        # several tiles in every dimension, ragged tails
    (700, 136, 1000, 2, 8),         # d not a multiple of the 64-wide K step
])
def test_midsize_bf16_end_to_end(T, d, V, groups, G):
    cfg = scaled_config(4, T=T, n_groups=groups, group_size=G, d=d, V=V, hi=400, seed=11,
                        drift=_drift(groups * G))
    case = small_case(cfg)
    p = oracle.RLParams()
    o = oracle_step(case, p)
    g = gpu_step(case, p, o["lr"])
    assert_step_parity(g, o)


@pytest.mark.parametrize("filt", ["none", "vanilla"])
def test_filter_modes_end_to_end(filt):
    cfg = scaled_config(4, T=900, n_groups=4, group_size=8, d=128, V=700, hi=300, seed=12,
                        drift=_drift(32))
    case = small_case(cfg)
    p = oracle.RLParams(filter=filt)
    o = oracle_step(case, p)
    g = gpu_step(case, p, o["lr"])
    assert_step_parity(g, o)


def test_peaked_softmax_pterm():
    # W std 0.1 at d=512: logits std ~2.3, so the softmax part of the gradient
    # is a visible share; compare it separately from the one-hot part.
    cfg = scaled_config(4, T=600, n_groups=2, group_size=8, d=512, V=2000, hi=200, seed=13,
                        w_std=0.1, drift=_drift(16))
    case = small_case(cfg)
    p = oracle.RLParams(filter="none")
    o = oracle_step(case, p)
    g = gpu_step(case, p, o["lr"])
    assert_step_parity(g, o)
    y = case["y"]
    W = case["W"].astype(np.float64)
    H = case["H"].astype(np.float64)
    onehot_o = o["dlogp"][:, None] * W[y]
    onehot_g = g["dlogp"].astype(np.float64)[:, None] * W[y]
    # the recompute pair's fp16 operand: 2^-11
    assert rel_fro(g["dH"] - onehot_g, o["dH"] - onehot_o) <= PTERM_RTOL_F16
    Wo = np.zeros_like(o["dW"])
    Wg = np.zeros_like(o["dW"])
    np.add.at(Wo, y, o["dlogp"][:, None] * H)
    np.add.at(Wg, y, g["dlogp"].astype(np.float64)[:, None] * H)
    assert rel_fro(g["dW"] - Wg, o["dW"] - Wo) <= PTERM_RTOL_F16


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("T,d,V", [(1, 8, 1), (1, 64, 7), (300, 136, 257), (257, 8, 513),
                                   (513, 64, 256)])
def test_edge_shapes_fwd_bwd(dtype, T, d, V):
    cfg = scaled_config(1, d=d, V=V, dtype=dtype, seed=20 + T + V)
    from workloads import make_tensors_numpy
    H, W, hb, wb = make_tensors_numpy(cfg, T)
    rng = np.random.default_rng(T * 7 + V)
    y = rng.integers(0, V, size=T)
    if T > 4:
        y[1] = -1          # ignored
        y[3] = V           # ignored (out of range)
        y[5:9] = y[4]      # duplicate targets
    case = dict(H=H, W=W, hb=hb, wb=wb, y=y)
    logp_o, lse_o = oracle.logprob_fwd(H, W, y)
    dlogp = rng.standard_normal(T) * 1e-2
    dH_o, dW_o = oracle.logprob_bwd(H, W, y, lse_o, dlogp)
    mc = _mc()
    Hd, Wd, yd = device_tensors(case)
    logp, lse = mc.logprob_fwd(Hd, Wd, yd)
    dl = torch.from_numpy(dlogp.astype(np.float32)).cuda()
    dH, dW = mc.logprob_bwd(Hd, Wd, yd, lse, dl)
    torch.cuda.synchronize()
    assert np.max(np.abs(logp.cpu().numpy() - logp_o)) <= LOGP_ATOL
    assert np.max(np.abs(lse.cpu().numpy() - lse_o)) <= LOGP_ATOL
    if T > 4:
        assert logp[1].item() == 0.0 and logp[3].item() == 0.0
    assert rel_fro(dH.cpu().numpy(), dH_o) <= GRAD_RTOL
    assert rel_fro(dW.cpu().numpy(), dW_o) <= GRAD_RTOL
    if T > 4:
        assert np.all(dH[1].cpu().numpy() == 0.0) and np.all(dH[3].cpu().numpy() == 0.0)
    # the same shapes with MC_BWD_SKIP_DEAD_TOKENS (the ignored targets dead)
    dHs, dWs = mc.logprob_bwd(Hd, Wd, yd, lse, dl, skip_dead_tokens=True)
    torch.cuda.synchronize()
    assert torch.equal(dWs, dW)
    assert rel_fro(dHs.double().cpu().numpy(), dH.double().cpu().numpy()) <= 1e-6
    if T > 4:
        assert not dHs[1].any() and not dHs[3].any()


def test_zero_weight_closed_form():
    # W = 0: logp = -ln V exactly up to fp32 rounding of ln V; dH = 0 exactly.
    mc = _mc()
    T, d, V = 300, 64, 1000
    H = torch.randn(T, d, device="cuda").to(torch.bfloat16)
    W = torch.zeros(V, d, device="cuda", dtype=torch.bfloat16)
    y = torch.randint(0, V, (T,), device="cuda")
    logp, lse = mc.logprob_fwd(H, W, y)
    assert torch.allclose(logp, torch.full_like(logp, -np.log(V)), atol=2e-6, rtol=0)
    dH, _ = mc.logprob_bwd(H, W, y, lse, torch.ones(T, device="cuda"), need_dweight=False)
    assert torch.count_nonzero(dH).item() == 0


def test_accumulate_flags_and_partial_outputs():
    cfg = scaled_config(4, T=400, n_groups=2, group_size=8, d=128, V=600, hi=100, seed=14,
                        drift=_drift(16))
    case = small_case(cfg)
    mc = _mc()
    H, W, y = device_tensors(case)
    logp, lse = mc.logprob_fwd(H, W, y)
    dl = torch.randn(len(case["y"]), device="cuda") * 1e-3
    dH, dW = mc.logprob_bwd(H, W, y, lse, dl)
    dH2 = torch.ones_like(dH)
    dW2 = torch.ones_like(dW)
    mc.logprob_bwd(H, W, y, lse, dl, dhidden=dH2, dweight=dW2, accumulate_dhidden=True,
                   accumulate_dweight=True)
    only_h, none_w = mc.logprob_bwd(H, W, y, lse, dl, need_dweight=False)
    none_h, only_w = mc.logprob_bwd(H, W, y, lse, dl, need_dhidden=False)
    torch.cuda.synchronize()
    assert none_w is None and none_h is None
    assert torch.allclose(dH2, dH + 1, atol=1e-6, rtol=0)
    assert torch.allclose(dW2, dW + 1, atol=1e-6, rtol=0)
    assert torch.equal(only_h, dH) and torch.equal(only_w, dW)


def test_dweight_split_tail_accumulate():
    # 12 tiles of dW (d = 256, V = 3000): the whole launch is one partial
    # round, computed as K slices (T = 1500: 4 slices of 384 tokens) summed
    # by the tail reduction; accumulate adds the stored dW after the sum
    cfg = scaled_config(4, T=1500, n_groups=2, group_size=8, d=256, V=3000, hi=200, seed=16,
                        drift=_drift(16))
    case = small_case(cfg)
    mc = _mc()
    H, W, y = device_tensors(case)
    logp, lse = mc.logprob_fwd(H, W, y)
    dl = torch.randn(len(case["y"]), device="cuda") * 1e-3
    _, dW = mc.logprob_bwd(H, W, y, lse, dl)
    dW2 = torch.full_like(dW, 0.5)
    mc.logprob_bwd(H, W, y, lse, dl, dweight=dW2, accumulate_dweight=True, need_dhidden=False)
    cache = mc.softmax_cache(H, W)
    _, lse_c = mc.logprob_fwd_cached(H, W, y, cache)
    dW3 = torch.full_like(dW, -0.25)
    mc.logprob_bwd_cached(H, W, y, lse_c, dl, cache, dweight=dW3, accumulate_dweight=True,
                          need_dhidden=False)
    torch.cuda.synchronize()
    assert torch.allclose(dW2, dW + 0.5, atol=1e-6, rtol=0)
    Wd = W.double().cpu().numpy()
    lo, so = oracle.logprob_fwd(H.float().cpu().numpy().astype(np.float64), Wd, y.cpu().numpy())
    _, dW_o = oracle.logprob_bwd(H.float().cpu().numpy().astype(np.float64), Wd, y.cpu().numpy(),
                                 so, dl.double().cpu().numpy())
    assert rel_fro((dW3 + 0.25).cpu().numpy(), dW_o) <= GRAD_RTOL
    assert rel_fro(dW.cpu().numpy(), dW_o) <= GRAD_RTOL


def test_determinism_bit_identical():
    cfg = scaled_config(4, T=1200, n_groups=4, group_size=8, d=256, V=1500, hi=300, seed=15,
                        drift=_drift(32))
    case = small_case(cfg)
    p = oracle.RLParams()
    lr = (oracle.logprob_fwd(case["H"], case["W"], case["y"])[0]
          + case["s"].rollout_delta).astype(np.float32)
    a = gpu_step(case, p, lr)
    b = gpu_step(case, p, lr)
    for k in ("logp", "lse", "dlogp", "dH", "dW", "loss", "adv", "stat_abs"):
        assert np.array_equal(a[k], b[k]), k


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_workspace_contents_do_not_matter(dtype):
    # The ABI promises that workspace contents on entry do not matter.  A
    # workspace of 0xFF bytes (NaN in both dtypes) must give results
    # bit-identical to a zeroed one.  The shape is ragged everywhere
    # (T, V and the shard widths are not multiples of 8) so every padded
    # region of every transient operand is exercised.
    mc = _mc()
    lib = mc.load_library()
    d, V = 136, 1003
    case = small_case(scaled_config(1, d=d, V=V, dtype=dtype, seed=61))   # T = 613
    H, W, y = device_tensors(case)
    T = H.shape[0]
    code = 1 if dtype == "bf16" else 0
    rng = np.random.default_rng(62)
    dl = torch.from_numpy((rng.standard_normal(T) * 1e-2).astype(np.float32)).cuda()

    def ws(nbytes, fill):
        return torch.full((max(int(nbytes), 1),), fill, dtype=torch.uint8, device="cuda")

    outs = []
    for fill in (0, 255):
        f_ws = ws(lib.mc_logprob_fwd_workspace_size(T, d, V, code), fill)
        logp, lse = mc.logprob_fwd(H, W, y, workspace=f_ws)
        b_ws = ws(lib.mc_logprob_bwd_workspace_size(T, d, V, code), fill)
        dH, dW = mc.logprob_bwd(H, W, y, lse, dl, workspace=b_ws)
        Ws = W[300:1003].contiguous()
        s_ws = ws(lib.mc_logprob_bwd_workspace_size(T, d, Ws.shape[0], code), fill)
        sh, sw = mc.logprob_bwd_shard(H, Ws, y, lse, dl, 300, V, workspace=s_ws)
        torch.cuda.synchronize()
        outs.append((logp, lse, dH, dW, sh, sw))
    for a, b in zip(*outs):
        assert torch.isfinite(b).all()
        assert torch.equal(a, b)
    lo, so = oracle.logprob_fwd(case["H"], case["W"], case["y"])
    dH_o, dW_o = oracle.logprob_bwd(case["H"], case["W"], case["y"], so,
                                    dl.cpu().numpy().astype(np.float64))
    assert np.max(np.abs(outs[1][0].cpu().numpy() - lo)) <= LOGP_ATOL
    assert rel_fro(outs[1][2].cpu().numpy(), dH_o) <= GRAD_RTOL
    assert rel_fro(outs[1][3].cpu().numpy(), dW_o) <= GRAD_RTOL


# ---------------------------------------------------------------------------
# mc_rl_loss alone: identical fp32 inputs on both sides
# ---------------------------------------------------------------------------
def _loss_parity(s, logp, lr, p):
    mc = _mc()
    st = structure_tensors(s)
    g = mc.rl_loss(torch.from_numpy(logp).cuda(), torch.from_numpy(lr).cuda(), st["mask"],
                   st["cu"], st["cg"], st["rewards"], to_params(p))
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in g.items()}
    o = oracle.rl_loss(logp, lr, s.loss_mask, s.cu_seqlens, s.cu_groups, s.rewards, p)
    assert g["error_flag"][0] == 0
    assert np.array_equal(g["seq_mask"], o["seq_mask"])
    assert np.array_equal(g["seq_len"], o["seq_len"])
    assert int(g["n_valid"][0]) == o["n_valid"]
    assert abs(g["loss"][0] - o["loss"]) <= LOSS_RTOL * max(abs(o["loss"]), 1e-30)
    np.testing.assert_allclose(g["dlogp"], o["dlogp"], rtol=1e-5, atol=1e-12)
    np.testing.assert_allclose(g["adv"], o["adv"], rtol=1e-6, atol=1e-7)
    np.testing.assert_allclose(g["stat_abs"], o["stat_abs"], rtol=1e-6, atol=1e-7)
    np.testing.assert_allclose(g["stat_signed"], o["stat_signed"], rtol=1e-6, atol=1e-7)
    assert abs(g["clip_frac"][0] - o["clip_frac"]) <= 1e-6
    return g, o


@pytest.mark.parametrize("cid", [1, 3, 4, 5])
@pytest.mark.parametrize("filt", ["mirrorpop", "vanilla", "none"])
def test_loss_full_size(cid, filt):
    s = make_structure(cid)
    rng = np.random.default_rng(100 + cid)
    logp = (-rng.uniform(0.5, 14.0, size=s.T)).astype(np.float32)
    lr = (logp.astype(np.float64) + s.rollout_delta).astype(np.float32)
    g, o = _loss_parity(s, logp, lr, oracle.RLParams(filter=filt))
    if cid == 4 and filt == "mirrorpop":
        assert o["seq_mask"][s.drifted].sum() == 0 and o["seq_mask"].sum() == s.B - 26


def test_loss_degenerate_cases():
    from workloads.gen import Structure
    # empty sequences, a group of one, equal rewards, all filtered
    cu = np.array([0, 0, 5, 5, 9, 12], np.int32)
    cg = np.array([0, 1, 4, 5], np.int32)
    mask = np.ones(12, np.uint8)
    mask[9:12] = 0
    s = Structure(cu, cg, mask, np.array([1, 0, 0, 0, 1], np.float32),
                  np.zeros(12, np.float32), np.zeros(5, bool))
    logp = -np.linspace(1, 5, 12).astype(np.float32)
    _loss_parity(s, logp, logp.copy(), oracle.RLParams())
    _loss_parity(s, logp, (logp + 1.0).astype(np.float32), oracle.RLParams())   # N = 0


def test_loss_flags_inconsistent_packing():
    mc = _mc()
    T = 10
    logp = torch.zeros(T, device="cuda")
    cu = torch.tensor([0, 4, 3, 10], dtype=torch.int32, device="cuda")    # decreasing
    cg = torch.tensor([0, 3], dtype=torch.int32, device="cuda")
    out = mc.rl_loss(logp, logp, None, cu, cg, torch.ones(3, device="cuda"))
    torch.cuda.synchronize()
    assert out["error_flag"].item() == 1


# ---------------------------------------------------------------------------
# Full-size workloads: sampled rows, same launch configuration as the bench
# ---------------------------------------------------------------------------
def _host_f32(t):
    return t.float().cpu().numpy()


@pytest.mark.parametrize("cid", [2, 4, 3, 5])
def test_fullsize_sampled(cid):
    mc = _mc()
    s, H, W, y = fullsize_inputs(cid)
    T, V = s.T, W.shape[0]
    logp, lse = mc.logprob_fwd(H, W, y)
    torch.cuda.synchronize()
    rows = sample_rows(T, 40, cid, extra=(T - 2, 8191, 8192))
    Hs = _host_f32(H[rows])
    Wh = _host_f32(W)
    ys = y[rows].cpu().numpy()
    lo, so = oracle.logprob_fwd(Hs, Wh, ys)
    assert np.max(np.abs(logp[rows].cpu().numpy() - lo)) <= LOGP_ATOL
    assert np.max(np.abs(lse[rows].cpu().numpy() - so)) <= LOGP_ATOL
    if CONFIGS[cid]["fwd_only"]:
        return
    # backward with dlogp nonzero on the sampled rows only: every other row of
    # the gradient of the logits is zero, so the oracle needs only these rows
    rng = np.random.default_rng(cid)
    dl = np.zeros(T, np.float32)
    dl[rows] = (rng.standard_normal(len(rows)) / T).astype(np.float32)
    dld = torch.from_numpy(dl).cuda()
    dH, dW = mc.logprob_bwd(H, W, y, lse, dld)
    torch.cuda.synchronize()
    lse_r = so
    dH_o = oracle.dhidden_rows(Hs, Wh, ys, lse_r, dl[rows].astype(np.float64))
    assert rel_fro(dH[rows].cpu().numpy(), dH_o) <= GRAD_RTOL
    others = torch.ones(T, dtype=torch.bool, device="cuda")
    others[torch.from_numpy(rows).cuda()] = False
    assert torch.count_nonzero(dH[others]).item() == 0
    vrows = np.unique(np.concatenate([ys[:16], rng.choice(V, 24, replace=False), [0, V - 1]]))
    dW_o = oracle.dweight_rows(Hs, Wh, ys, lse_r, dl[rows].astype(np.float64), vrows)
    assert rel_fro(dW[torch.from_numpy(vrows).cuda()].cpu().numpy(), dW_o) <= GRAD_RTOL
    del dH, dW
    torch.cuda.empty_cache()
