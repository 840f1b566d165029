"""The recompute backward's live-first token order, on the GPU, against the
oracle.

The recompute backward puts the tokens whose operand row can be nonzero
(nonzero dlogp, target in [0, V)) first.  Its softmax contraction skips the
256-token tiles of positions holding none of them, and the two gradient
contractions read the operand's rows past the live tokens as zeros (and
store dH's rows through the order).  Every result must be the one of the
plain definition:
dH and dW against the oracle for live sets of every size around the tile
edges (none, one, 255, 256, 257, all, scattered, only in the ragged last
tile, ignored targets with nonzero dlogp), exact zero rows of dH for the
dead tokens, and dH's live rows bit-identical to a call on the live tokens
alone (each row's logits, operand and contraction over the vocabulary do
not depend on where the token sits in the order).

MC_BWD_SKIP_DEAD_TOKENS makes dH and dW leave out the dead tokens' products,
which are exact zeros: dW must equal that of the call without it bit for
bit, and dH too up to the order of its fp32 sums (the live tiles' last
round is split along K when it would leave CUs idle), with the dead rows
exactly as without the flag; also when accumulating, and at full size on
the headline workload and on the 27B-class one (two vocabulary chunks),
through the chain bench.py times."""
import numpy as np
import pytest

import oracle
from _cases import (GRAD_RTOL, PTERM_RTOL_F16, device_tensors, fullsize_inputs, rel_fro,
                    structure_tensors, to_params)

# dH with MC_BWD_SKIP_DEAD_TOKENS against dH without: the same fp32 terms
# summed in another order (K slices), so within a few fp32 roundings
SKIP_DH_RTOL = 1e-6


def _same_dh(a, b, dead):
    """a, b: dH of the two calls (torch, on the GPU); dead: bool mask."""
    assert torch.equal(a[dead], b[dead])
    assert rel_fro(a.double().cpu().numpy(), b.double().cpu().numpy()) <= SKIP_DH_RTOL
from workloads import make_tensors_numpy, scaled_config

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

D, V = 128, 700   # a ragged vocabulary tile
# 1300 tokens: 5 whole token tiles and a ragged sixth.  5000 tokens: 20 token
# tile rows, which dH visits in a strided order (stride 3) once the live
# tokens come first.
T_SMALL, T_LARGE = 1300, 5000


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_04847_amd as mc
    mc.load_library()


def _live_set(kind, rng, T):
    live = np.zeros(T, dtype=bool)
    if kind == "one":
        live[T - 7] = True
    elif kind in ("255", "256", "257"):
        live[rng.choice(T, size=int(kind), replace=False)] = True
    elif kind == "all":
        live[:] = True
    elif kind == "scattered":
        live = rng.random(T) < 0.3
    elif kind == "ragged_tail":
        live[5 * 256 + 3: T - 2] = True
    elif kind == "spans":
        # long runs, like masked prompt / tool-output spans of packed sequences
        for a, b in ((0, 90), (300, 700), (1100, 1130)):
            live[a * T // T_SMALL:b * T // T_SMALL] = True
    return live


KINDS = ["none", "one", "255", "256", "257", "all", "scattered", "ragged_tail", "spans",
         "ignored"]


CASES = ([(k, dt, T_SMALL) for k in KINDS for dt in ("f32", "bf16")] +
         [(k, "bf16", T_LARGE) for k in ("scattered", "spans", "ignored")])


@pytest.mark.parametrize("kind,dtype,T", CASES)
def test_live_first_order(kind, dtype, T):
    import paper_2606_04847_amd as mc
    cfg = scaled_config(1, d=D, V=V, dtype=dtype, seed=61)
    Hn, Wn, hb, wb = make_tensors_numpy(cfg, T)
    rng = np.random.default_rng(62 + KINDS.index(kind) + T)
    y = rng.integers(0, V, size=T).astype(np.int64)
    dlogp = (rng.standard_normal(T) / T).astype(np.float32)
    if kind == "ignored":
        # a third of the tokens ignored (-1 or V) with nonzero dlogp: dead
        # all the same; a fifth of the rest with zero dlogp
        ign = rng.random(T) < 0.33
        y[ign] = np.where(rng.random(int(ign.sum())) < 0.5, -1, V)
        dlogp[~ign & (rng.random(T) < 0.2)] = 0.0
        live = ~ign & (dlogp != 0.0)
    else:
        live = _live_set(kind, rng, T)
        dlogp[~live] = 0.0
    case = dict(H=Hn, W=Wn, hb=hb, wb=wb, y=y)
    H, W, yd = device_tensors(case)
    dl = torch.from_numpy(dlogp).cuda()
    _, lse = mc.logprob_fwd(H, W, yd)
    dH, dW = mc.logprob_bwd(H, W, yd, lse, dl)
    dH_s, dW_s = mc.logprob_bwd(H, W, yd, lse, dl, skip_dead_tokens=True)
    torch.cuda.synchronize()
    assert torch.equal(dW, dW_s), (kind, dtype)
    if kind == "none":
        assert torch.equal(dH, dH_s)
    else:
        _same_dh(dH, dH_s, torch.from_numpy(~live).cuda())
    yc = np.where((y >= 0) & (y < V), y, -1)
    _, lse_o = oracle.logprob_fwd(Hn, Wn, yc)
    dl64 = dlogp.astype(np.float64)
    dH_o, dW_o = oracle.logprob_bwd(Hn, Wn, yc, lse_o, dl64)
    dH_g = dH.double().cpu().numpy()
    dW_g = dW.double().cpu().numpy()
    assert np.all(dH_g[~live] == 0.0), (kind, dtype)
    if not live.any():
        assert not dH_g.any() and not dW_g.any(), (kind, dtype)
        return
    assert rel_fro(dH_g, dH_o) <= GRAD_RTOL, (kind, dtype)
    assert rel_fro(dW_g, dW_o) <= GRAD_RTOL, (kind, dtype)
    # the softmax parts alone (the one-hot parts are exact in fp32)
    H64, W64 = Hn.astype(np.float64), Wn.astype(np.float64)
    g = np.where(yc >= 0, dl64, 0.0)
    onehot_h = g[:, None] * W64[np.maximum(yc, 0)]
    onehot_w = np.zeros_like(dW_o)
    np.add.at(onehot_w, np.maximum(yc, 0), g[:, None] * H64)
    assert rel_fro(dH_g - onehot_h, dH_o - onehot_h) <= PTERM_RTOL_F16, (kind, dtype)
    assert rel_fro(dW_g - onehot_w, dW_o - onehot_w) <= PTERM_RTOL_F16, (kind, dtype)
    if kind != "ignored":
        # the live tokens alone, in one call: the same rows of dH, bit for bit
        idx = torch.from_numpy(np.flatnonzero(live)).cuda()
        dH_l, _ = mc.logprob_bwd(H[idx].contiguous(), W, yd[idx].contiguous(),
                                 lse[idx].contiguous(), dl[idx].contiguous())
        torch.cuda.synchronize()
        assert torch.equal(dH[idx], dH_l), (kind, dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_skip_dead_tokens_accumulates_the_same(dtype):
    import paper_2606_04847_amd as mc
    T = T_LARGE
    cfg = scaled_config(1, d=D, V=V, dtype=dtype, seed=71)
    Hn, Wn, hb, wb = make_tensors_numpy(cfg, T)
    rng = np.random.default_rng(72)
    y = rng.integers(0, V, size=T).astype(np.int64)
    dlogp = (rng.standard_normal(T) / T).astype(np.float32)
    dlogp[_live_set("spans", rng, T) == 0] = 0.0
    H, W, yd = device_tensors(dict(H=Hn, W=Wn, hb=hb, wb=wb, y=y))
    dl = torch.from_numpy(dlogp).cuda()
    _, lse = mc.logprob_fwd(H, W, yd)
    g = torch.Generator(device="cuda").manual_seed(73)
    base_h = torch.randn(T, D, device="cuda", generator=g)
    base_w = torch.randn(V, D, device="cuda", generator=g)
    out = {}
    for skip in (False, True):
        dH, dW = base_h.clone(), base_w.clone()
        mc.logprob_bwd(H, W, yd, lse, dl, dhidden=dH, dweight=dW, accumulate_dhidden=True,
                       accumulate_dweight=True, skip_dead_tokens=skip)
        out[skip] = (dH, dW)
    torch.cuda.synchronize()
    dead = torch.from_numpy(dlogp == 0.0).cuda()
    assert torch.equal(out[False][1], out[True][1])
    _same_dh(out[False][0], out[True][0], dead)
    assert torch.equal(out[True][0][dead], base_h[dead])     # dead rows left as they were


@pytest.mark.parametrize("cid", [4, 3])
def test_skip_dead_tokens_full_size(cid):
    # the chain bench.py times, on the workload's own dlogp from the GPU loss
    import paper_2606_04847_amd as mc
    s, H, W, y = fullsize_inputs(cid)
    logp, lse = mc.logprob_fwd(H, W, y)
    lr = logp + torch.from_numpy(s.rollout_delta).cuda()
    st = structure_tensors(s)
    out = mc.rl_loss(logp, lr, st["mask"], st["cu"], st["cg"], st["rewards"],
                     to_params(oracle.RLParams()))
    dl = out["dlogp"]
    n_live = int(((dl != 0) & (y >= 0) & (y < W.shape[0])).sum().item())
    assert 0 < n_live < s.T
    dH, dW = mc.logprob_bwd(H, W, y, lse, dl)
    dH_s, dW_s = mc.logprob_bwd(H, W, y, lse, dl, skip_dead_tokens=True)
    torch.cuda.synchronize()
    print(f"[skip {cid}] T={s.T} live={n_live}", flush=True)
    assert torch.equal(dW, dW_s)
    _same_dh(dH, dH_s, ~((dl != 0) & (y >= 0) & (y < W.shape[0])))
