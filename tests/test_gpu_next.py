"""GPU parity of the rows beyond the core step: per-token entropy in the
forward epilogue, the vocabulary-sharded forward/merge/backward, the KL
regulariser of the objective and PrimeEcho rewards, against the oracle."""
import math

import numpy as np
import pytest

import oracle
from _cases import (GRAD_RTOL, LOGP_ATOL, LOSS_RTOL, device_tensors, rel_fro, small_case,
                    structure_tensors, to_params)
from workloads import make_tensors_numpy, scaled_config

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _mc():
    import paper_2606_04847_amd as mc
    return mc


def _case(dtype, T, d, V, seed, w_std=0.02):
    cfg = scaled_config(1, d=d, V=V, dtype=dtype, seed=seed, w_std=w_std)
    H, W, hb, wb = make_tensors_numpy(cfg, T)
    rng = np.random.default_rng(seed)
    y = rng.integers(0, V, size=T)
    y[2] = -1
    return dict(H=H, W=W, hb=hb, wb=wb, y=y), rng


@pytest.mark.parametrize("dtype,T,d,V,w_std", [("f32", 743, 128, 1024, 0.02),
                                               ("bf16", 600, 256, 3000, 0.02),
                                               ("bf16", 300, 512, 2000, 0.1)])
def test_entropy_matches_oracle(dtype, T, d, V, w_std):
    case, _ = _case(dtype, T, d, V, 31, w_std)
    mc = _mc()
    H, W, y = device_tensors(case)
    logp, lse, ent = mc.logprob_fwd(H, W, y, with_entropy=True)
    torch.cuda.synchronize()
    e_o = oracle.token_entropy(case["H"], case["W"])
    assert np.max(np.abs(ent.cpu().numpy() - e_o)) <= LOGP_ATOL
    # the entropy pass leaves logp and lse exactly as without it
    l2, s2 = mc.logprob_fwd(H, W, y)
    assert torch.equal(l2, logp) and torch.equal(s2, lse)


def test_entropy_uniform_closed_form():
    mc = _mc()
    T, d, V = 300, 64, 1000
    H = torch.randn(T, d, device="cuda").to(torch.bfloat16)
    W = torch.zeros(V, d, device="cuda", dtype=torch.bfloat16)
    y = torch.randint(0, V, (T,), device="cuda")
    _, _, ent = mc.logprob_fwd(H, W, y, with_entropy=True)
    assert torch.allclose(ent, torch.full_like(ent, math.log(V)), atol=2e-6, rtol=0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_vocab_shards_match_full(dtype):
    # three uneven shards of a 3000-entry vocabulary (ragged tiles in each);
    # targets land in every shard, one target is ignored
    T, d, V = 700, 136, 3000
    case, rng = _case(dtype, T, d, V, 41)
    bounds = [0, 1000, 2300, V]
    mc = _mc()
    H, W, y = device_tensors(case)
    parts = torch.stack([mc.logprob_fwd_shard(H, W[a:b].contiguous(), y, a, V)
                         for a, b in zip(bounds[:-1], bounds[1:])])
    logp, lse, ent = mc.logprob_merge_shards(parts, y, V)
    torch.cuda.synchronize()
    lo, so = oracle.logprob_fwd(case["H"], case["W"], case["y"])
    eo = oracle.token_entropy(case["H"], case["W"])
    assert np.max(np.abs(logp.cpu().numpy() - lo)) <= LOGP_ATOL
    assert np.max(np.abs(lse.cpu().numpy() - so)) <= LOGP_ATOL
    assert np.max(np.abs(ent.cpu().numpy() - eo)) <= LOGP_ATOL
    assert logp[2].item() == 0.0
    # backward per shard with the merged lse: shard parts of dH sum to dH,
    # shard rows of dW assemble dW
    dl = (rng.standard_normal(T) * 1e-2).astype(np.float32)
    dld = torch.from_numpy(dl).cuda()
    dH = np.zeros((T, d))
    dWs = []
    for a, b in zip(bounds[:-1], bounds[1:]):
        h, w = mc.logprob_bwd_shard(H, W[a:b].contiguous(), y, lse, dld, a, V)
        torch.cuda.synchronize()
        dH += h.cpu().numpy().astype(np.float64)
        dWs.append(w.cpu().numpy())
    dH_o, dW_o = oracle.logprob_bwd(case["H"], case["W"], case["y"], so, dl.astype(np.float64))
    assert rel_fro(dH, dH_o) <= GRAD_RTOL
    assert rel_fro(np.concatenate(dWs), dW_o) <= GRAD_RTOL
    # each shard's backward with MC_BWD_SKIP_DEAD_TOKENS (two thirds of the
    # tokens with zero dlogp): the shard's dW rows bit for bit, its dH part up
    # to the order of fp32 sums, dead rows exactly zero
    dl[rng.random(T) < 0.67] = 0.0
    dld = torch.from_numpy(dl).cuda()
    dead = torch.from_numpy(dl == 0.0).cuda()
    for a, b in zip(bounds[:-1], bounds[1:]):
        Ws = W[a:b].contiguous()
        h, w = mc.logprob_bwd_shard(H, Ws, y, lse, dld, a, V)
        hs, ws = mc.logprob_bwd_shard(H, Ws, y, lse, dld, a, V, skip_dead_tokens=True)
        torch.cuda.synchronize()
        assert torch.equal(w, ws), (a, b)
        assert not hs[dead].any() and not h[dead].any(), (a, b)
        assert rel_fro(hs.double().cpu().numpy(), h.double().cpu().numpy()) <= 1e-6, (a, b)


def test_vocab_shards_full_size():
    # one GPU's real shard shape: the headline workload (T = 16384, d = 4096,
    # V = 151936, bf16) split into 8 shards of V/8 = 18992 rows (ragged
    # 256-row tiles in each).  Merged shard partials against the unsharded
    # forward on every row and the oracle on sampled rows; the shards' dH parts
    # (summed) and dW rows (assembled) against the unsharded backward, whose
    # parity with the oracle at this size is tested elsewhere.
    from workloads import make_tensors_torch, sample_targets_torch
    T, d, V, S = 16384, 4096, 151936, 8
    cfg = scaled_config(4, T=T, d=d, V=V, seed=81)
    H, W = make_tensors_torch(cfg, T, "cuda")
    y = sample_targets_torch(cfg, H, W)
    y[5] = -1
    mc = _mc()
    logp_f, lse_f = mc.logprob_fwd(H, W, y)
    rng = np.random.default_rng(82)
    dl = (rng.standard_normal(T) / T).astype(np.float32)
    dl[rng.random(T) < 0.5] = 0.0
    dld = torch.from_numpy(dl).cuda()
    dH_f, dW_f = mc.logprob_bwd(H, W, y, lse_f, dld)
    Vs = V // S
    bounds = [k * Vs for k in range(S)] + [V]
    parts = torch.stack([mc.logprob_fwd_shard(H, W[a:b].contiguous(), y, a, V)
                         for a, b in zip(bounds[:-1], bounds[1:])])
    logp_s, lse_s, _ = mc.logprob_merge_shards(parts, y, V)
    dH_s = torch.zeros(T, d, dtype=torch.float64, device="cuda")
    dW_s = []
    for a, b in zip(bounds[:-1], bounds[1:]):
        h, w = mc.logprob_bwd_shard(H, W[a:b].contiguous(), y, lse_s, dld, a, V)
        dH_s += h.double()
        dW_s.append(w)
    dW_s = torch.cat(dW_s)
    torch.cuda.synchronize()
    assert torch.max(torch.abs(logp_s - logp_f)).item() <= 1e-4
    assert torch.max(torch.abs(lse_s - lse_f)).item() <= 1e-4
    assert logp_s[5].item() == 0.0
    rows = np.unique(np.concatenate([rng.choice(T, 60, replace=False), [0, T - 1]]))
    Hh = H[torch.from_numpy(rows).cuda()].float().cpu().numpy()
    Wh = W.float().cpu().numpy()
    lo, so = oracle.logprob_fwd(Hh, Wh, y[torch.from_numpy(rows).cuda()].cpu().numpy())
    assert np.max(np.abs(logp_s.cpu().numpy()[rows] - lo)) <= LOGP_ATOL
    assert np.max(np.abs(lse_s.cpu().numpy()[rows] - so)) <= LOGP_ATOL

    def rel(a, b):
        return (torch.linalg.vector_norm((a.double() - b.double()).flatten())
                / torch.linalg.vector_norm(b.double().flatten())).item()
    assert rel(dH_s, dH_f) <= 1e-5
    assert rel(dW_s, dW_f) <= 1e-5
    print(f"[shards 8 x {Vs}] |dlogp| {torch.max(torch.abs(logp_s - logp_f)).item():.2e} "
          f"dH {rel(dH_s, dH_f):.2e} dW {rel(dW_s, dW_f):.2e}", flush=True)


@pytest.mark.parametrize("beta", [0.05, 0.5])
def test_kl_term_matches_oracle(beta):
    cfg = scaled_config(4, T=1200, n_groups=4, group_size=8, hi=300, seed=51,
                        drift=dict(kind="frac_normal", count=3, mean=0.3, std=0.1))
    from workloads import make_structure
    s = make_structure(cfg)
    rng = np.random.default_rng(52)
    logp = (-rng.uniform(0.5, 10.0, size=s.T)).astype(np.float32)
    lr = (logp.astype(np.float64) + s.rollout_delta).astype(np.float32)
    ref = (logp + rng.normal(0, 0.2, size=s.T)).astype(np.float32)
    p = oracle.RLParams(kl_beta=beta)
    o = oracle.rl_loss(logp, lr, s.loss_mask, s.cu_seqlens, s.cu_groups, s.rewards, p,
                       logp_ref=ref)
    mc = _mc()
    st = structure_tensors(s)
    g = mc.rl_loss(torch.from_numpy(logp).cuda(), torch.from_numpy(lr).cuda(), st["mask"],
                   st["cu"], st["cg"], st["rewards"], to_params(p),
                   logp_ref=torch.from_numpy(ref).cuda())
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in g.items()}
    assert np.array_equal(g["seq_mask"], o["seq_mask"]) and int(g["n_valid"][0]) == o["n_valid"]
    assert abs(g["kl"][0] - o["kl"]) <= 1e-5 * max(o["kl"], 1e-30)
    assert abs(g["loss"][0] - o["loss"]) <= LOSS_RTOL * abs(o["loss"])
    np.testing.assert_allclose(g["dlogp"], o["dlogp"], rtol=1e-5, atol=1e-12)


def test_primeecho_rewards_match_oracle_and_feed_the_loss():
    rng = np.random.default_rng(61)
    B, K = 64, 3
    scores = rng.choice([-1.0, -0.5, 0.0, 0.3, 1.0, 1.4], size=(B, K)).astype(np.float32)
    success = (scores >= 1.0).astype(np.uint8)
    n_turns = rng.integers(1, K + 1, size=B).astype(np.int32)
    mc = _mc()
    for alpha, b1, b2 in ((0.75, 0.2, 0.1), (1.0, 0.0, 0.0), (0.0, 0.3, 0.05)):
        r = mc.primeecho_rewards(torch.from_numpy(scores).cuda(), torch.from_numpy(success).cuda(),
                                 torch.from_numpy(n_turns).cuda(), alpha=alpha, beta1=b1, beta2=b2)
        torch.cuda.synchronize()
        ro = oracle.trajectory_rewards(scores, success, n_turns, alpha, b1, b2)
        np.testing.assert_allclose(r.cpu().numpy(), ro, rtol=1e-6, atol=1e-6)
    # Eq. 12: the group-normalised advantage of the PrimeEcho reward
    T = 8 * B
    cu = (np.arange(B + 1) * 8).astype(np.int32)
    cg = (np.arange(B // 8 + 1) * 8).astype(np.int32)
    logp = (-rng.uniform(1, 5, size=T)).astype(np.float32)
    g = mc.rl_loss(torch.from_numpy(logp).cuda(), torch.from_numpy(logp).cuda(), None,
                   torch.from_numpy(cu).cuda(), torch.from_numpy(cg).cuda(), r)
    torch.cuda.synchronize()
    o = oracle.rl_loss(logp, logp, None, cu, cg, r.cpu().numpy())
    np.testing.assert_allclose(g["adv"].cpu().numpy(), o["adv"], rtol=1e-6, atol=1e-6)


# ---------------------------------------------------------------------------
# Token-level modes of the objective (TIS / IcePop readings)
# ---------------------------------------------------------------------------
def _wide_offsets(T, rng, edges, sigma=0.4, margin=5e-3):
    """Per-token log-ratio offsets spread wide enough that many tokens fall
    outside the token-mode bounds, kept `margin` away from every decision
    edge (clip edges and the mode's bounds), so every decision is unique."""
    x = rng.normal(0.0, sigma, size=T)
    for _ in range(1000):
        bad = np.zeros(T, bool)
        for e in edges:
            bad |= np.abs(-x - e) < margin
        if not bad.any():
            return x
        x[bad] = rng.normal(0.0, sigma, size=int(bad.sum()))
    raise RuntimeError("margin not reachable")


_TOKEN_MODES = [("tis", dict(tis_cap=1.5)), ("icepop", dict(icepop_lo=0.75, icepop_hi=1.3))]


def _edges(p):
    return [math.log(1 - p.eps_low), math.log(1 + p.eps_high),
            math.log(float(np.float32(p.tis_cap))), math.log(float(np.float32(p.icepop_lo))),
            math.log(float(np.float32(p.icepop_hi)))]


@pytest.mark.parametrize("cid", [3, 4, 5])
@pytest.mark.parametrize("mode,kw", _TOKEN_MODES)
def test_token_mode_loss_full_size(cid, mode, kw):
    from workloads import make_structure
    mc = _mc()
    s = make_structure(cid)
    p = oracle.RLParams(filter="none", token_mode=mode, **kw)
    rng = np.random.default_rng(200 + cid)
    logp = (-rng.uniform(0.5, 12.0, size=s.T)).astype(np.float32)
    x = _wide_offsets(s.T, rng, _edges(p))
    lr = (logp.astype(np.float64) + x).astype(np.float32)
    # the fp32 rounding of lr must not move a token across an edge
    ell = logp.astype(np.float64) - lr.astype(np.float64)
    assert min(np.min(np.abs(ell - e)) for e in _edges(p)) > 1e-3
    st = structure_tensors(s)
    g = mc.rl_loss(torch.from_numpy(logp).cuda(), torch.from_numpy(lr).cuda(), st["mask"],
                   st["cu"], st["cg"], st["rewards"], to_params(p))
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in g.items()}
    o = oracle.rl_loss(logp, lr, s.loss_mask, s.cu_seqlens, s.cu_groups, s.rewards, p)
    assert 0.05 < o["token_frac"] < 0.95                 # the mode really acts
    assert int(g["n_valid"][0]) == o["n_valid"]
    assert abs(g["loss"][0] - o["loss"]) <= LOSS_RTOL * abs(o["loss"])
    np.testing.assert_allclose(g["dlogp"], o["dlogp"], rtol=1e-5, atol=1e-12)
    assert np.array_equal(g["dlogp"] == 0.0, o["dlogp"] == 0.0)
    assert abs(g["token_frac"][0] - o["token_frac"]) <= 1e-6
    assert abs(g["clip_frac"][0] - o["clip_frac"]) <= 1e-6


@pytest.mark.parametrize("mode,kw", _TOKEN_MODES)
def test_token_mode_end_to_end(mode, kw):
    # GPU forward -> loss with the token mode -> backward, against the oracle
    from _cases import assert_step_parity, gpu_step
    cfg = scaled_config(4, T=1200, n_groups=4, group_size=8, d=256, V=1500, hi=200, seed=17,
                        drift=dict(kind="frac_normal", count=3, mean=0.3, std=0.1))
    case = small_case(cfg)
    p = oracle.RLParams(filter="mirrorpop", delta=0.24, token_mode=mode, **kw)
    s = case["s"]
    logp, lse = oracle.logprob_fwd(case["H"], case["W"], case["y"])
    rng = np.random.default_rng(18)
    x = _wide_offsets(s.T, rng, _edges(p), sigma=0.3)
    lr = (logp + x).astype(np.float32)
    o = oracle.rl_loss(logp, lr, s.loss_mask, s.cu_seqlens, s.cu_groups, s.rewards, p)
    assert 0.05 < o["token_frac"] < 0.95
    assert np.min(np.abs(o["stat_abs"] - p.delta)) > 1e-3      # unique sequence decisions
    assert 0 < o["seq_mask"].sum() < s.B
    dH, dW = oracle.logprob_bwd(case["H"], case["W"], case["y"], lse, o["dlogp"])
    o = dict(o, logp=logp, lse=lse, dH=dH, dW=dW)
    g = gpu_step(case, p, lr)
    assert_step_parity(g, o)


def test_side_stream_calls_match_current_stream():
    # every wrapper records the caller's stream on what it allocates: results
    # computed on a side stream while the current stream allocates and fills
    # memory of the same sizes are those of the current stream, bit for bit
    from _cases import gpu_step
    cfg = scaled_config(4, T=900, n_groups=2, group_size=8, d=256, V=1300, hi=150, seed=19,
                        drift=dict(kind="frac_normal", count=2, mean=0.3, std=0.1))
    case = small_case(cfg)
    p = oracle.RLParams()
    lr = (oracle.logprob_fwd(case["H"], case["W"], case["y"])[0]
          + case["s"].rollout_delta).astype(np.float32)
    ref = gpu_step(case, p, lr)
    mc = _mc()
    H, W, y = device_tensors(case)
    st = structure_tensors(case["s"])
    lrd = torch.from_numpy(lr).cuda()
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    res = []
    for _ in range(3):
        logp, lse = mc.logprob_fwd(H, W, y, stream=side)
        out = mc.rl_loss(logp, lrd, st["mask"], st["cu"], st["cg"], st["rewards"],
                         to_params(p), stream=side)
        dH, dW = mc.logprob_bwd(H, W, y, lse, out["dlogp"], stream=side)
        # the current stream churns the allocator meanwhile
        junk = [torch.full((n,), -7.0, device="cuda") for n in
                (H.shape[0], W.shape[0] * W.shape[1], H.shape[0] * H.shape[1], 1 << 20)]
        del junk
        res.append((logp, lse, out["dlogp"], dH, dW))
    side.synchronize()
    torch.cuda.synchronize()
    for logp, lse, dl, dH, dW in res:
        assert np.array_equal(logp.cpu().numpy(), ref["logp"])
        assert np.array_equal(lse.cpu().numpy(), ref["lse"])
        assert np.array_equal(dl.cpu().numpy(), ref["dlogp"])
        assert np.array_equal(dH.cpu().numpy(), ref["dH"])
        assert np.array_equal(dW.cpu().numpy(), ref["dW"])
