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
