"""Pins for the oracle's RL objective (Eq. 3/12, 4, 5, 17-21).

Values come from the paper's worked example, hand derivations from the
definitions (fixtures under tests/golden), closed forms and central finite
differences of the loss; none is recomputed with the oracle's own formula.
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import RLParams, rl_loss

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_paper_cancellation_example():
    g = _load("mirrorpop_cancellation.json")
    rho = np.array(g["rho"])
    ell = np.log(rho)
    logp_r = np.zeros(2)
    cu = np.array([0, 2], np.int32)
    groups = np.array([0, 1], np.int32)
    for filt, kept in (("mirrorpop", 0), ("vanilla", 1), ("none", 1)):
        out = rl_loss(ell, logp_r, None, cu, groups, np.array([1.0]),
                      RLParams(filter=filt, delta=0.1))
        assert abs(out["stat_signed"][0] - g["signed_mean_log_ratio"]) < 1e-15
        assert abs(math.exp(out["stat_signed"][0]) - g["geometric_mean_ratio"]) < 1e-15
        assert abs(out["stat_abs"][0] - math.log(10.0)) < 1e-15
        assert abs(math.exp(out["stat_abs"][0]) - g["mirrorpop_ratio_space_magnitude"]) < 1e-13
        assert out["seq_mask"][0] == kept
    # MirrorPop removes it for any threshold below ln 10 and keeps it above.
    for delta, kept in ((2.30, 0), (2.31, 1)):
        out = rl_loss(ell, logp_r, None, cu, groups, np.array([1.0]),
                      RLParams(delta=delta))
        assert out["seq_mask"][0] == kept
    # Eq. 19: m_t = exp|ell_t| = max(rho, 1/rho) = 10 for both tokens.
    np.testing.assert_allclose(np.exp(np.abs(ell)), g["mirror_deviation_per_token"],
                               rtol=1e-15)


def test_hand_derived_clip_cases():
    g = _load("clip_cases.json")
    p = RLParams(**g["params"])
    ell = np.log(np.array(g["rho"]))
    out = rl_loss(ell, np.zeros_like(ell), None, np.array(g["cu_seqlens"]),
                  np.array(g["cu_groups"]), np.array(g["rewards"]), p)
    np.testing.assert_allclose(out["adv"], g["adv"], rtol=0, atol=1e-15)
    assert out["n_valid"] == g["n_valid"]
    assert abs(out["loss"] - g["loss"]) < 1e-14
    np.testing.assert_allclose(out["dlogp"], g["dlogp"], rtol=0, atol=1e-14)
    assert abs(out["clip_frac"] - g["clip_frac"]) < 1e-15


def _batch(seed, B=12, G=4, maxlen=9, masked=True):
    rng = np.random.default_rng(seed)
    L = rng.integers(1, maxlen + 1, size=B)
    cu = np.concatenate([[0], np.cumsum(L)]).astype(np.int32)
    T = int(cu[-1])
    groups = np.arange(0, B + 1, G).astype(np.int32)
    mask = (rng.random(T) < 0.7).astype(np.uint8) if masked else np.ones(T, np.uint8)
    rewards = rng.choice([0.0, 0.25, 0.5, 1.0], size=B)
    logp = -rng.uniform(0.5, 8.0, size=T)
    return cu, groups, mask, rewards, logp, rng


def test_identical_rollout_closed_form():
    # rho = 1 everywhere: nothing is filtered, no token is clipped and
    # loss = -sum_i L_i A_i / sum_i L_i, dlogp_t = -A_i / N on valid tokens.
    cu, groups, mask, rewards, logp, _ = _batch(1)
    out = rl_loss(logp, logp, mask, cu, groups, rewards, RLParams())
    L = np.array([mask[cu[i]:cu[i + 1]].sum() for i in range(len(cu) - 1)])
    assert np.all(out["seq_mask"] == (L > 0))
    assert np.all(out["stat_abs"] == 0.0)
    N = int(L.sum())
    assert out["n_valid"] == N
    A = out["adv"]
    assert abs(out["loss"] - (-(L * A).sum() / N)) < 1e-15
    for i in range(len(L)):
        seg = slice(cu[i], cu[i + 1])
        np.testing.assert_allclose(out["dlogp"][seg],
                                   np.where(mask[seg] > 0, -A[i] / N, 0.0), atol=1e-17)
    assert out["clip_frac"] == 0.0


def test_identical_rollout_equal_lengths_gives_zero_loss():
    # Equal L_i within each group and rho = 1: the loss is -sum_g L sum_i A_i / N
    # and the advantages of a group sum to zero.
    B, G, L = 8, 4, 5
    cu = (np.arange(B + 1) * L).astype(np.int32)
    groups = np.arange(0, B + 1, G).astype(np.int32)
    rewards = np.array([0, 1, 1, 0.5, 0, 0, 0.25, 1.0])
    logp = -np.linspace(1, 3, B * L)
    out = rl_loss(logp, logp, None, cu, groups, rewards, RLParams())
    assert abs(out["loss"]) < 1e-15


def test_advantage_identities():
    rng = np.random.default_rng(3)
    r = rng.random(8)
    cu = np.arange(9).astype(np.int32)
    logp = np.zeros(8)
    for eps in (1e-6, 0.0):
        out = rl_loss(logp, logp, None, cu, np.array([0, 8]), r, RLParams(adv_eps=eps))
        A = out["adv"]
        sigma = r.std()
        assert abs(A.sum()) < 1e-13
        assert abs(A.std() - sigma / (sigma + eps)) < 1e-13
    # two sequences with rewards (0, 1): A = -+0.5/(0.5 + eps)
    out = rl_loss(np.zeros(2), np.zeros(2), None, np.array([0, 1, 2]),
                  np.array([0, 2]), np.array([0.0, 1.0]), RLParams())
    np.testing.assert_allclose(out["adv"], [-0.5 / (0.5 + 1e-6), 0.5 / (0.5 + 1e-6)],
                               rtol=1e-15)
    # an all-failed group (every reward equal, the Eq. 13 case) has A = 0
    out = rl_loss(np.zeros(4), np.zeros(4), None, np.arange(5), np.array([0, 4]),
                  np.full(4, -1.0), RLParams())
    assert np.all(out["adv"] == 0.0)
    # sample standard deviation when ddof = 1
    out = rl_loss(np.zeros(3), np.zeros(3), None, np.arange(4), np.array([0, 3]),
                  np.array([0.0, 1.0, 2.0]), RLParams(std_ddof=1, adv_eps=0.0))
    np.testing.assert_allclose(out["adv"], [-1.0, 0.0, 1.0], atol=1e-15)


def test_everything_filtered_gives_zero():
    cu, groups, mask, rewards, logp, _ = _batch(4)
    out = rl_loss(logp, logp + 1.0, mask, cu, groups, rewards, RLParams(delta=0.5))
    assert out["n_valid"] == 0 and out["loss"] == 0.0
    assert np.all(out["dlogp"] == 0.0) and np.all(out["seq_mask"] == 0)


def test_empty_sequences_contribute_nothing():
    cu = np.array([0, 0, 3, 3, 5], np.int32)
    groups = np.array([0, 4], np.int32)
    logp = -np.ones(5)
    out = rl_loss(logp, logp, None, cu, groups, np.array([1.0, 0.0, 1.0, 0.0]))
    assert list(out["seq_len"]) == [0, 3, 0, 2]
    assert list(out["seq_mask"]) == [0, 1, 0, 1]
    assert out["n_valid"] == 5


def test_statistic_triangle_inequality():
    cu, groups, mask, rewards, logp, rng = _batch(5)
    out = rl_loss(logp, logp + rng.normal(0, 0.3, size=len(logp)), mask, cu, groups,
                  rewards)
    assert np.all(out["stat_abs"] >= np.abs(out["stat_signed"]) - 1e-15)
    assert np.all(np.exp(out["stat_abs"]) >= 1.0)


def test_filter_reduces_to_plain_grpo_when_all_kept():
    # Eq. 17 with every M_i = 1 is Eq. 5: same loss as the unfiltered objective.
    cu, groups, mask, rewards, logp, rng = _batch(6, masked=False)
    lr = logp + rng.normal(0, 0.01, size=len(logp))
    a = rl_loss(logp, lr, None, cu, groups, rewards, RLParams(filter="mirrorpop", delta=10))
    b = rl_loss(logp, lr, None, cu, groups, rewards, RLParams(filter="none"))
    assert a["loss"] == b["loss"] and np.all(a["dlogp"] == b["dlogp"])


@pytest.mark.parametrize("seed", [7, 8, 9])
def test_dlogp_matches_central_differences(seed):
    cu, groups, mask, rewards, logp, rng = _batch(seed)
    lr = logp + rng.normal(0, 0.15, size=len(logp))
    p = RLParams(delta=0.2)
    out = rl_loss(logp, lr, mask, cu, groups, rewards, p)
    h = 1e-7
    lo, hi = math.log(1 - p.eps_low), math.log(1 + p.eps_high)
    for t in range(len(logp)):
        ell = logp[t] - lr[t]
        if min(abs(ell - lo), abs(ell - hi)) < 1e-4:
            continue   # at a kink the derivative is one-sided
        lp, lm = logp.copy(), logp.copy()
        lp[t] += h
        lm[t] -= h
        fp = rl_loss(lp, lr, mask, cu, groups, rewards, p)
        fm = rl_loss(lm, lr, mask, cu, groups, rewards, p)
        if not (np.array_equal(fp["seq_mask"], out["seq_mask"])
                and np.array_equal(fm["seq_mask"], out["seq_mask"])):
            continue   # the filter decision itself moved: no derivative
        fd = (fp["loss"] - fm["loss"]) / (2 * h)
        assert abs(fd - out["dlogp"][t]) < 1e-7


# ---------------------------------------------------------------------------
# Token-level modes (readings R12 / R13 of the oracle)
# ---------------------------------------------------------------------------
def _token_params(g, mode):
    kw = dict(g["params"])
    return RLParams(token_mode=mode, **kw)


@pytest.mark.parametrize("mode", ["none", "tis", "icepop"])
def test_hand_derived_token_modes(mode):
    g = _load("token_modes.json")
    ell = np.log(np.array(g["rho"]))
    out = rl_loss(ell, np.zeros_like(ell), None, np.array(g["cu_seqlens"]),
                  np.array(g["cu_groups"]), np.array(g["rewards"]), _token_params(g, mode))
    want = g["modes"][mode]
    np.testing.assert_allclose(out["adv"], g["adv"], rtol=0, atol=1e-15)
    assert out["n_valid"] == g["n_valid"]
    assert abs(out["loss"] - want["loss"]) < 1e-14
    np.testing.assert_allclose(out["dlogp"], want["dlogp"], rtol=0, atol=1e-14)
    assert abs(out["clip_frac"] - want["clip_frac"]) < 1e-15
    assert abs(out["token_frac"] - want["token_frac"]) < 1e-15


@pytest.mark.parametrize("mode", ["tis", "icepop"])
def test_token_modes_without_tokens_outside_bounds_equal_the_base_loss(mode):
    # every ratio inside [0.5, 2] (and below the cap 2): nothing to truncate or
    # drop, so the objective and its gradient are those of Eq. 17 unchanged
    cu, groups, mask, rewards, logp, rng = _batch(21)
    lr = logp + rng.normal(0, 0.1, size=len(logp))
    assert np.all(np.abs(logp - lr) < math.log(2.0) - 1e-3)
    base = rl_loss(logp, lr, mask, cu, groups, rewards, RLParams(delta=0.3))
    out = rl_loss(logp, lr, mask, cu, groups, rewards, RLParams(delta=0.3, token_mode=mode))
    assert out["loss"] == base["loss"] and np.array_equal(out["dlogp"], base["dlogp"])
    assert out["token_frac"] == 0.0 and out["clip_frac"] == base["clip_frac"]


def test_token_modes_reduce_to_the_base_loss_in_their_limits():
    # an unbounded cap / interval touches no token
    cu, groups, mask, rewards, logp, rng = _batch(22)
    lr = logp + rng.normal(0, 1.0, size=len(logp))
    p = dict(delta=10.0, filter="none")
    base = rl_loss(logp, lr, mask, cu, groups, rewards, RLParams(**p))
    tis = rl_loss(logp, lr, mask, cu, groups, rewards,
                  RLParams(token_mode="tis", tis_cap=1e30, **p))
    ice = rl_loss(logp, lr, mask, cu, groups, rewards,
                  RLParams(token_mode="icepop", icepop_lo=1e-30, icepop_hi=1e30, **p))
    for o in (tis, ice):
        assert o["loss"] == base["loss"] and np.array_equal(o["dlogp"], base["dlogp"])


def test_tis_truncated_tokens_keep_a_bounded_gradient():
    # a negative-advantage token far above the clip range: on the unclipped
    # branch of Eq. 5 its gradient grows with rho; truncated it stays at C A
    cu = np.array([0, 1, 2], np.int32)
    groups = np.array([0, 2], np.int32)
    rewards = np.array([1.0, 0.0])                  # A = (+1, -1) with eps 0
    for rho in (3.0, 30.0, 3000.0):
        ell = np.array([0.0, math.log(rho)])
        p = RLParams(filter="none", adv_eps=0.0, token_mode="tis", tis_cap=2.0)
        out = rl_loss(ell, np.zeros(2), None, cu, groups, rewards, p)
        assert abs(out["dlogp"][1] - 2.0 / 2) < 1e-15          # -(1/N) C A, N = 2
        base = rl_loss(ell, np.zeros(2), None, cu, groups, rewards,
                       RLParams(filter="none", adv_eps=0.0))
        assert abs(base["dlogp"][1] - rho / 2) < 1e-12 * rho


@pytest.mark.parametrize("seed", [23, 24])
def test_icepop_dlogp_matches_central_differences(seed):
    # the IcePop mask is piecewise constant in logp, so away from its bounds
    # (and from the clip kinks) the gradient is the derivative of the loss
    cu, groups, mask, rewards, logp, rng = _batch(seed)
    lr = logp + rng.normal(0, 0.6, size=len(logp))
    p = RLParams(delta=10.0, token_mode="icepop", icepop_lo=0.7, icepop_hi=1.6)
    out = rl_loss(logp, lr, mask, cu, groups, rewards, p)
    assert 0.0 < out["token_frac"] < 1.0
    h = 1e-7
    edges = [math.log(1 - p.eps_low), math.log(1 + p.eps_high),
             math.log(float(np.float32(0.7))), math.log(float(np.float32(1.6)))]
    checked = 0
    for t in range(len(logp)):
        ell = logp[t] - lr[t]
        if min(abs(ell - e) for e in edges) < 1e-4:
            continue
        lp, lm = logp.copy(), logp.copy()
        lp[t] += h
        lm[t] -= h
        fp = rl_loss(lp, lr, mask, cu, groups, rewards, p)
        fm = rl_loss(lm, lr, mask, cu, groups, rewards, p)
        fd = (fp["loss"] - fm["loss"]) / (2 * h)
        assert abs(fd - out["dlogp"][t]) < 1e-7
        checked += 1
    assert checked > len(logp) // 2
