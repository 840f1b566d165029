"""Pins for the oracle's per-token entropy, KL regulariser and PrimeEcho
reward: closed forms, the limits the paper states (Eq. 11), 50-digit brute
force and central finite differences."""
import math

import mpmath
import numpy as np
import pytest

from oracle import RLParams, rl_loss, token_entropy, trajectory_rewards


def test_entropy_closed_forms():
    H = np.random.default_rng(0).standard_normal((3, 8))
    for V in (1, 5, 1000):
        e = token_entropy(H, np.zeros((V, 8)))
        np.testing.assert_allclose(e, math.log(V), rtol=0, atol=1e-12)   # uniform: ln V
    W = np.random.default_rng(1).standard_normal((7, 8))
    e = token_entropy(H, W)
    assert np.all(e >= 0) and np.all(e <= math.log(7) + 1e-12)


def test_entropy_brute_force_50_digits():
    mpmath.mp.dps = 50
    rng = np.random.default_rng(2)
    H, W = rng.standard_normal((4, 3)), 2.0 * rng.standard_normal((6, 3))
    e = token_entropy(H, W)
    for t in range(4):
        z = [mpmath.fsum(mpmath.mpf(H[t, k]) * mpmath.mpf(W[v, k]) for k in range(3))
             for v in range(6)]
        Z = mpmath.fsum(mpmath.exp(x) for x in z)
        ref = -mpmath.fsum(mpmath.exp(x) / Z * (x - mpmath.log(Z)) for x in z)
        assert abs(float(ref) - e[t]) < 1e-13


def test_kl_single_token_closed_form():
    # one token, rho = 1, equal rewards (A = 0): only the KL term remains.
    # r = logp_ref - logp = ln 2: k3 = e^r - r - 1 = 1 - ln 2; d/dlogp = 1 - e^r = -1
    logp = np.array([-1.0])
    ref = logp + math.log(2.0)
    out = rl_loss(logp, logp, None, np.array([0, 1]), np.array([0, 1]), np.array([1.0]),
                  RLParams(kl_beta=0.5), logp_ref=ref)
    assert abs(out["kl"] - (1.0 - math.log(2.0))) < 1e-15
    assert abs(out["loss"] - 0.5 * (1.0 - math.log(2.0))) < 1e-15
    assert abs(out["dlogp"][0] - (-0.5)) < 1e-15
    # identical reference: KL 0 and no change to the loss or the gradient
    a = rl_loss(logp, logp, None, np.array([0, 1]), np.array([0, 1]), np.array([1.0]),
                RLParams(kl_beta=0.5), logp_ref=logp)
    assert a["kl"] == 0.0 and a["loss"] == 0.0 and a["dlogp"][0] == 0.0


@pytest.mark.parametrize("seed", [3, 4])
def test_kl_gradient_matches_central_differences(seed):
    rng = np.random.default_rng(seed)
    L = rng.integers(1, 8, size=8)
    cu = np.concatenate([[0], np.cumsum(L)]).astype(np.int32)
    T = int(cu[-1])
    groups = np.array([0, 4, 8], np.int32)
    rewards = rng.choice([0.0, 0.5, 1.0], size=8)
    logp = -rng.uniform(0.5, 6.0, size=T)
    lr = logp + rng.normal(0, 0.05, size=T)
    ref = logp + rng.normal(0, 0.3, size=T)
    mask = (rng.random(T) < 0.8).astype(np.uint8)
    p = RLParams(kl_beta=0.3, delta=1.0)
    out = rl_loss(logp, lr, mask, cu, groups, rewards, p, logp_ref=ref)
    assert out["kl"] >= 0.0
    h = 1e-7
    lo, hi = math.log(0.8), math.log(1.2)
    for t in range(T):
        if min(abs(logp[t] - lr[t] - lo), abs(logp[t] - lr[t] - hi)) < 1e-4:
            continue
        a, b = logp.copy(), logp.copy()
        a[t] += h
        b[t] -= h
        fa = rl_loss(a, lr, mask, cu, groups, rewards, p, logp_ref=ref)["loss"]
        fb = rl_loss(b, lr, mask, cu, groups, rewards, p, logp_ref=ref)["loss"]
        assert abs((fa - fb) / (2 * h) - out["dlogp"][t]) < 1e-7


def test_primeecho_limits_and_bonus():
    scores = np.array([[-1.0, 0.5, 1.2], [-0.5, 1.0, 0.0], [1.5, 0.0, 0.0], [-1.0, -1.0, -1.0]])
    success = np.array([[0, 0, 1], [0, 1, 0], [1, 0, 0], [0, 0, 0]], bool)
    K = np.array([3, 2, 1, 3])
    # Eq. 11: alpha = 1 -> first-turn score plus bonus; alpha = 0 -> best score plus bonus
    r1 = trajectory_rewards(scores, success, K, alpha=1.0, beta1=0.3, beta2=0.1)
    np.testing.assert_allclose(r1, [-1.0, -0.5 + 0.1, 1.5 + 0.3, -1.0], atol=1e-15)
    r0 = trajectory_rewards(scores, success, K, alpha=0.0, beta1=0.3, beta2=0.1)
    np.testing.assert_allclose(r0, [1.2, 1.0 + 0.1, 1.5 + 0.3, -1.0], atol=1e-15)
    # hand values at the paper's default alpha = 0.75 (Sec. 5.1)
    r = trajectory_rewards(scores, success, K, alpha=0.75, beta1=0.3, beta2=0.1)
    np.testing.assert_allclose(r, [0.75 * -1 + 0.25 * 1.2, 0.75 * -0.5 + 0.25 * 1.0 + 0.1,
                                   1.5 + 0.3, -1.0], atol=1e-15)
    # an earlier success earns at least as much as a later one (beta1 > beta2 >= 0)
    assert r1[2] - 1.5 > r1[1] + 0.5 > 0
