"""Pins for the oracle's log-prob forward and backward.

Each check compares the oracle against something that is not the oracle:
a closed form, brute force at 50 digits, an invariance of the softmax, or
central finite differences of the composite function.
"""
import math

import mpmath
import numpy as np
import pytest

from oracle import dhidden_rows, dweight_rows, logprob_bwd, logprob_fwd


def _rand(T, d, V, seed, wscale=0.5):
    rng = np.random.default_rng(seed)
    H = rng.standard_normal((T, d))
    W = wscale * rng.standard_normal((V, d))
    y = rng.integers(0, V, size=T)
    return H, W, y


def test_zero_weight_gives_minus_log_v_exactly():
    # W = 0: every logit is 0, lse = ln V, logp = -ln V (exact in fp64).
    for V in (1, 7, 1024, 151936):
        H = np.random.default_rng(V).standard_normal((3, 8))
        W = np.zeros((V, 8))
        y = np.array([0, V - 1, V // 2])
        logp, lse = logprob_fwd(H, W, y)
        assert np.all(lse == math.log(V))
        assert np.all(logp == -math.log(V))


def test_single_token_vocab_gives_zero():
    H, W, _ = _rand(4, 5, 1, 1)
    logp, lse = logprob_fwd(H, W, np.zeros(4, dtype=np.int64))
    assert np.all(logp == 0.0)
    np.testing.assert_allclose(lse, (H @ W.T)[:, 0], rtol=0, atol=1e-15)


def test_brute_force_50_digits():
    mpmath.mp.dps = 50
    H, W, y = _rand(5, 3, 7, 2, wscale=3.0)
    logp, lse = logprob_fwd(H, W, y)
    for t in range(5):
        z = [mpmath.fsum(mpmath.mpf(H[t, k]) * mpmath.mpf(W[v, k]) for k in range(3))
             for v in range(7)]
        # one-pass sum of exponentials, no max shift: a different algorithm
        ref_lse = mpmath.log(mpmath.fsum(mpmath.exp(zv) for zv in z))
        assert abs(float(ref_lse) - lse[t]) < 1e-13
        assert abs(float(z[y[t]] - ref_lse) - logp[t]) < 1e-13


def test_shift_invariance_of_softmax():
    # Adding the same vector c to every vocabulary row shifts row t of the
    # logits by h_t . c and leaves the log-softmax unchanged.
    H, W, y = _rand(6, 16, 50, 3)
    c = np.random.default_rng(9).standard_normal(16)
    a, _ = logprob_fwd(H, W, y)
    b, _ = logprob_fwd(H, W + c[None, :], y)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_vocab_permutation_equivariance():
    H, W, y = _rand(6, 16, 50, 4)
    perm = np.random.default_rng(5).permutation(50)
    inv = np.argsort(perm)
    a, la = logprob_fwd(H, W, y)
    b, lb = logprob_fwd(H, W[perm], inv[y])
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)
    np.testing.assert_allclose(la, lb, rtol=0, atol=1e-12)


def test_extreme_logits_stay_finite():
    # logits of +-1e4: the two-pass lse must not overflow.
    H = np.array([[100.0], [-100.0]])
    W = np.array([[100.0], [-100.0], [0.0]])
    logp, lse = logprob_fwd(H, W, np.array([0, 0]))
    assert np.isfinite(logp).all() and np.isfinite(lse).all()
    assert abs(logp[0]) < 1e-12 and abs(lse[0] - 1e4) < 1e-9
    assert abs(logp[1] + 2e4) < 1e-9


def test_ignored_targets():
    H, W, y = _rand(4, 8, 20, 6)
    y = y.copy()
    y[1] = -1
    y[3] = 20
    logp, lse = logprob_fwd(H, W, y)
    assert logp[1] == 0.0 and logp[3] == 0.0
    dH, dW = logprob_bwd(H, W, y, lse, np.ones(4))
    assert np.all(dH[1] == 0.0) and np.all(dH[3] == 0.0)


def _composite(H, W, y, c):
    logp, _ = logprob_fwd(H, W, y)
    return float(np.dot(c, logp))


@pytest.mark.parametrize("seed", [0, 1])
def test_gradients_match_central_differences(seed):
    H, W, y = _rand(5, 6, 9, seed + 10)
    c = np.random.default_rng(seed + 20).standard_normal(5)
    _, lse = logprob_fwd(H, W, y)
    dH, dW = logprob_bwd(H, W, y, lse, c)
    h = 1e-6
    rng = np.random.default_rng(seed + 30)
    for _ in range(12):
        t, k = rng.integers(5), rng.integers(6)
        Hp, Hm = H.copy(), H.copy()
        Hp[t, k] += h
        Hm[t, k] -= h
        fd = (_composite(Hp, W, y, c) - _composite(Hm, W, y, c)) / (2 * h)
        assert abs(fd - dH[t, k]) <= 1e-7 * max(1.0, abs(fd))
        v = rng.integers(9)
        Wp, Wm = W.copy(), W.copy()
        Wp[v, k] += h
        Wm[v, k] -= h
        fd = (_composite(H, Wp, y, c) - _composite(H, Wm, y, c)) / (2 * h)
        assert abs(fd - dW[v, k]) <= 1e-7 * max(1.0, abs(fd))


def test_vocab_gradient_sums_to_zero_and_zero_weight_gradient():
    # sum_v G_tv = dlogp_t (1 - sum_v p_tv) = 0, so the dW rows sum to 0.
    H, W, y = _rand(7, 5, 11, 7)
    c = np.random.default_rng(1).standard_normal(7)
    _, lse = logprob_fwd(H, W, y)
    _, dW = logprob_bwd(H, W, y, lse, c)
    np.testing.assert_allclose(dW.sum(axis=0), 0.0, atol=1e-12)
    # W = 0: dH = G W = 0 exactly.
    Wz = np.zeros_like(W)
    _, lz = logprob_fwd(H, Wz, y)
    dHz, _ = logprob_bwd(H, Wz, y, lz, c)
    assert np.all(dHz == 0.0)


def test_row_restricted_gradients_agree_with_full():
    # With dlogp nonzero only on rows S, dH[S] and dW[vrows] computed from the
    # rows S alone equal the full result.
    H, W, y = _rand(12, 6, 30, 8)
    S = np.array([1, 4, 5, 11])
    c = np.zeros(12)
    c[S] = np.random.default_rng(2).standard_normal(len(S))
    y = y.copy()
    y[4] = y[5]
    _, lse = logprob_fwd(H, W, y)
    dH, dW = logprob_bwd(H, W, y, lse, c)
    vrows = np.array([0, y[4], 7, 29])
    np.testing.assert_allclose(dhidden_rows(H[S], W, y[S], lse[S], c[S]), dH[S],
                               rtol=0, atol=1e-13)
    np.testing.assert_allclose(dweight_rows(H[S], W, y[S], lse[S], c[S], vrows),
                               dW[vrows], rtol=0, atol=1e-13)
