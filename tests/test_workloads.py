"""The synthetic workloads have the stated structure and keep their margins."""
import math

import numpy as np
import pytest

from oracle import RLParams, rl_loss
from workloads import (CONFIGS, bf16_bits_to_f32, f32_to_bf16_bits, make_structure,
                       make_tensors_numpy, sample_targets_numpy)


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_structure(cid):
    cfg = CONFIGS[cid]
    s = make_structure(cid)
    L = np.diff(s.cu_seqlens)
    assert s.B == cfg["n_groups"] * cfg["group_size"]
    assert s.NG == cfg["n_groups"]
    assert s.cu_seqlens[0] == 0 and np.all(L >= 1)
    assert np.all(np.diff(s.cu_groups) == cfg["group_size"]) and s.cu_groups[-1] == s.B
    if cfg["T"] is not None:
        assert s.T == cfg["T"]
    else:
        assert np.all((L >= 16) & (L <= 64))
    spec = cfg["lengths"]
    if spec.get("hi"):
        assert L.max() <= spec["hi"]
    if spec.get("force_extremes"):
        assert L.min() == spec["lo"] and L.max() == spec["hi"]
    assert len(s.loss_mask) == s.T and len(s.rollout_delta) == s.T
    if cfg["mask"] == "all":
        assert np.all(s.loss_mask == 1)
    valid_per_seq = np.add.reduceat(s.loss_mask.astype(np.int64), s.cu_seqlens[:-1])
    assert np.all(valid_per_seq >= 1)
    if cfg["mask"] == "spans70":
        assert int((s.loss_mask == 0).sum()) == int(round(0.7 * s.T))
        for i in range(s.B):
            m = s.loss_mask[s.cu_seqlens[i]:s.cu_seqlens[i + 1]]
            assert m[0] == 1
            runs = 1 + int(np.count_nonzero(np.diff(m)))
            assert runs <= 4
    if cfg["mask"] == "multiturn":
        for i in range(s.B):
            m = s.loss_mask[s.cu_seqlens[i]:s.cu_seqlens[i + 1]]
            k = int(m.sum())
            assert np.all(m[:k] == 1) and np.all(m[k:] == 0)   # first-turn prefix
    drift = cfg["drift"]
    if drift and drift["kind"] == "frac_normal":
        assert s.drifted.sum() == drift["count"]
    if drift and drift["kind"] == "one_seq_const":
        assert s.drifted.sum() == 1
    assert set(np.unique(s.rewards)) <= ({0.0, 1.0} if cfg["rewards"] == "bernoulli"
                                         else {0.0, 0.25, 0.5, 1.0})


@pytest.mark.parametrize("cid", [1, 3, 4, 5])
def test_margins_hold_under_the_oracle(cid):
    # With logp_rollout = logp + delta the log-ratio is -delta: the oracle's
    # statistics stay >= 1e-3 from the threshold and valid tokens of kept
    # sequences stay >= 5e-3 (log space) from the clip edges.
    s = make_structure(cid)
    logp = -np.linspace(1.0, 9.0, s.T)
    p = RLParams()
    out = rl_loss(logp, logp + s.rollout_delta.astype(np.float64), s.loss_mask,
                  s.cu_seqlens, s.cu_groups, s.rewards, p)
    has = out["seq_len"] > 0
    assert np.all(np.abs(out["stat_abs"][has] - p.delta) >= 1e-3 - 1e-9)
    assert np.all(np.abs(np.abs(out["stat_signed"][has]) - p.delta) >= 1e-3 - 1e-9)
    ell = -s.rollout_delta.astype(np.float64)[s.loss_mask > 0]
    for edge in (math.log(1 - p.eps_low), math.log(1 + p.eps_high)):
        assert np.all(np.abs(ell - edge) >= 5e-3 - 1e-6)
    if cid == 4:
        # drifted sequences are the ones MirrorPop removes
        assert np.all(out["seq_mask"][s.drifted] == 0)
        assert np.all(out["seq_mask"][~s.drifted] == 1)
    if cid == 1:
        assert out["seq_mask"][s.drifted].sum() == 0


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.00390625, 1.01171875, -2.5, 3.0e38, 1e-40], np.float32)
    b = f32_to_bf16_bits(x)
    back = bf16_bits_to_f32(b)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: rounds to the even mantissa (1.0)
    assert back[1] == 1.0
    # 1 + 3*2^-8 is a tie between 1+2^-7 and 1+2^-6: even is 1 + 2^-6
    assert back[2] == np.float32(1.015625)
    assert back[0] == 1.0 and back[3] == -2.5
    normal = np.abs(x) > 1e-37
    assert np.all(np.abs(back - x)[normal] <= np.abs(x)[normal] * 2.0 ** -8)
    # same bits as torch's fp32 -> bf16 conversion (a library routine)
    import torch
    r = np.random.default_rng(0).standard_normal(10000).astype(np.float32) * 37.0
    tb = torch.from_numpy(r).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(tb, f32_to_bf16_bits(r))


def test_tensors_and_targets_are_reproducible():
    H, W, hb, wb = make_tensors_numpy(1, 40)
    H2, W2, _, _ = make_tensors_numpy(1, 40)
    assert hb is None and np.array_equal(H, H2) and np.array_equal(W, W2)
    assert H.dtype == np.float32 and W.shape == (1024, 128)
    assert abs(W.std() - 0.02) < 1e-3
    y = sample_targets_numpy(1, H, W)
    assert np.array_equal(y, sample_targets_numpy(1, H, W))
    assert y.min() >= 0 and y.max() < 1024
