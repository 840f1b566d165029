"""Seeded synthetic inputs in the shapes of the paper's RL training batches.

The paper's RL data is private, so these stand in for it.  They follow the
shapes the paper states for its RL stage (group size 8, at most 3 turns,
loss on first-turn tokens only, rollouts produced asynchronously and thus
slightly off-policy; Section 5.1 "Training Details") and the LM-head sizes
of a 9B/27B-class model.

Nothing here computes a log-probability, a ratio, a sequence statistic, an
advantage or a loss.  The generator returns, per token, the offset between
the rollout policy's log-prob and the trainer's (``rollout_delta``); a
caller forms ``logp_rollout = logp_trainer + rollout_delta`` itself.  The
only place it looks at that offset is to keep inputs away from the two
decision boundaries of the objective (the sequence-filter threshold and the
clip edges), so that the integer decisions have a unique answer.

Two tensor back-ends exist:
  * numpy (PCG64), bit-reproducible on any host, used for the small shapes
    that the oracle evaluates in full;
  * torch on the GPU (seeded ``torch.Generator``), used for the full-size
    shapes whose tensors run to gigabytes.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

# ---------------------------------------------------------------------------
# Workload table.  Sizes: T packed tokens, d hidden width, V vocabulary.
# ---------------------------------------------------------------------------
CONFIGS = {
    1: dict(name="tiny-fp32", n_groups=4, group_size=4, T=None, d=128, V=1024,
            dtype="f32", seed=0,
            lengths=dict(kind="uniform", lo=16, hi=64),
            mask="all", noise=0.02, drift=dict(kind="one_seq_const", value=0.5),
            rewards="bernoulli", fwd_only=False),
    2: dict(name="9b-fwd", n_groups=16, group_size=8, T=8192, d=4096, V=151936,
            dtype="bf16", seed=2,
            lengths=dict(kind="lognormal", median=64, sigma=0.5, lo=1, hi=None),
            mask="all", noise=0.02, drift=None, rewards="bernoulli", fwd_only=True),
    3: dict(name="27b-fwdbwd", n_groups=32, group_size=8, T=32768, d=5120, V=151936,
            dtype="bf16", seed=3,
            lengths=dict(kind="lognormal", median=128, sigma=0.5, lo=1, hi=4096),
            mask="multiturn", noise=0.02, drift=None, rewards="bernoulli",
            fwd_only=False),
    4: dict(name="filter-stress", n_groups=32, group_size=8, T=16384, d=4096,
            V=151936, dtype="bf16", seed=4,
            lengths=dict(kind="lognormal", median=64, sigma=1.0, lo=8, hi=2048,
                         force_extremes=True),
            mask="spans70", noise=0.05,
            drift=dict(kind="frac_normal", count=26, mean=0.3, std=0.1),
            rewards="quarter", fwd_only=False),
    5: dict(name="large-vocab", n_groups=64, group_size=16, T=65536, d=4096,
            V=248320, dtype="bf16", seed=5,
            lengths=dict(kind="lognormal", median=64, sigma=0.5, lo=1, hi=None),
            mask="all", noise=0.02, drift=None, rewards="bernoulli", fwd_only=False),
}

# Objective parameters the margins are taken against (clip eps 0.2 as in the
# workloads; filter threshold delta = 0.1 nats, see the oracle's readings).
DEFAULT_EPS_LOW = 0.2
DEFAULT_EPS_HIGH = 0.2
DEFAULT_DELTA = 0.1
SEQ_MARGIN = 1e-3
TOKEN_MARGIN = 5e-3

_STREAMS = ("H", "W", "lengths", "targets", "mask", "noise", "drift", "rewards")


def scaled_config(base: int = 4, *, T=None, n_groups=None, group_size=None, d=None,
                  V=None, dtype=None, seed=None, median=None, hi=None, **over):
    """A copy of workload ``base`` with some sizes replaced (for tests at
    sizes the oracle evaluates in seconds)."""
    cfg = {k: (dict(v) if isinstance(v, dict) else v) for k, v in CONFIGS[base].items()}
    for key, val in dict(T=T, n_groups=n_groups, group_size=group_size, d=d, V=V,
                         dtype=dtype, seed=seed).items():
        if val is not None:
            cfg[key] = val
    if median is not None:
        cfg["lengths"]["median"] = median
    if hi is not None:
        cfg["lengths"]["hi"] = hi
    cfg.update(over)
    cfg["name"] = cfg["name"] + "-scaled"
    return cfg


def _cfg(cfg):
    return CONFIGS[cfg] if isinstance(cfg, int) else cfg


def _rngs(seed: int):
    ss = np.random.SeedSequence(seed)
    return {name: np.random.Generator(np.random.PCG64(s))
            for name, s in zip(_STREAMS, ss.spawn(len(_STREAMS)))}


# ---------------------------------------------------------------------------
# bf16 helpers (round-to-nearest-even, as the hardware conversion does)
# ---------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32)
            << np.uint32(16)).view(np.float32)


# ---------------------------------------------------------------------------
# Packing structure: lengths, groups, masks, rewards, rollout offsets
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class Structure:
    cu_seqlens: np.ndarray     # int32 [B+1], cu_seqlens[B] == T
    cu_groups: np.ndarray      # int32 [NG+1], offsets in sequence units
    loss_mask: np.ndarray      # uint8 [T]
    rewards: np.ndarray        # float32 [B]
    rollout_delta: np.ndarray  # float32 [T]: logp_rollout - logp_trainer
    drifted: np.ndarray        # bool [B], sequences given a systematic drift

    @property
    def T(self):
        return int(self.cu_seqlens[-1])

    @property
    def B(self):
        return len(self.cu_seqlens) - 1

    @property
    def NG(self):
        return len(self.cu_groups) - 1


def _fit_lengths(raw: np.ndarray, total: int, lo: int, hi: int | None,
                 fixed: np.ndarray) -> np.ndarray:
    """Scale free lengths so the sum is ``total`` within [lo, hi]; fixed
    entries keep their value; integer rounding by largest remainder."""
    hi_v = float("inf") if hi is None else float(hi)
    x = raw.astype(np.float64).copy()
    free = ~fixed
    target_free = total - x[fixed].sum()
    for _ in range(200):
        s = x[free].sum()
        x[free] *= target_free / s
        x[free] = np.clip(x[free], lo, hi_v)
        if abs(x[free].sum() - target_free) < 1e-6:
            break
    base = np.floor(x).astype(np.int64)
    base[fixed] = x[fixed].astype(np.int64)
    rem = total - base.sum()
    frac = np.where(free, x - np.floor(x), -1.0)
    order = np.argsort(-frac, kind="stable")
    i = 0
    while rem != 0:
        j = order[i % len(order)]
        i += 1
        if not free[j]:
            continue
        if rem > 0 and base[j] + 1 <= hi_v:
            base[j] += 1
            rem -= 1
        elif rem < 0 and base[j] - 1 >= lo:
            base[j] -= 1
            rem += 1
        if i > 100 * len(order):
            raise RuntimeError("cannot fit lengths")
    return base


def _lengths(cfg, rng) -> np.ndarray:
    B = cfg["n_groups"] * cfg["group_size"]
    spec = cfg["lengths"]
    if spec["kind"] == "uniform":
        return rng.integers(spec["lo"], spec["hi"] + 1, size=B).astype(np.int64)
    raw = rng.lognormal(math.log(spec["median"]), spec["sigma"], size=B)
    lo, hi = spec.get("lo", 1), spec.get("hi")
    fixed = np.zeros(B, dtype=bool)
    if spec.get("force_extremes"):
        i_lo, i_hi = rng.choice(B, size=2, replace=False)
        raw[i_lo], raw[i_hi] = lo, hi
        fixed[[i_lo, i_hi]] = True
    T = cfg["T"]
    if T < B * lo or (hi is not None and T > B * hi):
        raise ValueError("T incompatible with length bounds")
    return _fit_lengths(raw, T, lo, hi, fixed)


def _split(total: int, parts: int, rng) -> list[int]:
    """Random composition of ``total`` into ``parts`` positive integers."""
    if parts <= 1:
        return [total]
    cuts = np.sort(rng.choice(np.arange(1, total), size=parts - 1, replace=False))
    edges = np.concatenate([[0], cuts, [total]])
    return list(np.diff(edges).astype(int))


def _masks(cfg, lengths, rng) -> np.ndarray:
    T = int(lengths.sum())
    kind = cfg["mask"]
    if kind == "all":
        return np.ones(T, dtype=np.uint8)
    out = np.zeros(T, dtype=np.uint8)
    starts = np.concatenate([[0], np.cumsum(lengths)[:-1]])
    if kind == "multiturn":
        # K ~ U{1,2,3} turns; the loss covers the first turn only.
        for s, L in zip(starts, lengths):
            K = rng.integers(1, 4)
            nv = L if K == 1 else max(1, int(round(rng.uniform(0.3, 0.7) * L)))
            out[s:s + nv] = 1
        return out
    if kind == "spans70":
        # exactly round(0.7 T) masked tokens, >= 1 valid token per sequence,
        # 1-4 alternating valid/masked spans starting with a valid span.
        n_valid_total = T - int(round(0.7 * T))
        want = 0.3 * lengths.astype(np.float64)
        v = np.maximum(1, np.floor(want)).astype(np.int64)
        v = np.minimum(v, lengths)
        rem = n_valid_total - v.sum()
        order = np.argsort(-(want - np.floor(want)), kind="stable")
        i = 0
        while rem != 0:
            j = order[i % len(order)]
            i += 1
            if rem > 0 and v[j] < lengths[j]:
                v[j] += 1
                rem -= 1
            elif rem < 0 and v[j] > 1:
                v[j] -= 1
                rem += 1
            if i > 100 * len(order):
                raise RuntimeError("cannot place masks")
        for s, L, nv in zip(starts, lengths, v):
            nm = L - nv
            if nm == 0:
                out[s:s + L] = 1
                continue
            n_spans = int(rng.integers(2, 5))
            n_vs = min((n_spans + 1) // 2, nv)
            n_ms = min(n_spans // 2, nm)
            n_vs = min(n_vs, n_ms + 1)
            n_ms = min(n_ms, n_vs)
            vparts = _split(int(nv), n_vs, rng)
            mparts = _split(int(nm), n_ms, rng)
            pos = s
            for k in range(n_vs):
                out[pos:pos + vparts[k]] = 1
                pos += vparts[k]
                if k < n_ms:
                    pos += mparts[k]
            assert pos == s + L
        return out
    raise ValueError(kind)


def _near_edges(ell, eps_low, eps_high):
    lo_edge, hi_edge = math.log(1.0 - eps_low), math.log(1.0 + eps_high)
    return (np.abs(ell - lo_edge) < TOKEN_MARGIN) | (np.abs(ell - hi_edge) < TOKEN_MARGIN)


def make_structure(cfg, seed=None, eps_low=DEFAULT_EPS_LOW,
                   eps_high=DEFAULT_EPS_HIGH, delta=DEFAULT_DELTA) -> Structure:
    cfg = _cfg(cfg)
    rng = _rngs(cfg["seed"] if seed is None else seed)
    lengths = _lengths(cfg, rng["lengths"])
    B = len(lengths)
    T = int(lengths.sum())
    cu = np.zeros(B + 1, dtype=np.int32)
    cu[1:] = np.cumsum(lengths)
    G = cfg["group_size"]
    cu_groups = (np.arange(cfg["n_groups"] + 1) * G).astype(np.int32)
    mask = _masks(cfg, lengths, rng["mask"])

    if cfg["rewards"] == "bernoulli":
        rewards = (rng["rewards"].random(B) < 0.5).astype(np.float32)
    elif cfg["rewards"] == "quarter":
        rewards = rng["rewards"].choice(np.array([0.0, 0.25, 0.5, 1.0], np.float32), B)
    else:
        raise ValueError(cfg["rewards"])

    # Per-sequence systematic drift of the rollout policy.
    drift_kind = (cfg["drift"] or {}).get("kind")
    drifted = np.zeros(B, dtype=bool)
    if drift_kind == "one_seq_const":
        drifted[rng["drift"].integers(B)] = True
    elif drift_kind == "frac_normal":
        drifted[rng["drift"].choice(B, size=cfg["drift"]["count"], replace=False)] = True

    sigma = cfg["noise"]
    nrng, drng = rng["noise"], rng["drift"]

    def draw(n, is_drifted):
        x = nrng.normal(0.0, sigma, size=n)
        if is_drifted and drift_kind == "one_seq_const":
            x = x + cfg["drift"]["value"]
        elif is_drifted and drift_kind == "frac_normal":
            x = x + drng.normal(cfg["drift"]["mean"], cfg["drift"]["std"], size=n)
        return x

    delta_t = np.zeros(T, dtype=np.float64)
    for i in range(B):
        s, e = cu[i], cu[i + 1]
        valid = mask[s:e].astype(bool)
        for attempt in range(1000):
            x = draw(e - s, drifted[i])
            # token margin: the trainer/rollout log-ratio is -x; keep valid
            # tokens away from the two clip edges.
            for _ in range(1000):
                bad = _near_edges(-x, eps_low, eps_high) & valid
                if not bad.any():
                    break
                x[bad] = draw(int(bad.sum()), drifted[i])
            else:
                raise RuntimeError("token margin not reachable")
            # sequence margin: mean |offset| and |mean offset| over the valid
            # tokens away from delta.
            if valid.any():
                xv = x[valid]
                a = np.abs(xv).sum() / valid.sum()
                b = abs(xv.sum() / valid.sum())
                if abs(a - delta) < SEQ_MARGIN or abs(b - delta) < SEQ_MARGIN:
                    continue
            break
        else:
            raise RuntimeError("sequence margin not reachable")
        delta_t[s:e] = x
    return Structure(cu, cu_groups, mask, rewards, delta_t.astype(np.float32), drifted)


# ---------------------------------------------------------------------------
# Dense tensors H [T,d], W [V,d] and targets y [T]
# ---------------------------------------------------------------------------
def make_tensors_numpy(cfg, T: int, seed=None):
    """H ~ N(0,1), W ~ w_std N(0,1) (w_std = 0.02 unless the workload says
    otherwise), drawn in fp32 and rounded to bf16 for bf16
    workloads.  Returns (H, W) as float32 arrays holding the exact values the
    GPU consumes, plus their bf16 bit patterns (None for fp32 workloads)."""
    cfg = _cfg(cfg)
    rng = _rngs(cfg["seed"] if seed is None else seed)
    d, V = cfg["d"], cfg["V"]
    H = rng["H"].standard_normal((T, d), dtype=np.float32)
    W = (np.float32(cfg.get("w_std", 0.02)) * rng["W"].standard_normal((V, d), dtype=np.float32))
    if cfg["dtype"] == "bf16":
        hb, wb = f32_to_bf16_bits(H), f32_to_bf16_bits(W)
        return bf16_bits_to_f32(hb), bf16_bits_to_f32(wb), hb, wb
    return H, W, None, None


def sample_targets_numpy(cfg, H: np.ndarray, W: np.ndarray, seed=None) -> np.ndarray:
    """Targets drawn from softmax(H W^T) row by row with the Gumbel-max trick:
    y_t = argmax_v (z_tv + g_tv), g ~ Gumbel(0,1).  This is the rollout
    policy's sampler, not the trainer's log-prob."""
    cfg = _cfg(cfg)
    rng = _rngs(cfg["seed"] if seed is None else seed)["targets"]
    T = H.shape[0]
    y = np.empty(T, dtype=np.int64)
    H64, W64 = H.astype(np.float64), W.astype(np.float64)
    step = max(1, (1 << 22) // max(1, W.shape[0]))
    for s in range(0, T, step):
        z = H64[s:s + step] @ W64.T
        u = rng.random(z.shape)
        u = np.clip(u, 1e-300, 1.0 - 1e-16)
        y[s:s + step] = np.argmax(z - np.log(-np.log(u)), axis=1)
    return y


def make_tensors_torch(cfg, T: int, device, seed=None):
    """Device-side H, W in the workload dtype (torch tensors)."""
    import torch
    cfg = _cfg(cfg)
    s = cfg["seed"] if seed is None else seed
    g = torch.Generator(device=device)
    g.manual_seed(1000003 * s + 11)
    d, V = cfg["d"], cfg["V"]
    dt = torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32
    H = torch.randn(T, d, generator=g, device=device, dtype=torch.float32).to(dt)
    W = torch.empty(V, d, device=device, dtype=dt)
    step = 16384
    for v0 in range(0, V, step):
        n = min(step, V - v0)
        W[v0:v0 + n] = (cfg.get("w_std", 0.02) * torch.randn(n, d, generator=g, device=device,
                                           dtype=torch.float32)).to(dt)
    return H, W


def sample_targets_torch(cfg, H, W, seed=None):
    """Gumbel-max sampling from softmax(H W^T) on the device, in fp32 chunks."""
    import torch
    cfg = _cfg(cfg)
    s = cfg["seed"] if seed is None else seed
    g = torch.Generator(device=H.device)
    g.manual_seed(1000003 * s + 29)
    T = H.shape[0]
    y = torch.empty(T, dtype=torch.int64, device=H.device)
    Wf = W.float()
    step = 1024
    for t0 in range(0, T, step):
        z = H[t0:t0 + step].float() @ Wf.T
        u = torch.rand(z.shape, generator=g, device=H.device).clamp_(1e-30, 1.0 - 1e-7)
        z -= torch.log(-torch.log(u))
        y[t0:t0 + step] = torch.argmax(z, dim=1)
        del z, u
    del Wf
    return y


def zipf_targets(T: int, V: int, exponent: float = 1.2, seed: int = 0) -> np.ndarray:
    """Skewed targets: token ranks drawn with probability proportional to
    rank^-exponent over the whole vocabulary, ranks mapped to vocabulary
    entries through a seeded permutation.  With exponent 1.2 the most
    frequent entry takes about a fifth of the tokens (3250 of T = 16384 at
    V = 151936, seed 4), the shape of real token streams (a few very frequent tokens:
    whitespace, indentation, punctuation) that the near-uniform model samples
    of the workloads lack.  Stands in for such streams when timing or checking
    the target-bucketed parts of the backward."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed)))
    ranks = np.arange(1, V + 1, dtype=np.float64)
    p = ranks ** -exponent
    p /= p.sum()
    r = rng.choice(V, size=T, p=p)
    perm = rng.permutation(V)
    return perm[r].astype(np.int64)
