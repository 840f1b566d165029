"""Full-size parity of the step the benchmark times, on workloads 2-5.

The chain is the one bench.py times: GPU forward -> mc_rl_loss on the GPU's
own log-probs -> backward on the GPU's own dlogp.  It runs through both
pairs: recompute (mc_logprob_fwd / mc_logprob_bwd) and softmax cache
(mc_logprob_fwd_cached / mc_logprob_bwd_cached).  The oracle side:

  * logp and lse of every row: oracle.logprob_fwd on row slices, one test
    per part of 8192 rows, so that no single test runs long;
  * the loss on the oracle's own log-probs with the same rollout log-probs
    (rollout = oracle logp + the workload's offset, rounded to fp32);
  * dH on >= 256 sampled rows (masked, filtered, clipped and live tokens,
    tile and chunk boundaries) and dW on >= 256 sampled vocabulary rows
    (the heaviest target buckets, untargeted rows, tile and chunk
    boundaries) from the real dlogp over all T tokens;
  * the softmax part of each gradient alone (its one-hot part subtracted on
    both sides), held to the fp16 rounding bound of the transient operand
    (one rounding in the recompute pair, two with the softmax cache).

Compared: logp and lse on every row (<= 2e-3); seq_mask, seq_len and N bit
for bit; the loss (relative 1e-3); dlogp (relative Frobenius 1e-4, same zero
pattern); sampled dH and dW rows (relative Frobenius 1e-3); softmax parts
(relative Frobenius 2^-11, 2^-10 with the cache); and, at any size,
sum_v dW[v, :] = 0.
"""
import gc

import numpy as np
import pytest

import oracle
from _cases import (GRAD_RTOL, LOGP_ATOL, LOSS_RTOL, PTERM_RTOL, PTERM_RTOL_F16,
                    fullsize_inputs, rel_fro,
                    structure_tensors, to_params)
from workloads import CONFIGS

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

PART_ROWS = 8192        # rows of one forward-comparison test
SUB_ROWS = 2048         # rows per oracle call (bounds its fp64 logits to 4 GB)
N_SAMPLE = 256
PAIRS = ("recompute", "cached")
ORDER = (2, 4, 3, 5)


def _parts(T):
    return [(a, min(a + PART_ROWS, T)) for a in range(0, T, PART_ROWS)]


def _steps():
    out = []
    for cid in ORDER:
        out += [("fwd", cid, k) for k in range(len(_parts(CONFIGS[cid]["T"])))]
        out.append(("chain", cid, -1))
    return out


STEPS = _steps()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_04847_amd as mc
    mc.load_library()
    yield
    _drop_all()


def _mc():
    import paper_2606_04847_amd as mc
    return mc


def _chunk_cols(T, V):
    """Vocabulary chunk width of the recompute backward (same rule as the
    library: 8 GiB of bf16 operand, multiples of 256 columns)."""
    cap = max(256, (8 << 30) // (max(1, T) * 2) // 256 * 256)
    if cap >= V:
        return V
    n = -(-V // cap)
    return min(cap, -(-(-(-V // n)) // 256) * 256)


class _State:
    """Inputs, GPU forwards, oracle rows and GPU chains of one workload."""

    def __init__(self, cid):
        mc = _mc()
        self.cid = cid
        self.cfg = CONFIGS[cid]
        self.s, self.H, self.W, self.y = fullsize_inputs(cid)
        self.T, self.V, self.d = self.s.T, self.W.shape[0], self.W.shape[1]
        torch.cuda.synchronize()
        self.Hh = self.H.float().cpu().numpy()
        # widened once: the oracle would otherwise widen every block of W on
        # every call (the exact bf16 values either way)
        self.Wh = self.W.float().cpu().numpy().astype(np.float64)
        self.yh = self.y.cpu().numpy()
        self.logp_o = np.full(self.T, np.nan)
        self.lse_o = np.full(self.T, np.nan)
        self.parts_done = set()
        # GPU forwards of both pairs (the cached one keeps its cache for the
        # backward, as in the benchmarked step)
        self.fwd = {}
        logp, lse = mc.logprob_fwd(self.H, self.W, self.y)
        self.fwd["recompute"] = dict(logp=logp, lse=lse, cache=None)
        cache = mc.softmax_cache(self.H, self.W)
        logp_c, lse_c = mc.logprob_fwd_cached(self.H, self.W, self.y, cache)
        self.fwd["cached"] = dict(logp=logp_c, lse=lse_c,
                                  cache=None if self.cfg["fwd_only"] else cache)
        del cache
        torch.cuda.synchronize()
        self.fwd_host = {k: (v["logp"].cpu().numpy(), v["lse"].cpu().numpy())
                         for k, v in self.fwd.items()}

    def oracle_part(self, k):
        if k in self.parts_done:
            return
        a, b = _parts(self.T)[k]
        for r in range(a, b, SUB_ROWS):
            e = min(r + SUB_ROWS, b)
            lo, so = oracle.logprob_fwd(self.Hh[r:e], self.Wh, self.yh[r:e])
            self.logp_o[r:e] = lo
            self.lse_o[r:e] = so
        self.parts_done.add(k)

    def oracle_all(self):
        for k in range(len(_parts(self.T))):
            self.oracle_part(k)
        assert not np.isnan(self.logp_o).any()


_STATES = {}


def _state(cid):
    if cid not in _STATES:
        _drop_all()
        _STATES[cid] = _State(cid)
    return _STATES[cid]


def _drop_all():
    _STATES.clear()
    gc.collect()
    if torch.cuda.is_available():
        torch.cuda.empty_cache()


def _sample_dh_rows(rng, s, o, T):
    """>= 256 token rows: live, masked, filtered and clipped tokens and
    tile / chunk boundaries."""
    mask = s.loss_mask.astype(bool)
    seq_of = np.repeat(np.arange(s.B), np.diff(s.cu_seqlens))
    kept = o["seq_mask"][seq_of].astype(bool)
    live = np.nonzero(o["dlogp"] != 0.0)[0]
    masked = np.nonzero(~mask)[0]
    filtered = np.nonzero(mask & ~kept)[0]
    clipped = np.nonzero(mask & kept & (o["dlogp"] == 0.0))[0]

    def pick(pool, n):
        return rng.choice(pool, size=min(n, len(pool)), replace=False) if len(pool) else []

    rows = set(int(r) for r in pick(live, 96))
    rows |= set(int(r) for r in pick(masked, 32))
    rows |= set(int(r) for r in pick(filtered, 32))
    rows |= set(int(r) for r in pick(clipped, 32))
    rows |= {0, T - 1, 255, 256, min(8191, T - 1), min(8192, T - 1), T // 2}
    while len(rows) < N_SAMPLE:
        rows.add(int(rng.integers(T)))
    return np.array(sorted(rows), np.int64), dict(live=len(live), masked=len(masked),
                                                  filtered=len(filtered), clipped=len(clipped))


def _sample_dw_rows(rng, y, dlogp, T, V):
    """>= 256 vocabulary rows: the heaviest live target buckets, other live
    targets, untargeted rows, tile and chunk boundaries."""
    live_targets = y[dlogp != 0.0]
    vals, counts = np.unique(live_targets, return_counts=True)
    heavy = vals[np.argsort(-counts, kind="stable")[:32]]
    rows = set(int(v) for v in heavy)
    others = np.setdiff1d(vals, heavy)
    rows |= set(int(v) for v in rng.choice(others, size=min(64, len(others)), replace=False))
    untargeted = np.setdiff1d(np.arange(V), np.unique(y))
    rows |= set(int(v) for v in rng.choice(untargeted, size=min(64, len(untargeted)),
                                           replace=False))
    chunk = _chunk_cols(T, V)
    for c in range(0, V, chunk):
        rows |= {c, max(c - 1, 0), min(c + 255, V - 1), min(c + 256, V - 1)}
    rows |= {0, V - 1, 127, 128}
    while len(rows) < N_SAMPLE:
        rows.add(int(rng.integers(V)))
    return np.array(sorted(rows), np.int64)


def _onehot_dw(rows_v, y, dlogp, H64):
    """sum over tokens t with y_t = v of dlogp_t h_t, for the given rows v."""
    pos = {int(v): j for j, v in enumerate(rows_v)}
    out = np.zeros((len(rows_v), H64.shape[1]))
    sel = np.nonzero(np.isin(y, rows_v) & (dlogp != 0.0))[0]
    for t in sel:
        out[pos[int(y[t])]] += dlogp[t] * H64[t]
    return out


def _forward_rows(st, k):
    st.oracle_part(k)
    a, b = _parts(st.T)[k]
    for pair, (logp, lse) in st.fwd_host.items():
        assert np.max(np.abs(logp[a:b] - st.logp_o[a:b])) <= LOGP_ATOL, pair
        assert np.max(np.abs(lse[a:b] - st.lse_o[a:b])) <= LOGP_ATOL, pair
    # the cached forward's log-probs are the plain forward's, bit for bit
    assert np.array_equal(st.fwd_host["recompute"][0], st.fwd_host["cached"][0])


def _chain(st):
    mc = _mc()
    st.oracle_all()
    for pair, (logp, lse) in st.fwd_host.items():
        assert np.max(np.abs(logp - st.logp_o)) <= LOGP_ATOL, pair
        assert np.max(np.abs(lse - st.lse_o)) <= LOGP_ATOL, pair
    if st.cfg["fwd_only"]:
        return
    s = st.s
    p = oracle.RLParams()                      # the benchmarked objective
    lr = (st.logp_o + s.rollout_delta.astype(np.float64)).astype(np.float32)
    o = oracle.rl_loss(st.logp_o, lr, s.loss_mask, s.cu_seqlens, s.cu_groups, s.rewards, p)
    rng = np.random.default_rng(1000 + st.cid)
    rows, kinds = _sample_dh_rows(rng, s, o, st.T)
    vrows = _sample_dw_rows(rng, st.yh, o["dlogp"], st.T, st.V)
    H64 = st.Hh.astype(np.float64)
    dH_o = oracle.dhidden_rows(st.Hh[rows], st.Wh, st.yh[rows], st.lse_o[rows],
                               o["dlogp"][rows])
    dW_o = oracle.dweight_rows(st.Hh, st.Wh, st.yh, st.lse_o, o["dlogp"], vrows)
    Wy = st.Wh[st.yh[rows]].astype(np.float64)
    soft_h_o = dH_o - o["dlogp"][rows, None] * Wy
    soft_w_o = dW_o - _onehot_dw(vrows, st.yh, o["dlogp"], H64)
    live_rows = o["dlogp"][rows] != 0.0
    assert live_rows.sum() >= 64 and kinds["live"] > 0
    st_t = structure_tensors(s)
    lrd = torch.from_numpy(lr).cuda()
    rows_d = torch.from_numpy(rows).cuda()
    vrows_d = torch.from_numpy(vrows).cuda()
    for pair in PAIRS:
        f = st.fwd[pair]
        out = mc.rl_loss(f["logp"], lrd, st_t["mask"], st_t["cu"], st_t["cg"],
                         st_t["rewards"], to_params(p))
        if pair == "recompute":
            dH, dW = mc.logprob_bwd(st.H, st.W, st.y, f["lse"], out["dlogp"])
        else:
            dH, dW = mc.logprob_bwd_cached(st.H, st.W, st.y, f["lse"], out["dlogp"],
                                           f["cache"])
            f["cache"] = None
        # sum_v dW[v, :] = sum_t dlogp_t (1 - sum_v p_tv) h_t = 0, against the
        # scale of the one-hot part sum_t dlogp_t h_t
        col = dW.double().sum(dim=0)
        ref = (out["dlogp"].double()[:, None] * st.H.double()).sum(dim=0)
        col_rel = (torch.linalg.norm(col) / torch.linalg.norm(ref)).item()
        g = {k: v.cpu().numpy() for k, v in out.items()}
        dH_g = dH[rows_d].double().cpu().numpy()
        dW_g = dW[vrows_d].double().cpu().numpy()
        del dH, dW, out
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        assert g["error_flag"][0] == 0, pair
        assert np.array_equal(g["seq_mask"], o["seq_mask"]), pair
        assert np.array_equal(g["seq_len"], o["seq_len"]), pair
        assert int(g["n_valid"][0]) == o["n_valid"], pair
        assert abs(g["loss"][0] - o["loss"]) <= LOSS_RTOL * abs(o["loss"]), pair
        assert rel_fro(g["dlogp"], o["dlogp"]) <= 1e-4, pair
        assert np.array_equal(g["dlogp"] == 0.0, o["dlogp"] == 0.0), pair
        assert rel_fro(dH_g, dH_o) <= GRAD_RTOL, pair
        assert np.all(dH_g[~live_rows] == 0.0), pair        # masked / filtered / clipped
        soft_h_g = dH_g - g["dlogp"].astype(np.float64)[rows, None] * Wy
        # operand bound: one fp16 rounding (recompute pair), two (softmax cache)
        pbound = PTERM_RTOL_F16 if pair == "recompute" else PTERM_RTOL
        assert rel_fro(soft_h_g[live_rows], soft_h_o[live_rows]) <= pbound, pair
        assert rel_fro(dW_g, dW_o) <= GRAD_RTOL, pair
        soft_w_g = dW_g - _onehot_dw(vrows, st.yh, g["dlogp"].astype(np.float64), H64)
        assert rel_fro(soft_w_g, soft_w_o) <= pbound, pair
        assert col_rel <= GRAD_RTOL, pair
        print(f"[fullsize {st.cid} {pair}] N={o['n_valid']} rows={kinds} "
              f"dH {rel_fro(dH_g, dH_o):.2e} soft {rel_fro(soft_h_g[live_rows], soft_h_o[live_rows]):.2e} "
              f"dW {rel_fro(dW_g, dW_o):.2e} soft {rel_fro(soft_w_g, soft_w_o):.2e} "
              f"sum_v dW {col_rel:.2e}", flush=True)


@pytest.mark.parametrize("step", STEPS, ids=[f"{k}-{c}" + (f"-{p}" if p >= 0 else "")
                                            for k, c, p in STEPS])
def test_fullsize(step):
    kind, cid, k = step
    st = _state(cid)
    if kind == "fwd":
        _forward_rows(st, k)
    else:
        try:
            _chain(st)
        finally:
            _drop_all()
