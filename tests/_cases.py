"""Shared builders for the GPU parity tests: seeded inputs from `workloads`,
expected values from `oracle`, device copies for the HIP path."""
from __future__ import annotations

import numpy as np

import oracle
from workloads import (CONFIGS, make_structure, make_tensors_numpy, make_tensors_torch,
                       sample_targets_numpy, sample_targets_torch)

# Parity bar (fp32 accumulate everywhere; bf16 only in operands)
LOGP_ATOL = 2e-3          # |dlogp| and |dlse|
LOSS_RTOL = 1e-3          # relative error of the loss
GRAD_RTOL = 1e-3          # ||dGPU - dORACLE||_F / ||dORACLE||_F for dH and dW
# The softmax part of the gradient goes through a 2-byte transient operand,
# fp16 on bf16 inputs (the transposed W and H convert to it exactly).  The
# recompute pair rounds each element once: relative error <= 2^-11.  The
# softmax cache rounds twice (the cached exp in (0, 1], then the rescaled
# operand): <= 2^-10.
PTERM_RTOL = 2.0 ** -10
PTERM_RTOL_F16 = 2.0 ** -11


def to_params(p: oracle.RLParams):
    from paper_2606_04847_amd import RLParams
    return RLParams(p.eps_low, p.eps_high, p.delta, p.adv_eps, p.std_ddof, p.filter, p.kl_beta,
                    p.token_mode, p.tis_cap, p.icepop_lo, p.icepop_hi)


def small_case(cfg, seed=None):
    s = make_structure(cfg, seed=seed)
    H, W, hb, wb = make_tensors_numpy(cfg, s.T, seed=seed)
    y = sample_targets_numpy(cfg, H, W, seed=seed)
    return dict(cfg=CONFIGS[cfg] if isinstance(cfg, int) else cfg, s=s, H=H, W=W, hb=hb,
                wb=wb, y=y)


def device_tensors(case, dev="cuda"):
    import torch
    if case["hb"] is not None:
        H = torch.from_numpy(case["hb"].view(np.int16)).view(torch.bfloat16).to(dev)
        W = torch.from_numpy(case["wb"].view(np.int16)).view(torch.bfloat16).to(dev)
    else:
        H = torch.from_numpy(case["H"]).to(dev)
        W = torch.from_numpy(case["W"]).to(dev)
    y = torch.from_numpy(np.ascontiguousarray(case["y"], dtype=np.int64)).to(dev)
    return H, W, y


def structure_tensors(s, dev="cuda"):
    import torch
    return dict(mask=torch.from_numpy(s.loss_mask).to(dev),
                cu=torch.from_numpy(s.cu_seqlens).to(dev),
                cg=torch.from_numpy(s.cu_groups).to(dev),
                rewards=torch.from_numpy(s.rewards).to(dev))


def oracle_step(case, params: oracle.RLParams):
    s = case["s"]
    logp, lse = oracle.logprob_fwd(case["H"], case["W"], case["y"])
    lr = (logp + s.rollout_delta.astype(np.float64)).astype(np.float32)
    out = oracle.rl_loss(logp, lr, s.loss_mask, s.cu_seqlens, s.cu_groups, s.rewards, params)
    dH, dW = oracle.logprob_bwd(case["H"], case["W"], case["y"], lse, out["dlogp"])
    return dict(logp=logp, lse=lse, lr=lr, dH=dH, dW=dW, **{k: v for k, v in out.items()
                                                            if k != "dlogp"},
                dlogp=out["dlogp"])


def gpu_step(case, params: oracle.RLParams, lr: np.ndarray, dev="cuda"):
    import torch
    import paper_2606_04847_amd as mc
    H, W, y = device_tensors(case, dev)
    st = structure_tensors(case["s"], dev)
    logp, lse = mc.logprob_fwd(H, W, y)
    out = mc.rl_loss(logp, torch.from_numpy(lr).to(dev), st["mask"], st["cu"], st["cg"],
                     st["rewards"], to_params(params))
    dH, dW = mc.logprob_bwd(H, W, y, lse, out["dlogp"])
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy() for k, v in out.items()}
    res.update(logp=logp.cpu().numpy(), lse=lse.cpu().numpy(), dH=dH.cpu().numpy(),
               dW=dW.cpu().numpy())
    return res


def rel_fro(a, ref):
    a = np.asarray(a, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return np.linalg.norm(a - ref) / (den if den > 0 else 1.0)


def assert_step_parity(g, o, grad_rtol=GRAD_RTOL, logp_atol=LOGP_ATOL):
    assert np.max(np.abs(g["logp"] - o["logp"])) <= logp_atol
    assert np.max(np.abs(g["lse"] - o["lse"])) <= logp_atol
    assert np.array_equal(g["seq_mask"], o["seq_mask"])
    assert np.array_equal(g["seq_len"], o["seq_len"])
    assert int(g["n_valid"][0]) == o["n_valid"]
    assert abs(g["loss"][0] - o["loss"]) <= LOSS_RTOL * max(abs(o["loss"]), 1e-30)
    assert rel_fro(g["dlogp"], o["dlogp"]) <= 1e-4
    assert rel_fro(g["dH"], o["dH"]) <= grad_rtol
    assert rel_fro(g["dW"], o["dW"]) <= grad_rtol
    assert g["error_flag"][0] == 0


def fullsize_inputs(cid, dev="cuda"):
    """Device tensors of workload `cid` at its full size (torch generator)."""
    s = make_structure(cid)
    cfg = CONFIGS[cid]
    H, W = make_tensors_torch(cfg, s.T, dev)
    y = sample_targets_torch(cfg, H, W)
    return s, H, W, y


def sample_rows(T, n, seed, extra=()):
    rng = np.random.default_rng(seed)
    rows = set(int(r) for r in rng.choice(T, size=min(n, T), replace=False))
    rows |= {0, T - 1, min(255, T - 1), min(256, T - 1)}
    rows |= {int(r) for r in extra if 0 <= r < T}
    return np.array(sorted(rows), dtype=np.int64)
