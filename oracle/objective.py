"""The RL objective on top of per-token log-probs, fp64.

Follows the paper's RL section in its order:

  Eq. 4   importance ratio rho_t = pi_theta / pi_rollout, formed in log space:
          ell_t = logp_t - logp_rollout_t, rho_t = exp(ell_t)
  Eq. 19  mirror deviation m_t = max(rho_t, 1/rho_t) = exp|ell_t|
  Eq. 20  MirrorPop statistic: log of the length-normalised geometric mean of
          m, i.e. S_i = (1/L_i) sum_t |ell_t|
  Eq. 21  M_i = 1[S_i <= delta]
  Eq. 18  the signed ("vanilla") statistic (1/L_i) sum_t ell_t, reported as a
          diagnostic and usable as the filter instead
  Eq. 3   (and Eq. 12 for trajectory rewards) A_i = (r_i - mean_g r) / (std_g r + eps)
  Eq. 17  loss = -(1/sum_i M_i L_i) sum_i sum_t min(rho A_i, clip(rho, 1-eps_low,
          1+eps_high) A_i) M_i          (KL weight beta = 0)

Readings where the paper is silent or leaves a choice (each a parameter or
a convention; the paper prints no number that pins them):

  R1  natural logarithm throughout.
  R2  L_i counts the tokens of sequence i whose loss_mask is set (the loss is
      taken on first-turn tokens only); the same mask drives Eq. 18, 20, 21
      and 17.
  R3  L_i = 0: M_i = 0 and both statistics are 0; the sequence contributes
      nothing.
  R4  delta is a parameter (default 0.1 nats); the comparison is inclusive.
  R5  eps_low and eps_high are separate parameters (default 0.2 each).
  R6  std in Eq. 3 is the population standard deviation (ddof 0, a
      parameter) over all sequences of the group, whatever their M_i;
      eps defaults to 1e-6.  A group whose rewards are all equal (this
      includes a group of one sequence and the all-failed group of Eq. 13)
      has A = 0 exactly, also when eps = 0.
  R7  several groups in one batch: one global token mean,
      N = sum over all sequences of M_i L_i (reduces to Eq. 17 for one group).
  R8  N = 0: loss 0 and zero gradient.
  R9  gradient at a clip kink: the unclipped branch is taken when
      rho A <= clip(rho) A (ties count as unclipped); the clipped branch has
      zero gradient.  No gradient flows through M_i, S_i or A_i.
  R10 the filter "none" keeps every sequence with L_i > 0 (plain Eq. 5).
  R11 the KL term beta * D_KL(pi_theta || pi_ref) of Eq. 5 / Eq. 17: the paper
      names neither beta nor the estimator.  Reading: the per-token
      estimator k3 = exp(r) - r - 1 with r = logp_ref - logp (non-negative,
      zero iff the policies agree on the token), averaged with the same
      token mean as the surrogate, (1/N) sum_i M_i sum_t mask_t k3_t.  Its
      gradient is d k3 / d logp = 1 - exp(r).  Parity of this estimator with
      the paper is unpinned (the paper prints none); its arithmetic is pinned
      by closed forms and finite differences.
  R12 token-level truncation of the importance ratio (TIS, named in Sec. 4.5.2
      as an alternative to sequence masking, defined there by no formula):
      the policy-gradient weight rho_t A_i of a retained token is truncated
      at a cap C, i.e. its term of Eq. 17 is multiplied by the stop-gradient
      factor w_t = min(1, C / rho_t) = exp(min(0, ln C - ell_t)), so its
      gradient with respect to ell_t is min(rho_t, C) A_i on the unclipped
      branch.  C is a parameter (default 2); parity of this definition with
      the paper is unpinned.
  R13 token-level hard filtering of the importance ratio (IcePop, named in
      Sec. 4.5.2, defined there by no formula): a retained token whose ratio
      lies outside [alpha, beta] (decided in log space, ln alpha <= ell_t <=
      ln beta kept) contributes neither to the surrogate sum nor to the
      gradient; it still counts in N, in L_i and in the statistics of Eq. 18-21.
      alpha, beta are parameters (defaults 0.5, 2); parity of this definition
      with the paper is unpinned.
      Either mode combines with any sequence filter; `token_frac` reports the
      share of the N tokens it truncated (TIS) or dropped (IcePop).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

FILTERS = ("none", "vanilla", "mirrorpop")
TOKEN_MODES = ("none", "tis", "icepop")


@dataclasses.dataclass
class RLParams:
    eps_low: float = 0.2
    eps_high: float = 0.2
    delta: float = 0.1
    adv_eps: float = 1e-6
    std_ddof: int = 0
    filter: str = "mirrorpop"
    kl_beta: float = 0.0
    token_mode: str = "none"      # R12 / R13
    tis_cap: float = 2.0          # C of R12
    icepop_lo: float = 0.5        # alpha of R13
    icepop_hi: float = 2.0        # beta of R13


def _advantages(rewards, cu_groups, p: RLParams) -> np.ndarray:
    """Eq. 3 / Eq. 12: group-normalised advantage of each sequence."""
    A = np.zeros(len(rewards), dtype=np.float64)
    for g in range(len(cu_groups) - 1):
        a, b = int(cu_groups[g]), int(cu_groups[g + 1])
        r = np.asarray(rewards[a:b], dtype=np.float64)
        n = b - a
        if n == 0:
            continue
        if np.all(r == r[0]):
            continue                                       # R6: equal rewards
        mean = r.sum() / n
        dof = n - p.std_ddof
        var = ((r - mean) ** 2).sum() / dof if dof > 0 else 0.0
        A[a:b] = (r - mean) / (math.sqrt(var) + p.adv_eps)
    return A


def rl_loss(logp, logp_rollout, loss_mask, cu_seqlens, cu_groups, rewards,
            params: RLParams | None = None, logp_ref=None) -> dict:
    p = params or RLParams()
    if p.filter not in FILTERS:
        raise ValueError(p.filter)
    if p.token_mode not in TOKEN_MODES:
        raise ValueError(p.token_mode)
    logp = np.asarray(logp, dtype=np.float64)
    logp_rollout = np.asarray(logp_rollout, dtype=np.float64)
    T = len(logp)
    mask = (np.ones(T, dtype=bool) if loss_mask is None
            else np.asarray(loss_mask).astype(bool))
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    B = len(cu) - 1

    # Eq. 4 in log space (masked tokens may hold anything in logp_rollout).
    ell = np.where(mask, logp - np.where(mask, logp_rollout, 0.0), 0.0)
    rho = np.exp(ell)

    seq_len = np.zeros(B, dtype=np.int64)
    stat_abs = np.zeros(B, dtype=np.float64)
    stat_signed = np.zeros(B, dtype=np.float64)
    keep = np.zeros(B, dtype=bool)
    for i in range(B):
        s, e = cu[i], cu[i + 1]
        valid = mask[s:e]
        L = int(valid.sum())
        seq_len[i] = L
        if L == 0:
            continue                                      # R3
        stat_abs[i] = np.abs(ell[s:e][valid]).sum() / L   # Eq. 20 (log space)
        stat_signed[i] = ell[s:e][valid].sum() / L        # Eq. 18 (log space)
        if p.filter == "mirrorpop":
            keep[i] = stat_abs[i] <= p.delta              # Eq. 21
        elif p.filter == "vanilla":
            keep[i] = abs(stat_signed[i]) <= p.delta
        else:
            keep[i] = True

    A = _advantages(rewards, cu_groups, p)
    N = int((seq_len * keep).sum())

    lo, hi = 1.0 - p.eps_low, 1.0 + p.eps_high
    # R12 / R13 bounds in log space (float parameters widened to fp64)
    log_cap = math.log(float(np.float32(p.tis_cap)))
    log_alo = math.log(float(np.float32(p.icepop_lo)))
    log_ahi = math.log(float(np.float32(p.icepop_hi)))
    dlogp = np.zeros(T, dtype=np.float64)
    total = 0.0
    kl_total = 0.0
    n_clipped = 0
    n_token = 0
    use_kl = logp_ref is not None and p.kl_beta != 0.0
    if use_kl:
        logp_ref = np.asarray(logp_ref, dtype=np.float64)
    for i in range(B):
        if not keep[i]:
            continue
        s, e = cu[i], cu[i + 1]
        for t in range(s, e):
            if not mask[t]:
                continue
            weight = 1.0
            dropped = False
            if p.token_mode == "tis" and ell[t] > log_cap:          # R12
                weight = math.exp(log_cap - ell[t])
                n_token += 1
            elif p.token_mode == "icepop" and not (log_alo <= ell[t] <= log_ahi):   # R13
                dropped = True
                n_token += 1
            if not dropped:
                unclipped = rho[t] * A[i]
                clipped = min(max(rho[t], lo), hi) * A[i]
                total += weight * min(unclipped, clipped)
                if unclipped <= clipped:                      # R9
                    dlogp[t] = weight * unclipped             # d(rho A)/d ell = rho A
                else:
                    n_clipped += 1
            if use_kl:                                    # R11
                r = logp_ref[t] - logp[t]
                kl_total += math.exp(r) - r - 1.0
                # loss carries +beta k3 against the -(...) surrogate: undo the
                # common -1/N below with a minus sign here
                dlogp[t] -= p.kl_beta * (1.0 - math.exp(r))
    if N > 0:
        loss = -total / N + (p.kl_beta * kl_total / N if use_kl else 0.0)
        dlogp *= -1.0 / N
        clip_frac = n_clipped / N
        token_frac = n_token / N
        kl = kl_total / N
    else:                                                 # R8
        loss, clip_frac, token_frac, kl = 0.0, 0.0, 0.0, 0.0
        dlogp[:] = 0.0
    return dict(loss=loss, dlogp=dlogp, seq_mask=keep.astype(np.uint8),
                seq_len=seq_len.astype(np.int32), n_valid=N, adv=A,
                stat_abs=stat_abs, stat_signed=stat_signed, clip_frac=clip_frac,
                token_frac=token_frac, kl=kl)
