"""Per-token log-probability over the full vocabulary and its gradient, fp64.

Definition (the numerator of the importance ratio, Eq. 4, evaluated by the
trainer for the token the rollout sampled):

    z_tv    = sum_k H[t,k] W[v,k]                       (logits, never rounded)
    lse_t   = log sum_v exp(z_tv)                       (two passes: max, then sum)
    logp_t  = z_{t,y_t} - lse_t

Targets outside [0, V) mark ignored tokens: their log-prob is the constant 0
and they receive no gradient.

Gradient, for an upstream dlogp_t = d loss / d logp_t (chain rule through the
log-softmax; the paper gives no text for this part):

    p_tv    = exp(z_tv - lse_t)
    G_tv    = dlogp_t (1[v = y_t] - p_tv)               (zero row for ignored t)
    dH      = G W,        dW = G^T H

Inputs are the exact values the GPU consumes (bf16 or fp32), widened to fp64.
The matrix products are library matmuls in fp64; logits are formed in
column blocks of W only to bound memory.
"""
from __future__ import annotations

import numpy as np

_BLOCK_ELEMS = 1 << 25   # logits kept per block (32M doubles = 256 MB)


def _logits(H64: np.ndarray, W: np.ndarray) -> np.ndarray:
    T, V = H64.shape[0], W.shape[0]
    z = np.empty((T, V), dtype=np.float64)
    step = max(1, _BLOCK_ELEMS // max(1, T))
    for v0 in range(0, V, step):
        z[:, v0:v0 + step] = H64 @ np.asarray(W[v0:v0 + step], dtype=np.float64).T
    return z


def _valid(y: np.ndarray, V: int) -> np.ndarray:
    return (y >= 0) & (y < V)


def logprob_fwd(H, W, y):
    """Return (logp[T], lse[T]) in float64."""
    H64 = np.asarray(H, dtype=np.float64)
    y = np.asarray(y, dtype=np.int64)
    V = W.shape[0]
    z = _logits(H64, W)
    m = z.max(axis=1)                                   # pass 1: row max
    s = np.exp(z - m[:, None]).sum(axis=1)              # pass 2: sum of exp
    lse = m + np.log(s)
    ok = _valid(y, V)
    logp = np.zeros(len(y), dtype=np.float64)
    rows = np.nonzero(ok)[0]
    logp[rows] = z[rows, y[rows]] - lse[rows]
    return logp, lse


def token_entropy(H, W):
    """Entropy of the model's next-token distribution at each row,
    -sum_v p_tv log p_tv (the entropy diagnostic of the MirrorPop ablation,
    Sec. 5.4), from the same two-pass log-sum-exp."""
    H64 = np.asarray(H, dtype=np.float64)
    z = _logits(H64, W)
    m = z.max(axis=1)
    lse = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
    logq = z - lse[:, None]
    return -(np.exp(logq) * logq).sum(axis=1)


def _grad_logits(z, y, lse, dlogp, V, cols=None):
    """G restricted to the given vocabulary columns (all when None)."""
    T = z.shape[0]
    p = np.exp(z - lse[:, None])
    ok = _valid(y, V)
    onehot = np.zeros_like(z)
    if cols is None:
        r = np.nonzero(ok)[0]
        onehot[r, y[r]] = 1.0
    else:
        pos = {int(c): j for j, c in enumerate(cols)}
        for t in range(T):
            j = pos.get(int(y[t]))
            if ok[t] and j is not None:
                onehot[t, j] = 1.0
    G = dlogp[:, None] * (onehot - p)
    G[~ok] = 0.0
    return G


def logprob_bwd(H, W, y, lse, dlogp):
    """Return (dH[T,d], dW[V,d]) in float64 for the full problem."""
    H64 = np.asarray(H, dtype=np.float64)
    W64 = np.asarray(W, dtype=np.float64)
    y = np.asarray(y, dtype=np.int64)
    lse = np.asarray(lse, dtype=np.float64)
    dlogp = np.asarray(dlogp, dtype=np.float64)
    z = H64 @ W64.T
    G = _grad_logits(z, y, lse, dlogp, W.shape[0])
    return G @ W64, G.T @ H64


def dhidden_rows(H_rows, W, y_rows, lse_rows, dlogp_rows):
    """dH for the given token rows: G_rows W (needs the full vocabulary)."""
    H64 = np.asarray(H_rows, dtype=np.float64)
    y = np.asarray(y_rows, dtype=np.int64)
    z = _logits(H64, W)
    G = _grad_logits(z, y, np.asarray(lse_rows, np.float64),
                     np.asarray(dlogp_rows, np.float64), W.shape[0])
    out = np.zeros((H64.shape[0], W.shape[1]), dtype=np.float64)
    step = max(1, _BLOCK_ELEMS // max(1, H64.shape[0]))
    for v0 in range(0, W.shape[0], step):
        out += G[:, v0:v0 + step] @ np.asarray(W[v0:v0 + step], dtype=np.float64)
    return out


def dweight_rows(H_rows, W, y_rows, lse_rows, dlogp_rows, vrows):
    """dW[vrows] = sum_t G[t, vrows]^T h_t over the given token rows.

    Exact for the whole batch when every token with a nonzero dlogp is among
    the rows passed (all other rows of G are zero)."""
    H64 = np.asarray(H_rows, dtype=np.float64)
    y = np.asarray(y_rows, dtype=np.int64)
    vrows = np.asarray(vrows, dtype=np.int64)
    Wsel = np.asarray(W[vrows], dtype=np.float64)
    z = H64 @ Wsel.T
    G = _grad_logits(z, y, np.asarray(lse_rows, np.float64),
                     np.asarray(dlogp_rows, np.float64), W.shape[0], cols=vrows)
    return G.T @ H64
