"""PrimeEcho trajectory reward (Sec. 4.4.3, Eq. 9-11), fp64.

For trajectory i with K_i turns, turn scores s_ik and success flags:

    R_i = alpha * s_i1 + (1 - alpha) * max_{k <= K_i} s_ik + b_early(i)        (Eq. 9)
    b_early(i) = beta1 * 1[success_i1] + beta2 * 1[not success_i1 and success_i2]   (Eq. 10)

The group-normalised advantage of Eq. 12 is Eq. 3 applied to R (see
objective.rl_loss); the paper applies it to first-turn tokens, which is the
loss mask.  Default alpha = 0.75 (Sec. 5.1); beta1 > beta2 >= 0 are
parameters the paper does not set.
"""
from __future__ import annotations

import numpy as np


def trajectory_rewards(scores, success, n_turns, alpha=0.75, beta1=0.0, beta2=0.0):
    """scores, success: [B, Kmax]; n_turns: [B] (1 <= K_i <= Kmax)."""
    scores = np.asarray(scores, dtype=np.float64)
    success = np.asarray(success).astype(bool)
    B = scores.shape[0]
    R = np.zeros(B, dtype=np.float64)
    for i in range(B):
        K = int(n_turns[i])
        first = scores[i, 0]
        best = max(scores[i, k] for k in range(K))
        b = 0.0
        if success[i, 0]:
            b = beta1
        elif K >= 2 and success[i, 1]:
            b = beta2
        R[i] = alpha * first + (1.0 - alpha) * best + b
    return R
