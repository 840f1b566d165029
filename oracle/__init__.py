"""fp64 CPU oracle for the fused RL log-prob path.

TEST INFRASTRUCTURE.  Only the tests, the package entry's smoke check and
the benchmark's CPU-baseline leg may import or call anything in here.  The
product path (the HIP library and its Python binding) never does, and this
package shares no code, header, table or helper with it.

It computes the plain definitions, in float64, in the order the paper states
them:

* ``logprob``: per-token log pi_theta(o_t | x, o_<t) over the full vocabulary
  (the quantity in the numerator of the importance ratio, Eq. 4) as
  ``z = H W^T``, a two-pass log-sum-exp and a gather; and its gradient, the
  chain rule through the log-softmax (the paper gives no text for it).
* ``objective``: log-ratios (Eq. 4), MirrorPop and signed sequence statistics
  and masks (Eq. 18-21), group-normalised advantages (Eq. 3 / Eq. 12) and the
  sequence-masked clipped surrogate (Eq. 17, with the KL weight beta = 0) and
  its gradient with respect to the per-token log-probs, with an optional KL
  regulariser (estimator k3, a reading: the paper names none);
* ``logprob.token_entropy``: the per-token entropy diagnostic;
* ``primeecho``: the first-turn-anchored trajectory reward (Eq. 9-11).

Readings of points the paper leaves open are listed in ``objective.py``.
Every function here is pinned by tests against values that do not come from
this code: the paper's cancellation example, closed forms, brute force at
50 digits, invariances and central finite differences.
"""
from .logprob import (dhidden_rows, dweight_rows, logprob_bwd, logprob_fwd,  # noqa: F401
                      token_entropy)
from .objective import RLParams, rl_loss  # noqa: F401
from .primeecho import trajectory_rewards  # noqa: F401
