"""Which decisions a flagged near-tie allows (tests only).

The oracle flags a decision when one of its margins lies within TIE of the
boundary (fused-logit units for Algorithm 2, log-probability units for
Algorithm 3).  There the GPU, whose logits differ from the oracle's by
rounding order, may take either side; these checks accept exactly the
decisions that rows within TIE of the oracle's would give:

* every accepted draft passes its test to within TIE;
* a rejected draft (n < k) fails it to within TIE;
* the next token is within TIE of its row's maximum (and, under the greedy
  rule after a rejection, is not the rejected draft).
"""
import numpy as np

import oracle

TIE = 1e-3


def greedy_allowed(z, drafts, n, t, tie=TIE):
    """Algorithm 2 at temperature 0 on the oracle's fused rows z [k+1][V]."""
    z = np.asarray(z, dtype=np.float64)
    k = len(drafts)
    if not 0 <= n <= k or not 0 <= t < z.shape[-1]:
        return False
    for i in range(n):
        if z[i][int(drafts[i])] < z[i].max() - tie:
            return False
    if n < k:
        x = int(drafts[n])
        if np.delete(z[n], x).max() < z[n][x] - tie or t == x:
            return False
    return z[n][t] >= z[n].max() - tie


def typical_allowed(z, o, drafts, n, t, eps, delta, entropy_of="fused", tie=TIE):
    """Algorithm 3 (log p_i(x_i) against min(log eps, log delta - H_i)) on
    the oracle's fused rows z and original rows o."""
    z = np.asarray(z, dtype=np.float64)
    k = len(drafts)
    if not 0 <= n <= k or not 0 <= t < z.shape[-1]:
        return False
    lpz = oracle.log_softmax(z)
    H = oracle.entropy(z if entropy_of == "fused" else np.asarray(o, dtype=np.float64))
    with np.errstate(divide="ignore"):
        log_eps, log_delta = np.log(np.float64(eps)), np.log(np.float64(delta))
    margin = [float(lpz[i][int(drafts[i])] - min(log_eps, log_delta - H[i])) for i in range(k)]
    if any(m <= -tie for m in margin[:n]):
        return False
    if n < k and margin[n] > tie:
        return False
    return z[n][t] >= z[n].max() - tie
