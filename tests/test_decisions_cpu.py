"""The near-tie allowance used by the GPU parity tests, on hand-made rows (CPU)."""
import numpy as np

import oracle
from decisions import greedy_allowed, typical_allowed


def rows(*vals):
    return np.array(vals, dtype=np.float64)


def test_greedy_clear_decision_is_the_only_one_allowed():
    # drafts 1, 2; row 0 argmax 1 (accept), row 1 argmax 0 (reject draft 2), t = 0
    z = rows([0.0, 3.0, 1.0], [2.0, 0.0, 1.0], [0.0, 0.0, 5.0])
    assert greedy_allowed(z, [1, 2], 1, 0)
    assert not greedy_allowed(z, [1, 2], 2, 2)   # draft 2 is 1.0 below the maximum
    assert not greedy_allowed(z, [1, 2], 0, 1)   # draft 1 is the clear maximum
    assert not greedy_allowed(z, [1, 2], 1, 2)   # t is not the row maximum
    assert not greedy_allowed(z, [1, 2], 3, 0)   # n beyond k


def test_greedy_near_tie_allows_both_sides():
    # row 0: draft 1 ties id 0 within 5e-4; either accepting it or rejecting
    # it (with t = 0) is allowed, rejecting with t = 1 is not
    z = rows([3.0, 2.9995, 1.0], [0.0, 0.0, 4.0])
    assert greedy_allowed(z, [1], 1, 2)
    assert greedy_allowed(z, [1], 0, 0)
    assert not greedy_allowed(z, [1], 0, 1)
    # the same rows with the gap widened past the band: only the rejection
    z2 = rows([3.0, 2.99, 1.0], [0.0, 0.0, 4.0])
    assert greedy_allowed(z2, [1], 0, 0) and not greedy_allowed(z2, [1], 1, 2)


def test_typical_allowance_follows_the_log_domain_margins():
    z = rows([2.0, 1.0, 0.0, -1.0], [0.5, 0.4, 0.3, 0.2], [1.0, 0.0, 0.0, 0.0])
    drafts = [0, 2]
    eps, delta = 0.3, 0.9
    lp = oracle.log_softmax(z)
    H = oracle.entropy(z)
    m = [lp[i][drafts[i]] - min(np.log(eps), np.log(delta) - H[i]) for i in range(2)]
    n = next((i for i, mi in enumerate(m) if not mi > 0), 2)
    t = int(np.argmax(z[n]))
    assert typical_allowed(z, z, drafts, n, t, eps, delta)
    others = [(nn, int(np.argmax(z[nn]))) for nn in range(3) if nn != n]
    # away from the band no other n is allowed
    assert all(abs(mi) > 1e-3 for mi in m)
    assert not any(typical_allowed(z, z, drafts, nn, tt, eps, delta) for nn, tt in others)
    # eps chosen so that draft 0's margin is 1e-4: accepting or rejecting it is allowed
    eps0 = float(np.exp(lp[0][0] - 1e-4))
    delta0 = 1e9  # threshold min(log eps, log delta - H) = log eps
    n1, t1, m1 = oracle.accept_typical(z, z, drafts, eps0, delta0)
    assert n1 >= 1 and abs(m1[0] - 1e-4) < 1e-9
    assert typical_allowed(z, z, drafts, n1, t1, eps0, delta0)
    assert typical_allowed(z, z, drafts, 0, int(np.argmax(z[0])), eps0, delta0)
