"""Pins of the oracle's method steps (CPU only): block construction (Eq. 1,
Algorithm 1), fusion (Eq. 2), the exact-match rule (Algorithm 2), and the
single-pass claim checked by brute-force token-by-token decoding."""
import json
import os

import numpy as np
import pytest
import scipy.special
import scipy.stats

import oracle
import workload

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_block_layout_golden():
    g = load("block_layout.json")
    block, shift, orig, refl = oracle.reflective_block(g["history"], g["drafts"], g["probe"], g["prefix_pos"])
    assert block == g["expected_block"]
    assert len(block) - 1 == g["expected_reflective_tokens"]  # row 0 is the pending committed token
    assert shift == g["expected_shift"]
    # Algorithm 1's m is 1-indexed over [c, reflective_draft] outputs: o_m sits at block row m - 1
    assert shift == g["expected_m"] - 1
    assert orig == g["expected_orig_rows"] and refl == g["expected_refl_rows"]
    # the second copy is the same drafts, each predicted by the row before it
    k = len(g["drafts"])
    assert block[shift + 1: shift + 1 + k] == g["drafts"] == block[1: 1 + k]


def test_block_degenerate_cases():
    h = [5, 6, 7]
    # empty probe (Table 2's empty-prompt variant) and P = 0 (Algorithm 1 literally)
    block, shift, orig, refl = oracle.reflective_block(h, [1, 2], [], 0)
    assert block == [7, 1, 2, 1, 2] and shift == 2 and refl == [2, 3, 4]
    # k = 0: one greedy decode step, original and reflective rows coincide
    block, shift, orig, refl = oracle.reflective_block(h, [], [], 0)
    assert block == [7] and orig == [0] and refl == [0]
    with pytest.raises(ValueError):
        oracle.reflective_block(h, [1], [], 4)


@pytest.mark.parametrize("case", load("accept_cases.json")["cases"], ids=lambda c: c["name"])
def test_accept_rule_golden(case):
    o = np.array(case["o"], dtype=np.float64)
    r = np.array(case["r"], dtype=np.float64)
    z = oracle.fuse(o, r, case["alpha"])
    if "expected_z_row0" in case:
        np.testing.assert_allclose(z[0], case["expected_z_row0"], atol=1e-6)
    n, t = oracle.accept_greedy(z, case["drafts"])
    assert (n, t) == (case["n"], case["t"])


def test_fusion_end_points_and_shift_invariance():
    rng = np.random.default_rng(0)
    o = (rng.standard_normal((5, 300)) * 3).astype(np.float32).astype(np.float64)
    r = (rng.standard_normal((5, 300)) * 3).astype(np.float32).astype(np.float64)
    np.testing.assert_array_equal(oracle.fuse(o, r, 0.0), o.astype(np.float32))
    np.testing.assert_array_equal(oracle.fuse(o, r, 1.0), r.astype(np.float32))
    # fusing logits equals fusing log-probabilities (softmax shift invariance):
    # p ~ p_o^(1-a) * p_r^a
    a = 0.3
    lp = oracle.log_softmax(oracle.fuse(o, r, a))
    lp2 = scipy.special.log_softmax((1 - a) * scipy.special.log_softmax(o, axis=-1)
                                    + a * scipy.special.log_softmax(r, axis=-1), axis=-1)
    np.testing.assert_allclose(lp, lp2, atol=1e-5)
    np.testing.assert_allclose(np.exp(lp).sum(-1), 1.0, atol=1e-12)
    np.testing.assert_allclose(oracle.log_softmax(o), scipy.special.log_softmax(o, axis=-1), atol=1e-12)


def test_margins_flag_near_ties():
    z = np.array([[0.0, 1.0, 1.0005, 0.0], [2.0, 0.0, 0.0, 0.0]], dtype=np.float32)
    n, t = oracle.accept_greedy(z, [2])
    ms, gap, near = oracle.decision_margins(z, [2], n)
    assert n == 1 and t == 0 and near and abs(ms[0] - 0.0005) < 1e-6
    z2 = np.array([[0.0, 1.0, 1.5, 0.0], [2.0, 0.0, 0.0, 0.0]], dtype=np.float32)
    assert not oracle.decision_margins(z2, [2], 1)[2]


# ------------------------------------------------------------ on a tiny model

SHAPE = workload.TINY
SEED = 0


@pytest.fixture(scope="module")
def history():
    return list(workload.random_ids(SHAPE.vocab, 40, 99, 0))


def test_bruteforce_rows_equal_single_pass(history):
    """Each o_i and r_i equals decoding the corresponding prefix from scratch."""
    drafts = list(workload.random_ids(SHAPE.vocab, 3, 99, 1))
    probe = list(workload.random_ids(SHAPE.vocab, 4, 99, 2))
    P = 4
    res = oracle.verify(SHAPE, SEED, history, drafts, probe, 0.3, P)
    k = len(drafts)
    for i in range(k + 1):
        seq_o = history + drafts[:i]
        lo = oracle.forward(SHAPE, SEED, seq_o, [len(seq_o) - 1])[0]
        np.testing.assert_allclose(res["o"][i], lo, rtol=0, atol=1e-9)
        seq_r = history + drafts + probe + history[-P:] + drafts[:i]
        lr = oracle.forward(SHAPE, SEED, seq_r, [len(seq_r) - 1])[0]
        np.testing.assert_allclose(res["r"][i], lr, rtol=0, atol=1e-9)


def test_probe_does_not_change_original_rows(history):
    drafts = list(workload.random_ids(SHAPE.vocab, 4, 98, 1))
    a = oracle.verify(SHAPE, SEED, history, drafts, list(workload.random_ids(SHAPE.vocab, 5, 98, 2)), 0.3, 4)
    b = oracle.verify(SHAPE, SEED, history, drafts, list(workload.random_ids(SHAPE.vocab, 5, 98, 3)), 0.3, 4)
    np.testing.assert_allclose(a["o"], b["o"], atol=1e-9)
    assert np.abs(a["r"] - b["r"]).max() > 1e-3


def test_greedy_drafts_fully_accepted_at_alpha_zero(history):
    g = oracle.greedy_continuation(SHAPE, SEED, history, 5)
    res = oracle.verify(SHAPE, SEED, history, g[:4], [], 0.0, 0)
    assert res["accept_len"] == 4 and res["next_id"] == g[4]
    # k = 0 is a single greedy decode step
    res0 = oracle.verify(SHAPE, SEED, history, [], [], 0.0, 0)
    assert res0["accept_len"] == 0 and res0["next_id"] == g[0]


def test_alpha_zero_is_standard_verification(history):
    drafts = list(workload.corrupt(oracle.greedy_continuation(SHAPE, SEED, history, 4), 0.5, SHAPE.vocab,
                                   np.random.default_rng(3)))
    res = oracle.verify(SHAPE, SEED, history, drafts, list(workload.random_ids(SHAPE.vocab, 8, 3, 3)), 0.0, 4)
    np.testing.assert_array_equal(res["z"], res["o"].astype(np.float32))
    n, t = oracle.accept_greedy(res["o"], drafts)
    assert (res["accept_len"], res["next_id"]) == (n, t)
    np.testing.assert_allclose(np.exp(res["lp_z"]).sum(-1), 1.0, atol=1e-9)


# ------------------------------------------------------------ Algorithm 3

@pytest.mark.parametrize("case", load("typical_cases.json")["cases"], ids=lambda c: c["name"])
def test_typical_rule_golden(case):
    o = np.array(case["o"], dtype=np.float64)
    r = np.array(case["r"], dtype=np.float64)
    z = oracle.fuse(o, r, case["alpha"]).astype(np.float64)
    n, t, margins = oracle.accept_typical(z, o, case["drafts"], float(case["eps"]), float(case["delta"]),
                                          case["entropy_of"])
    assert (n, t) == (case["n"], case["t"])
    # every tested draft but a rejected last one has a positive margin
    assert all(m > 0 for m in margins[:n]) and (n == len(case["drafts"]) or margins[n] <= 0)


def test_entropy_closed_forms():
    # uniform over V: ln V; a two-point distribution: the binary entropy;
    # a dominant logit: ~0; arbitrary rows: scipy's entropy of softmax
    for V in (2, 7, 4096):
        assert abs(oracle.entropy(np.zeros((1, V)))[0] - np.log(V)) < 1e-12
    a = 0.3
    h2 = -(a * np.log(a) + (1 - a) * np.log(1 - a))
    assert abs(oracle.entropy(np.log(np.array([[a, 1 - a]])))[0] - h2) < 1e-12
    assert oracle.entropy(np.array([[200.0, 0, 0, 0]]))[0] < 1e-80
    rng = np.random.default_rng(3)
    x = rng.standard_normal((6, 50)) * 2
    ref = scipy.stats.entropy(scipy.special.softmax(x, axis=-1), axis=-1)
    np.testing.assert_allclose(oracle.entropy(x), ref, rtol=1e-12)
    # ids at -inf have probability 0 and add nothing (0 log 0 = 0): the
    # entropy is that of the row without them
    xm = x.copy()
    xm[:, ::3] = -np.inf
    ref = scipy.stats.entropy(scipy.special.softmax(x[:, [j for j in range(50) if j % 3]], axis=-1), axis=-1)
    np.testing.assert_allclose(oracle.entropy(xm), ref, rtol=1e-12)


def test_typical_monotone_and_end_points():
    rng = np.random.default_rng(11)
    for trial in range(20):
        k, V = 6, 40
        # fp32-representable logits, as the fusion produces fp32
        o = (rng.standard_normal((k + 1, V)) * 3).astype(np.float32).astype(np.float64)
        r = (rng.standard_normal((k + 1, V)) * 3).astype(np.float32).astype(np.float64)
        z = oracle.fuse(o, r, 0.3).astype(np.float64)
        drafts = [int(np.argsort(z[i])[-1 - rng.integers(0, 3)]) for i in range(k)]
        ns = [oracle.accept_typical(z, o, drafts, 0.5, d)[0] for d in (0.0, 0.05, 0.2, 0.5, 1.0, 5.0)]
        # a larger delta raises every threshold: the accepted prefix never grows
        assert ns == sorted(ns, reverse=True)
        assert ns[0] == k  # delta = 0: threshold 0
        n_all, t_all, _ = oracle.accept_typical(z, o, drafts, float("inf"), 0.0)
        assert n_all == k and t_all == int(np.argmax(z[k]))
        # alpha = 0: the fused rows are the original rows, so both entropy sources agree
        z0 = oracle.fuse(o, r, 0.0).astype(np.float64)
        for d in (0.1, 0.4):
            assert oracle.accept_typical(z0, o, drafts, 0.3, d, "fused") == \
                oracle.accept_typical(z0, o, drafts, 0.3, d, "original")


# ------------------------------------------------------------ Algorithm 1 (sampling)

def test_philox_matches_numpy_stream():
    """numpy's Philox bit generator is Philox4x64-10; it advances the counter
    before each block, so its first block is counter + 1."""
    for key, ctr in (((123, 456), (0, 0, 0, 0)), ((2**64 - 1, 7), (2**64 - 1, 5, 0, 9)), ((0, 0), (3, 1, 4, 1))):
        bg = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=np.array(ctr, dtype=np.uint64))
        raw = [int(x) for x in bg.random_raw(12)]
        c = list(ctr)
        mine = []
        for _ in range(3):
            # 256-bit little-endian increment
            for j in range(4):
                c[j] = (c[j] + 1) & (2**64 - 1)
                if c[j]:
                    break
            mine += oracle.philox4x64(c, key)
        assert mine == raw


def test_uniform24_range_and_moments():
    u = np.array([oracle.acceptance_uniform(5, s, i) for s in range(50) for i in range(200)])
    assert (u > 0).all() and (u < 1).all()
    assert np.array_equal(u.astype(np.float32).astype(np.float64), u)  # exact in fp32
    assert abs(u.mean() - 0.5) < 0.01 and abs(u.var() - 1 / 12) < 0.005
    g = oracle.gumbel_uniforms(9, 0, 4099)
    assert g.shape == (4099,) and (g > 0).all() and (g < 1).all() and len(np.unique(g)) > 4000


def test_sampling_p_equals_q_accepts_everything():
    rng = np.random.default_rng(4)
    for seed in range(20):
        z = (rng.standard_normal((4, 9)) * 2).astype(np.float32).astype(np.float64)
        q = np.exp(oracle.log_softmax(z))
        drafts = [int(rng.choice(9, p=q[i] / q[i].sum())) for i in range(3)]
        n, t, margins, gap, near = oracle.accept_sampling(z, q[:3], drafts, seed, 0)
        assert n == 3 and all(m >= 0 for m in margins)


def _first_token_counts(z, q, trials, sample_bonus_from_p=False):
    """Emitted first token over many (seed, drafts): x_1 if accepted, else t."""
    rng = np.random.default_rng(12)
    V = z.shape[-1]
    counts = np.zeros(V)
    for seed in range(trials):
        drafts = [int(rng.choice(V, p=q[i])) for i in range(q.shape[0])]
        if sample_bonus_from_p:
            # planted mistake: the rejected position re-draws from p, not from the residual
            n, _, _, _, _ = oracle.accept_sampling(z, q, drafts, seed, 1)
            tok = drafts[0] if n >= 1 else int(rng.choice(V, p=np.exp(oracle.log_softmax(z[0]))))
        else:
            n, t, _, _, _ = oracle.accept_sampling(z, q, drafts, seed, 1)
            tok = drafts[0] if n >= 1 else t
        counts[tok] += 1
    return counts


def test_sampling_first_token_follows_p():
    """Speculative sampling is exact: the first emitted token is distributed
    as p_1 whatever the draft distribution (chi-square test)."""
    rng = np.random.default_rng(21)
    V, k, trials = 6, 2, 6000
    z = (rng.standard_normal((k + 1, V)) * 1.5).astype(np.float32).astype(np.float64)
    ql = rng.standard_normal((k, V)) * 1.5
    q = np.exp(ql - scipy.special.logsumexp(ql, axis=-1, keepdims=True))
    p1 = np.exp(oracle.log_softmax(z[0]))
    counts = _first_token_counts(z, q, trials)
    assert scipy.stats.chisquare(counts, p1 * trials).pvalue > 1e-3
    # the test has the power to see a wrong residual draw
    bad = _first_token_counts(z, q, trials, sample_bonus_from_p=True)
    assert scipy.stats.chisquare(bad, p1 * trials).pvalue < 1e-6


def test_sampling_bonus_draw_follows_p_when_all_accepted():
    """With no drafts the bonus token is a Gumbel-max draw from p_1."""
    rng = np.random.default_rng(8)
    V, trials = 5, 8000
    z = (rng.standard_normal((1, V)) * 1.2).astype(np.float32).astype(np.float64)
    counts = np.zeros(V)
    for seed in range(trials):
        _, t, _, _, _ = oracle.accept_sampling(z, np.zeros((0, V)), [], seed, 3)
        counts[t] += 1
    p = np.exp(oracle.log_softmax(z[0]))
    assert scipy.stats.chisquare(counts, p * trials).pvalue > 1e-3
