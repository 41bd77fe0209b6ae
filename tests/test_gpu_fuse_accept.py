"""The fusion / log-softmax / accept stage on hand-built logits (GPU, through
the C ABI's rv_debug_fuse_accept, which runs rv_verify's own kernels).

* The hand-worked fixtures of Algorithm 2 (accept_cases.json) and Algorithm 3
  (typical_cases.json): n and t bit-exact.
* Eq. 2 in fp32 bit-exact against numpy's fp32 arithmetic; alpha = 0 and 1
  give o and r exactly.
* Exact ties resolve to the lowest id, inside a vocabulary chunk and across
  chunks.
* Rows holding -inf entries (ids ruled out): decisions, log-softmax and
  entropy (0 log 0 = 0) as the oracle computes them.
* k = 0, every draft accepted, the history append, and out-of-range drafts.
"""
import json
import os

import numpy as np
import pytest

import oracle
import workload

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
PAD = -1e30  # softmax weight exactly 0 in fp32; finite, so Eq. 2 stays finite at alpha = 0 and 1

# vocabulary 16 for the hand-worked fixtures (rows padded with PAD), 8192 (four
# chunks of the LM-head tail) for ties across chunks
SMALL = workload.ModelShape("head-v16", 1, 128, 4, 4, 32, 128, 16, "f32")
WIDE = workload.ModelShape("head-v8192", 1, 128, 4, 4, 32, 128, 8192, "f32")


def load(name):
    with open(os.path.join(HERE, "golden", name)) as f:
        return json.load(f)


@pytest.fixture(scope="module")
def small(rv, gpu):
    v = rv.Verifier(SMALL, 0, 1, 64, max_block=8, max_drafts=8)
    yield v
    v.close()


@pytest.fixture(scope="module")
def wide(rv, gpu):
    v = rv.Verifier(WIDE, 0, 3, 64, max_block=8, max_drafts=8)
    yield v
    v.close()


def run(rv, v, o, r, drafts, alpha, L, **kw):
    """o, r: [B][k+1][V]; drafts [B][k].  Returns (n, t, outputs)."""
    import torch
    o = np.asarray(o, np.float32)
    r = np.asarray(r, np.float32)
    B, k1, V = o.shape
    logits = torch.from_numpy(np.ascontiguousarray(np.concatenate([o, r], axis=1))).cuda()
    d = torch.from_numpy(np.asarray(drafts, np.int32).reshape(B, k1 - 1)).cuda() if k1 > 1 else None
    rv.rv_debug_fuse_accept(v.cache, logits, L, d, k1 - 1, alpha, v.accept_len, v.next_id, **kw)
    torch.cuda.synchronize()
    v.k, v.kb = k1 - 1, None
    out = {w: v.output(w).cpu().numpy() for w in range(9)}
    return v.accept_len.cpu().numpy().copy(), v.next_id.cpu().numpy().copy(), out


def pad(rows, V):
    rows = np.asarray(rows, dtype=np.float64)
    out = np.full(rows.shape[:-1] + (V,), PAD)
    out[..., :rows.shape[-1]] = rows
    return out


def history(rv, v, b, pos0, n):
    import torch
    ids = torch.empty(n, dtype=torch.int32, device="cuda")
    rv.rv_debug_export_ids(v.cache, b, pos0, n, ids)
    torch.cuda.synchronize()
    return ids.cpu().tolist()


@pytest.mark.parametrize("case", load("accept_cases.json")["cases"], ids=lambda c: c["name"])
def test_accept_golden(rv, small, case):
    V = SMALL.vocab
    o, r = pad(case["o"], V)[None], pad(case["r"], V)[None]
    n, t, out = run(rv, small, o, r, [case["drafts"]], case["alpha"], [5])
    assert (int(n[0]), int(t[0])) == (case["n"], case["t"])
    z = out[rv.RV_OUT_FUSED][0]
    np.testing.assert_array_equal(z, oracle.fuse(o[0], r[0], case["alpha"]))
    if "expected_z_row0" in case:
        np.testing.assert_allclose(z[0][:6], case["expected_z_row0"], atol=1e-6)
    if case["alpha"] == 0.0:
        np.testing.assert_array_equal(z, o[0].astype(np.float32))
    if case["alpha"] == 1.0:
        np.testing.assert_array_equal(z, r[0].astype(np.float32))
    # the decision is appended to the history: x_1..x_n, t
    assert history(rv, small, 0, 5, case["n"] + 1) == case["drafts"][:case["n"]] + [case["t"]]


@pytest.mark.parametrize("case", load("typical_cases.json")["cases"], ids=lambda c: c["name"])
def test_typical_golden(rv, small, case):
    V = SMALL.vocab
    o, r = pad(case["o"], V)[None], pad(case["r"], V)[None]
    src = rv.RV_ENTROPY_FUSED if case["entropy_of"] == "fused" else rv.RV_ENTROPY_ORIGINAL
    n, t, out = run(rv, small, o, r, [case["drafts"]], case["alpha"], [5], rule=rv.RV_RULE_TYPICAL,
                    epsilon=float(case["eps"]), delta=float(case["delta"]), entropy_src=src)
    assert (int(n[0]), int(t[0])) == (case["n"], case["t"])
    # margins: every accepted draft positive, a rejected one not
    mg = out[rv.RV_OUT_MARGINS][0]
    assert (mg[:case["n"]] > 0).all()
    if case["n"] < len(case["drafts"]):
        assert not mg[case["n"]] > 0


def test_ties_go_to_the_lowest_id_across_chunks(rv, wide):
    V = WIDE.vocab
    rng = np.random.default_rng(21)
    B, k = 3, 2
    o = rng.standard_normal((B, k + 1, V)).astype(np.float32)
    r = rng.standard_normal((B, k + 1, V)).astype(np.float32)
    # sequence 0, row 0: the maximum at ids 3000, 100 and 7000 (three chunks)
    o[0, 0, [3000, 100, 7000]] = 9.0
    # sequence 1, row 0: at the chunk boundary 2047 / 2048; row 1: inside one
    # chunk, held by different threads (5 and 261)
    o[1, 0, [2048, 2047]] = 9.0
    o[1, 1, [261, 5]] = 9.0
    # sequence 2: the draft is one of the tied ids but not the lowest
    o[2, 0, [4097, 4100]] = 9.0
    drafts = [[3000, 1], [2047, 5], [4100, 3]]
    n, t, out = run(rv, wide, o, r, drafts, 0.0, [7, 9, 11])
    assert (n.tolist(), t.tolist()) == ([0, 2, 0], [100, int(np.argmax(o[1, 2])), 4097])
    np.testing.assert_array_equal(out[rv.RV_OUT_FUSED], o)


@pytest.mark.parametrize("alpha", [0.0, 0.3, 1.0])
def test_random_rows_match_the_oracle(rv, wide, alpha):
    V = WIDE.vocab
    rng = np.random.default_rng(int(alpha * 10) + 3)
    B, k = 3, 4
    o = (rng.standard_normal((B, k + 1, V)) * 2).astype(np.float32)
    r = (rng.standard_normal((B, k + 1, V)) * 2).astype(np.float32)
    # sequence 1 drafts its own argmaxes: all accepted; sequence 2 the first two
    drafts = rng.integers(0, V, (B, k))
    z = np.stack([oracle.fuse(o[b], r[b], alpha) for b in range(B)])
    drafts[1] = np.argmax(z[1][:k], -1)
    drafts[2, :2] = np.argmax(z[2][:2], -1)
    n, t, out = run(rv, wide, o, r, drafts, alpha, [3, 4, 5])
    np.testing.assert_array_equal(out[rv.RV_OUT_FUSED], z)
    for b in range(B):
        n_ref, t_ref = oracle.accept_greedy(z[b].astype(np.float64), drafts[b])
        assert (int(n[b]), int(t[b])) == (n_ref, t_ref), b
        lp = oracle.log_softmax(z[b])
        assert np.abs(out[rv.RV_OUT_LOGP_FUSED][b] - lp).max() < 2e-5
        # the fused distribution itself: exp of the log-probabilities, rows sum to 1
        p = out[rv.RV_OUT_PROB_FUSED][b].astype(np.float64)
        np.testing.assert_allclose(p, np.exp(lp), rtol=5e-5, atol=1e-12)
        assert np.abs(p.sum(-1) - 1).max() < 1e-5
        assert np.abs(out[rv.RV_OUT_ENTROPY][0][b] - oracle.entropy(z[b])).max() < 2e-4
        assert np.abs(out[rv.RV_OUT_ENTROPY][1][b] - oracle.entropy(o[b])).max() < 2e-4
    assert int(n[1]) == k and int(n[2]) >= 2
    assert history(rv, wide, 1, 4, k + 1) == list(drafts[1]) + [int(t[1])]


def test_rows_with_minus_infinity(rv, wide):
    """Ids ruled out with -inf (in both o and r, so Eq. 2 keeps them at -inf
    for alpha in (0, 1)); one whole vocabulary chunk of row 0 is -inf."""
    V = WIDE.vocab
    rng = np.random.default_rng(5)
    B, k = 3, 2
    o = rng.standard_normal((B, k + 1, V)).astype(np.float32)
    r = rng.standard_normal((B, k + 1, V)).astype(np.float32)
    dead = rng.random((B, k + 1, V)) < 0.4
    dead[0, 0, 2048:4096] = True
    o[dead] = -np.inf
    r[dead] = -np.inf
    alpha = 0.3
    z = np.stack([oracle.fuse(o[b], r[b], alpha) for b in range(B)])
    drafts = np.stack([np.argmax(z[b][:k], -1) for b in range(B)])
    drafts[2, 0] = int(np.flatnonzero(dead[2, 0])[0])  # a draft the target rules out
    n, t, out = run(rv, wide, o, r, drafts, alpha, [3, 4, 5])
    for b in range(B):
        n_ref, t_ref = oracle.accept_greedy(z[b].astype(np.float64), drafts[b])
        assert (int(n[b]), int(t[b])) == (n_ref, t_ref), b
        lp = out[rv.RV_OUT_LOGP_FUSED][b]
        assert np.isneginf(lp[dead[b]]).all() and np.isfinite(lp[~dead[b]]).all()
        assert np.abs(np.exp(lp.astype(np.float64)).sum(-1) - 1).max() < 1e-5
        h = out[rv.RV_OUT_ENTROPY][0][b]
        assert np.isfinite(h).all()
        np.testing.assert_allclose(h, oracle.entropy(z[b]), atol=2e-4)
    assert (int(n[2]), int(t[2])) == (0, int(np.argmax(z[2][0])))


def test_no_drafts_and_out_of_range_drafts(rv, wide):
    V = WIDE.vocab
    rng = np.random.default_rng(8)
    o = rng.standard_normal((3, 1, V)).astype(np.float32)
    r = rng.standard_normal((3, 1, V)).astype(np.float32)
    n, t, _ = run(rv, wide, o, r, np.zeros((3, 0)), 0.5, [2, 2, 2])
    z = np.stack([oracle.fuse(o[b], r[b], 0.5) for b in range(3)])
    assert n.tolist() == [0, 0, 0] and t.tolist() == [int(np.argmax(z[b][0])) for b in range(3)]
    # an id outside the vocabulary voids the sequence: -1, -1, history untouched
    o = rng.standard_normal((3, 3, V)).astype(np.float32)
    before = history(rv, wide, 1, 20, 3)
    n, t, _ = run(rv, wide, o, o, [[1, 2], [V, 3], [4, -1]], 0.3, [10, 20, 30])
    assert n.tolist()[1:] == [-1, -1] and t.tolist()[1:] == [-1, -1] and int(n[0]) >= 0
    assert history(rv, wide, 1, 20, 3) == before


def test_argument_errors(rv, wide):
    import torch
    V = WIDE.vocab
    logits = torch.zeros((3, 4, V), dtype=torch.float32, device="cuda")
    d = torch.zeros((3, 1), dtype=torch.int32, device="cuda")

    def code(**kw):
        args = dict(logits=logits, prefix_len=[3, 3, 3], draft_ids=d, k=1, alpha=0.3, accept_len=wide.accept_len,
                    next_id=wide.next_id)
        args.update(kw)
        try:
            rv.rv_debug_fuse_accept(wide.cache, **args)
        except rv.RVError as e:
            return e.name
        return "RV_OK"

    assert code(alpha=-0.1) == "RV_E_ARG"
    assert code(k=9) == "RV_E_ARG"
    assert code(draft_ids=None) == "RV_E_ARG"
    assert code(rule=rv.RV_RULE_SAMPLING) == "RV_E_ARG"
    assert code(prefix_len=[0, 3, 3]) == "RV_E_RANGE"
    assert code(prefix_len=[3, 63, 3]) == "RV_E_RANGE"
    assert code() == "RV_OK"
    torch.cuda.synchronize()
