"""GPU path vs the CPU oracle on small configurations (through the C ABI).

Bars: accept_len / next_id identical unless the oracle flags a near-tie
(a decision margin within 1e-3 in fused-logit units), where they must be a
decision the oracle's rows allow within 1e-3 (tests/decisions.py); logits max-abs <= 1e-4
for fp32 models, per-row max|diff| / max|ref| <= 2e-2 for bf16 models;
log-softmax rows sum to 1.
"""
import numpy as np
import pytest

import oracle
import workload
from decisions import greedy_allowed, typical_allowed

pytestmark = pytest.mark.gpu

F32_ATOL = 1e-4
BF16_REL = 2e-2


def logits_close(shape, got, ref):
    got = np.asarray(got, dtype=np.float64)
    if shape.dtype == "f32":
        err = np.abs(got - ref).max()
        assert err <= F32_ATOL, f"max abs logit diff {err}"
    else:
        rel = (np.abs(got - ref).max(axis=-1) / np.abs(ref).max(axis=-1)).max()
        assert rel <= BF16_REL, f"max per-row relative logit diff {rel}"


class Case:
    """Prefill + one verify on the GPU; the oracle recomputes each sequence."""

    def __init__(self, rv, shape, seed, histories, drafts, probe, alpha, P, max_len=None, typical=None):
        """typical: None (Algorithm 2) or (epsilon, delta, entropy_of) for Algorithm 3."""
        import torch
        self.typical = typical
        self.shape, self.seed = shape, seed
        self.histories = [list(map(int, h)) for h in histories]
        self.drafts = np.asarray(drafts, dtype=np.int32).reshape(len(histories), -1)
        self.probe = np.asarray(probe, dtype=np.int32)
        self.alpha, self.P = alpha, P
        B = len(histories)
        k = self.drafts.shape[1]
        S = 1 + 2 * k + len(self.probe) + P
        max_len = max_len or (max(len(h) for h in histories) + S + 8)
        self.v = rv.Verifier(shape, seed, B, max_len, max_block=max(S, 8), max_drafts=max(k, 1))
        self.lens = self.v.prefill(self.histories)
        kw = {}
        if typical:
            eps, delta, src = typical
            kw = dict(rule=rv.RV_RULE_TYPICAL, epsilon=eps, delta=delta,
                      entropy_src=rv.RV_ENTROPY_FUSED if src == "fused" else rv.RV_ENTROPY_ORIGINAL)
        acc, nxt = self.v.verify(self.lens, self.drafts, self.probe, alpha, P, **kw)
        torch.cuda.synchronize()
        self.accept_len = acc.cpu().numpy().copy()
        self.next_id = nxt.cpu().numpy().copy()
        self.out = {w: self.v.output(w).cpu().numpy() for w in range(8)}

    def oracle(self, b):
        kw = {}
        if self.typical:
            eps, delta, src = self.typical
            kw = dict(rule="typical", eps=eps, delta=delta, entropy_of=src)
        return oracle.verify(self.shape, self.seed, self.histories[b], self.drafts[b], self.probe,
                             self.alpha, self.P, **kw)

    def check(self, rv):
        for b in range(len(self.histories)):
            ref = self.oracle(b)
            logits_close(self.shape, self.out[rv.RV_OUT_ORIG][b], ref["o"])
            logits_close(self.shape, self.out[rv.RV_OUT_REFL][b], ref["r"])
            logits_close(self.shape, self.out[rv.RV_OUT_FUSED][b], ref["z"])
            if len(self.probe) == 0 and self.P == 0:
                # block row k feeds both o_{k+1} and r_1 (shift = k): the LM head
                # reads one source row twice, so the two rows agree bit for bit
                k = self.drafts.shape[1]
                np.testing.assert_array_equal(self.out[rv.RV_OUT_ORIG][b][k], self.out[rv.RV_OUT_REFL][b][0])
            for w in (rv.RV_OUT_LOGP_ORIG, rv.RV_OUT_LOGP_REFL, rv.RV_OUT_LOGP_FUSED):
                s = np.exp(self.out[w][b].astype(np.float64)).sum(-1)
                assert np.abs(s - 1).max() < 1e-4
            lp_ref = ref["lp_z"]
            assert np.abs(self.out[rv.RV_OUT_LOGP_FUSED][b] - lp_ref).max() < (
                1e-4 if self.shape.dtype == "f32" else 0.05 * np.abs(lp_ref).max())
            # entropies of the fused and original rows
            h_tol = 5e-4 if self.shape.dtype == "f32" else 2e-2 * max(1.0, float(np.abs(ref["h_z"]).max()))
            assert np.abs(self.out[rv.RV_OUT_ENTROPY][0][b] - ref["h_z"]).max() < h_tol
            assert np.abs(self.out[rv.RV_OUT_ENTROPY][1][b] - ref["h_o"]).max() < h_tol
            n, t = int(self.accept_len[b]), int(self.next_id[b])
            if not ref["near_tie"]:
                assert (n, t) == (ref["accept_len"], ref["next_id"]), (b, ref["margins"], ref["gap"])
                mg = self.out[rv.RV_OUT_MARGINS][b]
                n_tested = len(ref["margins"])
                m_tol = 1e-3 if self.shape.dtype == "f32" else 5e-2
                np.testing.assert_allclose(mg[:n_tested], ref["margins"], atol=m_tol)
                assert np.isnan(mg[n_tested:-1]).all()
            elif self.typical:
                eps, delta, src = self.typical
                assert typical_allowed(ref["z"], ref["o"], self.drafts[b], n, t, eps, delta, src), (b, n, t)
            else:
                assert greedy_allowed(ref["z"], self.drafts[b], n, t), (b, n, t, ref["margins"], ref["gap"])
        return True


def tiny_histories(shape, B, L, key):
    return [workload.random_ids(shape.vocab, L + 3 * b, key, b) for b in range(B)]


@pytest.mark.parametrize("shape", [workload.TINY, workload.TINY_GQA_BF16], ids=lambda s: s.name)
def test_weights_bit_exact(rv, gpu, shape):
    import torch
    v = rv.Verifier(shape, 11, 1, 64)
    torch.cuda.synchronize()
    rng = np.random.default_rng(5)
    names = ["embed"] + [(l, n) for l in range(shape.n_layers) for n in oracle.TENSOR_NAMES] + ["lm_head"]
    for t, nm in enumerate(names):
        layer, name = (None, nm) if isinstance(nm, str) else nm
        rows, cols = oracle.tensor_dims(shape, name)
        idx = np.unique(np.concatenate([rng.integers(0, rows * cols, 300), [0, rows * cols - 1, cols, cols - 1]]))
        got = rv.rv_debug_weight_bits(v.model, t, idx)
        exp = oracle.weight_bits(shape, 11, layer, name, idx.astype(np.uint64))
        np.testing.assert_array_equal(got, exp, err_msg=f"tensor {t} {nm}")
    v.close()


def draft_case(shape, seed, hist, k, p, key):
    g = oracle.greedy_continuation(shape, seed, hist, k)
    return list(workload.corrupt(g, p, shape.vocab, np.random.default_rng(key)))


@pytest.mark.parametrize("alpha,P,n_probe,k", [(0.3, 4, 8, 4), (0.0, 4, 8, 4), (1.0, 4, 8, 4), (0.3, 0, 0, 4),
                                               (0.3, 4, 0, 1), (0.0, 0, 0, 0), (0.3, 2, 5, 6)])
def test_tiny_f32_matches_oracle(rv, gpu, alpha, P, n_probe, k):
    shape = workload.TINY
    hist = list(workload.random_ids(shape.vocab, 128, 0, 0, 2))
    drafts = draft_case(shape, 0, hist, k, 0.3, 17) if k else []
    probe = workload.random_ids(shape.vocab, n_probe, 0, 0xBEEF)
    c = Case(rv, shape, 0, [hist], [drafts], probe, alpha, P)
    c.check(rv)
    c.v.close()


def test_tiny_f32_batch_ragged(rv, gpu):
    shape = workload.TINY
    hists = [workload.random_ids(shape.vocab, L, 1, b) for b, L in enumerate([5, 77, 130, 64])]
    drafts = [draft_case(shape, 0, h, 4, 0.3, 30 + b) for b, h in enumerate(hists)]
    probe = workload.random_ids(shape.vocab, 8, 1, 0xBEEF)
    c = Case(rv, shape, 0, hists, drafts, probe, 0.3, 4)
    c.check(rv)
    c.v.close()


# (0.3, 4, 16, 8): 37 block rows x 4 query heads per kv head = 148 queries,
# the 192-query (12-wave) attention workgroup
@pytest.mark.parametrize("alpha,P,n_probe,k", [(0.3, 4, 8, 4), (1.0, 2, 3, 2), (0.0, 0, 0, 0), (0.3, 4, 16, 8)])
def test_tiny_bf16_gqa_matches_oracle(rv, gpu, alpha, P, n_probe, k):
    shape = workload.TINY_GQA_BF16
    hists = [workload.random_ids(shape.vocab, L, 2, b) for b, L in enumerate([40, 150, 300])]
    drafts = [draft_case(shape, 1, h, k, 0.3, 40 + b) if k else [] for b, h in enumerate(hists)]
    probe = workload.random_ids(shape.vocab, n_probe, 2, 0xBEEF)
    c = Case(rv, shape, 1, hists, drafts, probe, alpha, P)
    c.check(rv)
    c.v.close()


@pytest.mark.parametrize("shape", [workload.TINY, workload.TINY_GQA_BF16], ids=lambda s: s.name)
@pytest.mark.parametrize("max_len", [128, 150])
def test_block_fills_the_cache_exactly(rv, gpu, shape, max_len):
    """Largest allowed prefix: sequence 0's block ends at the cache's last
    position (max_len a multiple of the 64-key tile, and not), the block is
    the cache's largest and the batch its full size."""
    k, n_probe, P = 4, 6, 4
    S = 1 + 2 * k + n_probe + P
    lens = [max_len - S + 1, 57]
    hists = [workload.random_ids(shape.vocab, L, 12, b) for b, L in enumerate(lens)]
    drafts = [draft_case(shape, 3, h, k, 0.3, 120 + b) for b, h in enumerate(hists)]
    probe = workload.random_ids(shape.vocab, n_probe, 12, 0xBEEF)
    c = Case(rv, shape, 3, hists, drafts, probe, 0.3, P, max_len=max_len)
    c.check(rv)
    c.v.close()


@pytest.mark.parametrize("shape", [workload.TINY, workload.TINY_GQA_BF16], ids=lambda s: s.name)
@pytest.mark.parametrize("alpha,typical", [(0.3, (0.09, 0.3, "fused")), (1.0, (0.3, 0.1, "original")),
                                           (0.3, (float("inf"), 0.0, "fused")), (0.0, (0.05, 2.0, "fused"))])
def test_typical_rule_matches_oracle(rv, gpu, shape, alpha, typical):
    """Algorithm 3's entropy-thresholded rule against the oracle."""
    hists = [workload.random_ids(shape.vocab, L, 5, b) for b, L in enumerate([60, 97])]
    drafts = [draft_case(shape, 3, h, 5, 0.5, 50 + b) for b, h in enumerate(hists)]
    probe = workload.random_ids(shape.vocab, 6, 5, 0xBEEF)
    c = Case(rv, shape, 3, hists, drafts, probe, alpha, 4, typical=typical)
    c.check(rv)
    if typical[0] == float("inf") and typical[1] == 0.0:
        assert (c.accept_len == 5).all()
    c.v.close()


def sampling_case_q(shape, drafts, key, mass=0.4):
    """Draft distributions that put `mass` on the draft token and spread the
    rest by a random softmax (fp32, rows sum to 1)."""
    rng = np.random.default_rng(key)
    B, k = len(drafts), len(drafts[0])
    lg = rng.standard_normal((B, k, shape.vocab)) * 2
    q = np.exp(lg - lg.max(-1, keepdims=True))
    q *= (1 - mass) / q.sum(-1, keepdims=True)
    for b in range(B):
        for i in range(k):
            q[b, i, drafts[b][i]] += mass
    return q.astype(np.float32)


@pytest.mark.parametrize("shape", [workload.TINY, workload.TINY_GQA_BF16], ids=lambda s: s.name)
@pytest.mark.parametrize("alpha,temperature,seed", [(0.3, 1.0, 7), (0.3, 0.05, 11), (1.0, 0.1, 12345678901234)])
def test_sampling_rule_matches_oracle(rv, gpu, shape, alpha, temperature, seed):
    """Algorithm 1's speculative-sampling rule against the oracle: same
    Philox4x64-10 random numbers, same decisions unless near a tie."""
    import torch
    hists = [workload.random_ids(shape.vocab, L, 6, b) for b, L in enumerate([50, 81, 64])]
    drafts = [draft_case(shape, 4, h, 4, 0.3, 70 + b) for b, h in enumerate(hists)]
    probe = workload.random_ids(shape.vocab, 5, 6, 0xBEEF)
    q = sampling_case_q(shape, drafts, seed % 1000)
    k, P = 4, 3
    S = 1 + 2 * k + len(probe) + P
    v = rv.Verifier(shape, 4, len(hists), max(len(h) for h in hists) + S + 8, max_block=S, max_drafts=k)
    lens = v.prefill([list(map(int, h)) for h in hists])
    acc, nxt = v.verify_sampled(lens, np.array(drafts), q, probe, alpha, P, seed, temperature=temperature)
    torch.cuda.synchronize()
    acc, nxt = acc.cpu().numpy().copy(), nxt.cpu().numpy().copy()
    z = v.output(rv.RV_OUT_FUSED).cpu().numpy()
    mg = v.output(rv.RV_OUT_MARGINS).cpu().numpy()
    decided = 0
    for b in range(len(hists)):
        ref = oracle.verify(shape, 4, list(map(int, hists[b])), drafts[b], probe, alpha, P, rule="sampling",
                            temperature=temperature, q=q[b], rng_seed=seed, slot=b)
        logits_close(shape, z[b], ref["z"])
        if ref["near_tie"]:
            continue
        decided += 1
        assert (int(acc[b]), int(nxt[b])) == (ref["accept_len"], ref["next_id"]), (b, ref["margins"], ref["gap"])
        n_tested = len(ref["margins"])
        np.testing.assert_allclose(mg[b][:n_tested], ref["margins"], atol=1e-3 if shape.dtype == "f32" else 5e-2)
    assert decided >= 2
    # the same call again: the same outputs (the draw is a function of the seed)
    acc2, nxt2 = v.verify_sampled(lens, np.array(drafts), q, probe, alpha, P, seed, temperature=temperature)
    torch.cuda.synchronize()
    assert (acc2.cpu().numpy() == acc).all() and (nxt2.cpu().numpy() == nxt).all()
    v.close()


def test_kv_cache_matches_oracle(rv, gpu):
    """Prefill + verify write the KV the oracle computes at every position."""
    import torch
    shape = workload.TINY_GQA_BF16
    hist = list(workload.random_ids(shape.vocab, 90, 3, 0))
    drafts = list(workload.random_ids(shape.vocab, 3, 3, 1))
    probe = workload.random_ids(shape.vocab, 4, 3, 2)
    c = Case(rv, shape, 2, [hist], [drafts], probe, 0.3, 4)
    block, _, _, _ = oracle.reflective_block(hist, drafts, probe, 4)
    seq = hist[:-1] + block
    _, ks, vs = oracle.forward(shape, 2, seq, [0], return_kv=True)
    n = len(seq)
    for layer in range(shape.n_layers):
        # bf16 cache: hi plane then lo plane, value = hi + lo
        dk = torch.empty((2, shape.n_kv_heads, n, shape.head_dim), dtype=torch.bfloat16, device="cuda")
        dv = torch.empty_like(dk)
        rv.rv_debug_export_kv(c.v.cache, layer, 0, 0, n, dk, dv)
        torch.cuda.synchronize()
        gk = dk.double().sum(0).cpu().numpy().transpose(1, 0, 2)
        gv = dv.double().sum(0).cpu().numpy().transpose(1, 0, 2)
        for got, ref in ((gk, ks[layer]), (gv, vs[layer])):
            # fp32 vs fp64 accumulation, then the pair's 2^-17 relative rounding
            rel = np.abs(got - ref).max() / np.abs(ref).max()
            assert rel < 1e-4, (layer, rel)
    c.v.close()


def test_history_commit_and_idempotence(rv, gpu):
    import torch
    shape = workload.TINY
    hist = list(workload.random_ids(shape.vocab, 60, 4, 0))
    drafts = draft_case(shape, 0, hist, 4, 0.0, 4)  # uncorrupted greedy drafts
    probe = workload.random_ids(shape.vocab, 8, 4, 2)
    c = Case(rv, shape, 0, [hist], [drafts], probe, 0.0, 4)
    n, t = int(c.accept_len[0]), int(c.next_id[0])
    assert n == 4
    ids = torch.empty(len(hist) + n + 1, dtype=torch.int32, device="cuda")
    rv.rv_debug_export_ids(c.v.cache, 0, 0, len(hist) + n + 1, ids)
    torch.cuda.synchronize()
    assert ids.cpu().tolist() == hist + drafts[:n] + [t]
    # same call again: same outputs bit for bit
    z1 = c.out[rv.RV_OUT_FUSED].copy()
    acc, nxt = c.v.verify(c.lens, c.drafts, c.probe, 0.0, 4)
    torch.cuda.synchronize()
    assert (int(acc[0]), int(nxt[0])) == (n, t)
    np.testing.assert_array_equal(c.v.output(rv.RV_OUT_FUSED).cpu().numpy(), z1)
    # next step from the committed state continues the greedy sequence
    g = oracle.greedy_continuation(shape, 0, hist, 6)
    acc, nxt = c.v.verify([len(hist) + n + 1], np.array([[g[5]]]), [], 0.0, 0)
    torch.cuda.synchronize()
    assert int(acc[0]) == 1
    c.v.close()


def test_out_of_range_ids_reported(rv, gpu):
    import torch
    shape = workload.TINY
    v = rv.Verifier(shape, 0, 2, 64, max_block=16, max_drafts=4)
    lens = v.prefill([list(range(10)), list(range(20, 40))])
    acc, nxt = v.verify(lens, np.array([[1, 2], [3, shape.vocab + 5]]), [7], 0.3, 2)
    torch.cuda.synchronize()
    assert int(acc[1]) == -1 and int(nxt[1]) == -1
    assert int(acc[0]) >= 0
    v.close()


def test_validation_errors_enqueue_nothing(rv, gpu):
    import torch
    shape = workload.TINY
    v = rv.Verifier(shape, 0, 1, 40, max_block=16, max_drafts=4)
    lens = v.prefill([list(range(10))])
    d = torch.zeros((1, 2), dtype=torch.int32, device="cuda")
    probe = torch.zeros(3, dtype=torch.int32, device="cuda")
    v.accept_len.fill_(-11)
    v.next_id.fill_(-12)

    def history():
        ids = torch.empty(40, dtype=torch.int32, device="cuda")
        rv.rv_debug_export_ids(v.cache, 0, 0, 40, ids)
        torch.cuda.synchronize()
        return ids.cpu().tolist()

    hist0 = history()

    def code(**kw):
        args = dict(prefix_len=lens, draft_ids=d, k=2, probe_ids=probe, n_probe=3, alpha=0.3, prefix_pos=2,
                    accept_len=v.accept_len, next_id=v.next_id)
        args.update(kw)
        try:
            rv.rv_verify(v.cache, **args)
        except rv.RVError as e:
            return e.name
        return "RV_OK"

    assert code(alpha=1.5) == "RV_E_ARG"
    assert code(alpha=float("nan")) == "RV_E_ARG"
    assert code(k=-1) == "RV_E_ARG"
    assert code(k=5) == "RV_E_ARG"
    assert code(prefix_pos=-1) == "RV_E_ARG"
    assert code(rule=3) == "RV_E_ARG"
    typ = dict(rule=rv.RV_RULE_TYPICAL)
    assert code(epsilon=0.0, **typ) == "RV_E_ARG"
    assert code(epsilon=float("nan"), **typ) == "RV_E_ARG"
    assert code(delta=-0.1, **typ) == "RV_E_ARG"
    assert code(entropy_src=2, **typ) == "RV_E_ARG"
    assert code(temperature=0.0) == "RV_E_ARG"
    assert code(temperature=float("inf")) == "RV_E_ARG"
    assert code(rule=rv.RV_RULE_SAMPLING) == "RV_E_ARG"  # needs the draft distributions
    q = torch.full((1, 2, shape.vocab), 1.0 / shape.vocab, dtype=torch.float32, device="cuda")

    def code_s(**kw):
        args = dict(prefix_len=lens, draft_ids=d, k=2, draft_probs=q, probe_ids=probe, n_probe=3, alpha=0.3,
                    prefix_pos=2, seed=1, accept_len=v.accept_len, next_id=v.next_id)
        args.update(kw)
        try:
            rv.rv_verify_sampled(v.cache, **args)
        except rv.RVError as e:
            return e.name
        return "RV_OK"

    assert code_s(rule=rv.RV_RULE_GREEDY) == "RV_E_ARG"
    assert code_s(draft_probs=None) == "RV_E_ARG"
    assert code(prefix_len=[1], prefix_pos=2) == "RV_E_RANGE"
    assert code(prefix_len=[41]) == "RV_E_RANGE"
    assert code(prefix_len=[35]) == "RV_E_CAPACITY"
    assert code(n_probe=12) == "RV_E_CAPACITY"
    assert code(probe_ids=None) == "RV_E_ARG"
    # none of the rejected calls enqueued anything: outputs and history as set above
    torch.cuda.synchronize()
    assert v.accept_len.cpu().tolist() == [-11] and v.next_id.cpu().tolist() == [-12]
    assert history() == hist0
    assert code() == "RV_OK"
    torch.cuda.synchronize()
    assert int(v.accept_len[0]) >= 0 and history() != hist0
    v.close()


@pytest.mark.parametrize("shape", [workload.TINY, workload.TINY_GQA_BF16], ids=lambda s: s.name)
@pytest.mark.parametrize("typical", [None, (0.09, 0.3, "fused")])
def test_ragged_draft_counts_match_oracle(rv, gpu, shape, typical):
    """A draft count per sequence (dynamic draft length): each sequence gets
    what the oracle computes for its own block."""
    import torch
    kl = [0, 3, 5, 1]
    hists = [workload.random_ids(shape.vocab, L, 9, b) for b, L in enumerate([44, 70, 52, 61])]
    drafts = [draft_case(shape, 2, h, k, 0.3, 90 + b) if k else [] for b, (h, k) in enumerate(zip(hists, kl))]
    probe = workload.random_ids(shape.vocab, 6, 9, 0xBEEF)
    P, alpha = 4, 0.3
    S = 1 + 2 * max(kl) + len(probe) + P
    v = rv.Verifier(shape, 2, len(hists), max(len(h) for h in hists) + S + 8, max_block=S, max_drafts=max(kl))
    lens = v.prefill([list(map(int, h)) for h in hists])
    kw = {}
    if typical:
        kw = dict(rule=rv.RV_RULE_TYPICAL, epsilon=typical[0], delta=typical[1])
    acc, nxt = v.verify_ragged(lens, drafts, probe, alpha, P, **kw)
    torch.cuda.synchronize()
    acc, nxt = acc.cpu().numpy().copy(), nxt.cpu().numpy().copy()
    out = {w: v.output(w).cpu().numpy() for w in range(8)}
    row = 0
    for b in range(len(hists)):
        okw = dict(rule="typical", eps=typical[0], delta=typical[1], entropy_of=typical[2]) if typical else {}
        ref = oracle.verify(shape, 2, list(map(int, hists[b])), drafts[b], probe, alpha, P, **okw)
        rows = slice(row, row + kl[b] + 1)
        logits_close(shape, out[rv.RV_OUT_ORIG][rows], ref["o"])
        logits_close(shape, out[rv.RV_OUT_REFL][rows], ref["r"])
        logits_close(shape, out[rv.RV_OUT_FUSED][rows], ref["z"])
        s = np.exp(out[rv.RV_OUT_LOGP_FUSED][rows].astype(np.float64)).sum(-1)
        assert np.abs(s - 1).max() < 1e-4
        h_tol = 5e-4 if shape.dtype == "f32" else 2e-2 * max(1.0, float(np.abs(ref["h_z"]).max()))
        assert np.abs(out[rv.RV_OUT_ENTROPY][0][rows] - ref["h_z"]).max() < h_tol
        if not ref["near_tie"]:
            assert (int(acc[b]), int(nxt[b])) == (ref["accept_len"], ref["next_id"]), (b, ref["margins"])
        elif typical:
            assert typical_allowed(ref["z"], ref["o"], drafts[b], int(acc[b]), int(nxt[b]), *typical), b
        else:
            assert greedy_allowed(ref["z"], drafts[b], int(acc[b]), int(nxt[b])), (b, ref["margins"])
        # history: prefix + accepted drafts + t
        n = int(acc[b])
        ids = torch.empty(lens[b] + n + 1, dtype=torch.int32, device="cuda")
        rv.rv_debug_export_ids(v.cache, b, 0, lens[b] + n + 1, ids)
        torch.cuda.synchronize()
        assert ids.cpu().tolist() == list(map(int, hists[b])) + list(drafts[b][:n]) + [int(nxt[b])]
        row += kl[b] + 1
    v.close()


def test_ragged_with_equal_counts_is_the_uniform_call(rv, gpu):
    import torch
    shape = workload.TINY_GQA_BF16
    hists = [workload.random_ids(shape.vocab, L, 10, b) for b, L in enumerate([40, 57])]
    drafts = [draft_case(shape, 1, h, 3, 0.3, 100 + b) for b, h in enumerate(hists)]
    probe = workload.random_ids(shape.vocab, 4, 10, 0xBEEF)
    v = rv.Verifier(shape, 1, 2, 100, max_block=16, max_drafts=3)
    lens = v.prefill([list(map(int, h)) for h in hists])
    a1, n1 = v.verify(lens, np.array(drafts), probe, 0.3, 4)
    torch.cuda.synchronize()
    r1 = (a1.cpu().numpy().copy(), n1.cpu().numpy().copy(), {w: v.output(w).cpu().numpy() for w in range(8)})
    a2, n2 = v.verify_ragged(lens, drafts, probe, 0.3, 4)
    torch.cuda.synchronize()
    assert (a2.cpu().numpy() == r1[0]).all() and (n2.cpu().numpy() == r1[1]).all()
    for w in range(6):
        np.testing.assert_array_equal(v.output(w).cpu().numpy().reshape(r1[2][w].shape), r1[2][w])
    v.close()


@pytest.mark.parametrize("shape,B", [(workload.TINY, 256), (workload.TINY_GQA_BF16, 64)], ids=["tiny-f32", "tiny-bf16"])
def test_maximum_drafts_and_batch(rv, gpu, shape, B):
    """k = RV_MAX_DRAFTS drafts for a batch of up to RV_MAX_BATCH sequences
    (blocks of 1 + 2k + |R| + P = 73 rows), at alpha = 0.3 and 0.  Every
    sequence's decision must be Algorithm 2 applied to the fused rows the
    pass itself returns (lowest id on ties).  Sequences 0 and 1 share a
    history whose drafts are the oracle's greedy continuation (sequence 1's
    replaced half way), and the last sequence has random drafts; those three
    are compared with the oracle.  At alpha = 0 (z = o, Eq. 2) all 32 greedy
    drafts are accepted and the replaced one is rejected."""
    import torch
    k, P = rv.RV_MAX_DRAFTS, 4
    hists = [list(map(int, workload.random_ids(shape.vocab, 24 + b % 17, 31, b))) for b in range(B)]
    hists[1] = hists[0]
    drafts = np.stack([workload.random_ids(shape.vocab, k, 31, 7, b) for b in range(B)]).astype(np.int32)
    past = oracle.prefix_kv(shape, 5, hists[0][:-1])
    drafts[0] = oracle.greedy_continuation(shape, 5, hists[0], k, past=past)
    drafts[1] = drafts[0]
    drafts[1, k // 2] = (drafts[1, k // 2] + 1) % shape.vocab
    probe = workload.random_ids(shape.vocab, 4, 31, 0xBEEF)
    S = 1 + 2 * k + len(probe) + P
    v = rv.Verifier(shape, 5, B, max(len(h) for h in hists) + S + 8, max_block=S, max_drafts=k)
    got = {}
    try:
        lens = v.prefill(hists)
        for alpha in (0.3, 0.0):
            acc, nxt = v.verify(lens, drafts, probe, alpha, P)
            torch.cuda.synchronize()
            got[alpha] = (acc.cpu().numpy().copy(), nxt.cpu().numpy().copy(), v.output(rv.RV_OUT_FUSED).cpu().numpy())
    finally:
        v.close()
    for alpha, (acc, nxt, z) in got.items():
        for b in range(B):
            am = np.argmax(z[b], axis=-1)
            n = next((i for i in range(k) if am[i] != drafts[b][i]), k)
            assert (int(acc[b]), int(nxt[b])) == (n, int(am[n])), (alpha, b)
    for b in (0, 1, B - 1):
        ref = oracle.verify(shape, 5, hists[b], drafts[b], probe, 0.3, P, past=past if b < 2 else None)
        acc, nxt, z = got[0.3]
        logits_close(shape, z[b], ref["z"])
        if not ref["near_tie"]:
            assert (int(acc[b]), int(nxt[b])) == (ref["accept_len"], ref["next_id"]), (b, ref["margins"])
        else:
            assert greedy_allowed(ref["z"], drafts[b], int(acc[b]), int(nxt[b])), b
        z0 = oracle.fuse(ref["o"], ref["r"], 0.0).astype(np.float64)
        n0, t0 = oracle.accept_greedy(z0, drafts[b])
        acc, nxt, z = got[0.0]
        logits_close(shape, z[b], z0)
        if not oracle.decision_margins(z0, drafts[b], n0)[2]:
            assert (int(acc[b]), int(nxt[b])) == (n0, t0), b
    assert int(got[0.0][0][0]) == k and int(got[0.0][0][1]) == k // 2
