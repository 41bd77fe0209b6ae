"""GPU tests at the real model shapes (through the C ABI).

* Matrix kernels at every 8B matrix shape and the LM head, in the launch
  shapes a verify pass uses, on seeded operands: sampled output columns are
  compared with the oracle's fp64 dot products (the oracle computes them one
  by one from its own weight generator).
* A reduced-depth model with the 8B widths (2 layers, vocab 128256): full
  verify parity against the oracle.
* The full 8B-shaped verify (32 layers, prefix 1024): properties that hold
  at any size (Eq. 2 exactly, log-softmax sums, the rule on its own logits,
  repeatability, probe independence).  The comparison of that whole pass with
  the oracle is in test_gpu_fulldepth.py, against results the oracle stored.
"""
import numpy as np
import pytest

import oracle
import workload

pytestmark = pytest.mark.gpu

SHAPE = workload.LLAMA8B


def split_planes(x):
    """bf16 hi/lo planes [2][M][K] of an fp32 matrix, and their exact sum."""
    import torch
    x32 = torch.from_numpy(np.asarray(x, dtype=np.float32))
    hi = x32.to(torch.bfloat16)
    lo = (x32 - hi.float()).to(torch.bfloat16)
    planes = torch.stack([hi, lo]).contiguous()
    exact = hi.double().numpy() + lo.double().numpy()
    return planes, exact


@pytest.fixture(scope="module")
def model8b(rv, gpu):
    v = rv.Verifier(SHAPE, 0, 1, 1100, max_block=64, max_drafts=16)
    yield v
    v.close()


@pytest.mark.parametrize("M", [12, 31, 100, 496])
@pytest.mark.parametrize("layer,matrix", [(0, "qkv"), (31, "o"), (0, "gateup"), (17, "down"), (None, "lm_head")])
def test_matrix_kernel_full_shape(rv, model8b, M, layer, matrix):
    import torch
    mat = {"qkv": rv.RV_MAT_QKV, "o": rv.RV_MAT_O, "gateup": rv.RV_MAT_GATEUP, "down": rv.RV_MAT_DOWN,
           "lm_head": rv.RV_MAT_LM_HEAD}[matrix]
    parts = {"qkv": ["q", "k", "v"], "o": ["o"], "gateup": ["gate", "up"], "down": ["down"],
             "lm_head": ["lm_head"]}[matrix]
    K = oracle.tensor_dims(SHAPE, parts[0])[1]
    sizes = [oracle.tensor_dims(SHAPE, p)[0] for p in parts]
    N = sum(sizes)
    rng = np.random.default_rng([M, K, N])
    x = rng.standard_normal((M, K)).astype(np.float32)
    planes, xe = split_planes(x)
    y = torch.empty((M, N), dtype=torch.float32, device="cuda")
    rv.rv_debug_linear(model8b.cache, layer if layer is not None else 0, mat, planes.cuda(), y)
    torch.cuda.synchronize()
    got = y.cpu().numpy()
    # 48 sampled output columns, always including both ends of every part
    cols = set(rng.integers(0, N, 40).tolist())
    off = 0
    for p, n in zip(parts, sizes):
        cols.update([off, off + n - 1])
        off += n
    for col in sorted(cols):
        off = 0
        for p, n in zip(parts, sizes):
            if col < off + n:
                wrow = oracle.weight(SHAPE, 0, layer, p, col - off, 1)[0]
                break
            off += n
        ref = xe @ wrow
        scale = np.sqrt((xe * xe).sum(1) * (wrow * wrow).sum())
        err = np.abs(got[:, col] - ref)
        assert (err <= 2e-6 * scale + 1e-6).all(), (matrix, col, float((err / scale).max()))


def test_reduced_depth_8b_width_matches_oracle(rv, gpu):
    """Full widths, vocabulary and head layout of the 8B shape, 2 layers."""
    import torch
    shape = SHAPE.with_layers(2)
    hists = [workload.random_ids(shape.vocab, L, 11, b) for b, L in enumerate([64, 45])]
    drafts = [workload.random_ids(shape.vocab, 5, 11, 10 + b) for b in range(2)]
    # sequence 1 drafts the model's own greedy continuation (accepted at alpha = 0)
    g = oracle.greedy_continuation(shape, 0, list(map(int, hists[1])), 2)
    drafts[1][:2] = g
    probe = workload.random_ids(shape.vocab, 16, 11, 0xBEEF)
    v = rv.Verifier(shape, 0, 2, 160, max_block=64, max_drafts=8)
    lens = v.prefill([list(map(int, h)) for h in hists])
    for alpha in (0.3, 0.0):
        acc, nxt = v.verify(lens, np.array(drafts), probe, alpha, 4)
        torch.cuda.synchronize()
        outs = {w: v.output(w).cpu().numpy() for w in (rv.RV_OUT_ORIG, rv.RV_OUT_REFL, rv.RV_OUT_FUSED)}
        for b in range(2):
            ref = oracle.verify(shape, 0, list(map(int, hists[b])), drafts[b], probe, alpha, 4)
            for w, key in ((rv.RV_OUT_ORIG, "o"), (rv.RV_OUT_REFL, "r"), (rv.RV_OUT_FUSED, "z")):
                rel = (np.abs(outs[w][b] - ref[key]).max(-1) / np.abs(ref[key]).max(-1)).max()
                assert rel <= 2e-2, (alpha, b, key, rel)
                # the hi/lo operand contract keeps GPU and oracle far closer than the bar
                assert np.abs(outs[w][b] - ref[key]).max() < 1e-3, (alpha, b, key)
            if not ref["near_tie"]:
                assert (int(acc[b]), int(nxt[b])) == (ref["accept_len"], ref["next_id"]), (alpha, b, ref["margins"])
            if alpha == 0.0 and b == 1:
                assert int(acc[b]) >= 2
    v.close()


# ---------------------------------------------------------------- full 8B verify

@pytest.fixture(scope="module")
def verify8b(rv, model8b):
    import torch
    w = workload.WORKLOADS["8b-bf16-b1"]
    lens = [int(x) for x in workload.prefix_lengths(w)]
    prefix = [int(t) for t in workload.prefix_ids(w, lens)[0]]
    model8b.prefill([prefix])
    # greedy continuation through single-row verifies (k = 0, no probe)
    greedy, cur = [], lens[0]
    for _ in range(w.k + 1):
        _, nxt = model8b.verify([cur], np.zeros((1, 0), np.int32), [], 0.0, 0)
        greedy.append(int(nxt[0]))
        cur += 1
    torch.cuda.synchronize()
    return dict(w=w, lens=lens, prefix=prefix, greedy=greedy, probe=workload.probe_ids(w))


def _run(rv, v, lens, drafts, probe, alpha, P):
    import torch
    acc, nxt = v.verify(lens, np.array([drafts]), probe, alpha, P)
    torch.cuda.synchronize()
    return int(acc[0]), int(nxt[0]), {w: v.output(w).cpu().numpy()[0] for w in range(6)}


def test_full_8b_properties(rv, model8b, verify8b):
    d = verify8b
    w = d["w"]
    drafts = list(workload.corrupt(d["greedy"][:w.k], 0.3, SHAPE.vocab, np.random.default_rng(7)))
    n, t, out = _run(rv, model8b, d["lens"], drafts, d["probe"], w.alpha, w.prefix_pos)
    o, r, z = out[rv.RV_OUT_ORIG], out[rv.RV_OUT_REFL], out[rv.RV_OUT_FUSED]
    # Eq. 2 exactly, in fp32
    a = np.float32(w.alpha)
    np.testing.assert_array_equal(z, (np.float32(1) - a) * o + a * r)
    # log-softmax rows sum to one
    for wh in (rv.RV_OUT_LOGP_ORIG, rv.RV_OUT_LOGP_REFL, rv.RV_OUT_LOGP_FUSED):
        s = np.exp(out[wh].astype(np.float64)).sum(-1)
        assert np.abs(s - 1).max() < 1e-4
    # the decision is the exact-match rule applied to the GPU's own fused logits
    xhat = np.argmax(z, -1)
    n_ref = next((i for i in range(w.k) if xhat[i] != drafts[i]), w.k)
    assert (n, t) == (n_ref, int(xhat[n_ref]))
    # repeating the call gives bit-identical results
    n2, t2, out2 = _run(rv, model8b, d["lens"], drafts, d["probe"], w.alpha, w.prefix_pos)
    assert (n2, t2) == (n, t)
    for k_ in out:
        np.testing.assert_array_equal(out[k_], out2[k_])
    # another probe of the same length leaves the original rows bit-identical
    probe2 = workload.random_ids(SHAPE.vocab, w.n_probe, 99, 1)
    _, _, out3 = _run(rv, model8b, d["lens"], drafts, probe2, w.alpha, w.prefix_pos)
    np.testing.assert_array_equal(out3[rv.RV_OUT_ORIG], o)
    assert np.abs(out3[rv.RV_OUT_REFL] - r).max() > 1e-3


def test_full_8b_greedy_drafts_accepted_at_alpha_zero(rv, model8b, verify8b):
    d = verify8b
    w = d["w"]
    n, t, out = _run(rv, model8b, d["lens"], d["greedy"][:w.k], d["probe"], 0.0, w.prefix_pos)
    assert (n, t) == (w.k, d["greedy"][w.k])
    np.testing.assert_array_equal(out[rv.RV_OUT_FUSED], out[rv.RV_OUT_ORIG])


def test_full_8b_commit_matches_fresh_prefill(rv, gpu, model8b, verify8b):
    """After a verify accepts n drafts, the KV kept at positions L-1..L-1+n is
    what a prefill of the extended prefix computes (the template and second
    copy leave no trace, Section 3.1)."""
    import torch
    d = verify8b
    w = d["w"]
    drafts = list(d["greedy"][:3]) + [int(x) for x in workload.random_ids(SHAPE.vocab, 2, 5, 5)]
    n, t, _ = _run(rv, model8b, d["lens"], drafts, d["probe"], w.alpha, w.prefix_pos)
    L = d["lens"][0]
    ext = d["prefix"] + drafts[:n] + [t]
    ids = torch.empty(len(ext), dtype=torch.int32, device="cuda")
    rv.rv_debug_export_ids(model8b.cache, 0, 0, len(ext), ids)
    npos = n + 1
    kv_a = []
    def export(cache, layer):
        # bf16 cache: hi plane then lo plane, value = hi + lo
        k_ = torch.empty((2, SHAPE.n_kv_heads, npos, SHAPE.head_dim), dtype=torch.bfloat16, device="cuda")
        v_ = torch.empty_like(k_)
        rv.rv_debug_export_kv(cache, layer, 0, L - 1, npos, k_, v_)
        torch.cuda.synchronize()
        return k_.double().sum(0).cpu().numpy(), v_.double().sum(0).cpu().numpy()

    for layer in (0, 15, 31):
        kv_a.append(export(model8b.cache, layer))
    torch.cuda.synchronize()
    assert ids.cpu().tolist() == ext
    fresh = rv.Verifier(SHAPE, 0, 1, len(ext) + 8, max_block=16, max_drafts=4)
    fresh.prefill([ext])
    for (ka, va), layer in zip(kv_a, (0, 15, 31)):
        kb, vb = export(fresh.cache, layer)
        for a_, b_ in ((ka, kb), (va, vb)):
            # different launch shapes sum in a different order: fp32 rounding
            # differences that grow slowly through the layers
            assert np.abs(a_ - b_).max() <= 1e-3 * np.abs(b_).max(), (layer, float(np.abs(a_ - b_).max()))
    fresh.close()


def test_full_8b_typical_rule_properties(rv, model8b, verify8b):
    """Algorithm 3's rule at the full 8B shape: the decision equals the rule
    applied to the GPU's own log-probabilities and entropies; eps = inf with
    delta = 0 accepts every draft."""
    import torch
    d = verify8b
    w = d["w"]
    drafts = list(workload.corrupt(d["greedy"][:w.k], 0.5, SHAPE.vocab, np.random.default_rng(9)))
    for eps, delta, src in ((0.09, 0.3, rv.RV_ENTROPY_FUSED), (0.5, 2.0, rv.RV_ENTROPY_ORIGINAL)):
        acc, nxt = model8b.verify(d["lens"], np.array([drafts]), d["probe"], w.alpha, w.prefix_pos,
                                  rule=rv.RV_RULE_TYPICAL, epsilon=eps, delta=delta, entropy_src=src)
        torch.cuda.synchronize()
        n, t = int(acc[0]), int(nxt[0])
        lp = model8b.output(rv.RV_OUT_LOGP_FUSED).cpu().numpy()[0].astype(np.float64)
        z = model8b.output(rv.RV_OUT_FUSED).cpu().numpy()[0]
        H = model8b.output(rv.RV_OUT_ENTROPY).cpu().numpy()[:, 0].astype(np.float64)
        h = H[0] if src == rv.RV_ENTROPY_FUSED else H[1]
        # the entropies are those of the GPU's own log-probabilities
        lpo = model8b.output(rv.RV_OUT_LOGP_ORIG).cpu().numpy()[0].astype(np.float64)
        np.testing.assert_allclose(H[0], -(np.exp(lp) * lp).sum(-1), atol=2e-3)
        np.testing.assert_allclose(H[1], -(np.exp(lpo) * lpo).sum(-1), atol=2e-3)
        margins = [lp[i][drafts[i]] - min(np.log(eps), np.log(delta) - h[i]) for i in range(w.k)]
        n_ref = next((i for i, m in enumerate(margins) if not m > 0), w.k)
        if all(abs(m) > 1e-3 for m in margins[:n_ref + 1]):
            assert (n, t) == (n_ref, int(np.argmax(z[n_ref])))
    acc, nxt = model8b.verify(d["lens"], np.array([drafts]), d["probe"], w.alpha, w.prefix_pos,
                              rule=rv.RV_RULE_TYPICAL, epsilon=float("inf"), delta=0.0)
    torch.cuda.synchronize()
    z = model8b.output(rv.RV_OUT_FUSED).cpu().numpy()[0]
    assert (int(acc[0]), int(nxt[0])) == (w.k, int(np.argmax(z[w.k])))


def test_full_8b_sampling_rule_properties(rv, model8b, verify8b):
    """Algorithm 1's rule at the full 8B shape: with q equal to the fused
    distribution every draft is accepted; with another q the decision equals
    the rule applied to the GPU's own probabilities and the Philox uniforms."""
    import torch
    d = verify8b
    w = d["w"]
    V = SHAPE.vocab
    drafts = list(d["greedy"][:w.k])
    T = 0.8
    # the fused distribution at temperature T, from a greedy-rule call
    model8b.verify(d["lens"], np.array([drafts]), d["probe"], w.alpha, w.prefix_pos, temperature=T)
    torch.cuda.synchronize()
    lp = model8b.output(rv.RV_OUT_LOGP_FUSED).cpu().numpy()[0].astype(np.float64)
    p = np.exp(lp)
    acc, nxt = model8b.verify_sampled(d["lens"], np.array([drafts]), p[None, :w.k].astype(np.float32), d["probe"],
                                      w.alpha, w.prefix_pos, 99, temperature=T)
    torch.cuda.synchronize()
    assert int(acc[0]) == w.k
    # a flatter q: decisions from the GPU's own p and the same uniforms
    q = (0.5 * p[:w.k] + 0.5 / V).astype(np.float32)
    for seed in (1, 2, 3):
        acc, nxt = model8b.verify_sampled(d["lens"], np.array([drafts]), q[None], d["probe"], w.alpha,
                                          w.prefix_pos, seed, temperature=T)
        torch.cuda.synchronize()
        n = int(acc[0])
        lp_s = model8b.output(rv.RV_OUT_LOGP_FUSED).cpu().numpy()[0].astype(np.float64)
        margins = [lp_s[i][drafts[i]] - np.log(oracle.acceptance_uniform(seed, 0, i) * float(q[i][drafts[i]]))
                   for i in range(w.k)]
        n_ref = next((i for i, m in enumerate(margins) if m < 0), w.k)
        if all(abs(m) > 1e-4 for m in margins[:n_ref + 1]):
            assert n == n_ref, (seed, margins)
        t = int(nxt[0])
        assert 0 <= t < V
        if n < w.k:  # the residual draw never picks a token with p <= q
            assert np.exp(lp_s[n][t]) > q[n][t] * (1 - 1e-5)
