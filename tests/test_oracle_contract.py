"""Pins of the oracle's precision contract (CPU only).

The GPU library keeps every matmul result and the residual stream in fp32
and every value that feeds a later matmul (norm outputs, rotated queries,
the K/V cache, attention outputs, SwiGLU outputs) as a bf16 pair
hi = bf16(x), lo = bf16(x - hi) of its fp32 value; the oracle's "contract"
mode rounds at exactly those points.  These tests pin that mode to things
other than itself:

* its distance from the fp64 "exact" mode (which is pinned to a library
  Llama) is what ~16-bit operands and fp32 results allow, and a single-bf16
  operand planted at any one rounding point, which is what a wrong rounding
  point would look like, moves it well past that;
* the values it stores have the representation the contract names (fp32
  results, hi/lo operands that carry more than bf16), so a dropped fp32
  rounding or a missing lo plane is caught even where it moves the result
  towards the exact one;
* the hi/lo split agrees with torch's float32 -> bfloat16 conversion and
  meets its error bound, and the fp32 rotary table is the correctly rounded
  fp64 one;
* the temperature division of the fused logits is the correctly rounded
  fp32 quotient and leaves greedy decisions unchanged;
* reusing a prefix's K/V gives what recomputing it from scratch gives.
"""
import numpy as np
import pytest
import torch

import oracle
import workload

# contract vs exact relative to the largest logit, measured: 6.2e-6 (tiny
# GQA bf16) and 1.4e-5 (8B widths, two layers)
CONTRACT_REL = {"tiny-gqa-bf16": 2e-5, "8b-width-2-layers": 5e-5}


def _rel(a, b):
    return float(np.abs(a - b).max() / np.abs(b).max())


@pytest.mark.parametrize("shape,n", [(workload.TINY_GQA_BF16, 25), (workload.LLAMA8B.with_layers(2), 20)],
                         ids=["tiny-gqa-bf16", "8b-width-2-layers"])
def test_contract_is_close_to_exact(request, shape, n):
    tokens = workload.random_ids(shape.vocab, n, 7, 3)
    ex = oracle.forward(shape, 4, tokens, [n - 1, n - 6], mode="exact")
    ct = oracle.forward(shape, 4, tokens, [n - 1, n - 6], mode="contract")
    rel = _rel(ct, ex)
    assert 0 < rel < CONTRACT_REL[request.node.callspec.id], rel


def _single_bf16(monkeypatch, point):
    """Plant a single-bf16 operand (no lo plane) at one rounding point."""
    real_mm = oracle._matmul_wT
    real_att = oracle.causal_attention
    consumers = {"norm_out": ("q", "k", "v", "gate", "up", "lm_head"), "att_out": ("o",), "act": ("down",)}
    if point in consumers:
        names = consumers[point]

        def mm(shape, seed, layer, name, a, rnd, *args, **kw):
            if name in names:
                a = oracle.round_bf16(a)
            return real_mm(shape, seed, layer, name, a, rnd, *args, **kw)
        monkeypatch.setattr(oracle, "_matmul_wT", mm)
    elif point == "q":
        monkeypatch.setattr(oracle, "causal_attention",
                            lambda q, k, v, q_pos=None, **kw: real_att(oracle.round_bf16(q), k, v, q_pos, **kw))
    elif point == "kv":
        monkeypatch.setattr(oracle, "causal_attention",
                            lambda q, k, v, q_pos=None, **kw: real_att(q, oracle.round_bf16(k), oracle.round_bf16(v),
                                                                       q_pos, **kw))
    else:
        raise ValueError(point)


@pytest.mark.parametrize("point", ["norm_out", "q", "kv", "att_out", "act"])
def test_planted_single_bf16_operand_breaks_the_bound(monkeypatch, point):
    shape = workload.TINY_GQA_BF16
    tokens = workload.random_ids(shape.vocab, 25, 7, 3)
    ex = oracle.forward(shape, 4, tokens, [24, 19], mode="exact")
    _single_bf16(monkeypatch, point)
    bad = oracle.forward(shape, 4, tokens, [24, 19], mode="contract")
    # measured 1.2e-4 (q) to several 1e-3 (the others)
    assert _rel(bad, ex) > 3 * CONTRACT_REL["tiny-gqa-bf16"], (point, _rel(bad, ex))


def _is_f32(x):
    x = np.asarray(x, dtype=np.float64)
    return np.array_equal(x, x.astype(np.float32).astype(np.float64))


def _is_pair(x):
    """A fixed point of the hi/lo split, i.e. exactly hi + lo."""
    x = np.asarray(x, dtype=np.float64)
    return np.array_equal(oracle.split_bf16(x), x)


def _bf16_fraction(x):
    x = np.asarray(x, dtype=np.float64)
    return float(np.mean(oracle.round_bf16(x) == x))


RESULTS = ("o_proj", "gate", "up", "down", "resid", "resid_mid")
OPERANDS = ("norm_in", "q", "k", "v", "att", "ffn_in", "act")


def _trace(shape, mode="contract"):
    tokens = workload.random_ids(shape.vocab, 30, 8, 1)
    tr = {}
    oracle.forward(shape, 2, tokens, [29, 10], mode=mode, trace=tr)
    return tr


def test_stored_values_have_the_contract_representation():
    tr = _trace(workload.TINY_GQA_BF16)
    for key in RESULTS:
        for layer, x in enumerate(tr[key]):
            assert _is_f32(x), (key, layer)
    assert _is_f32(tr["logits"])
    for key in OPERANDS:
        for layer, x in enumerate(tr[key]):
            assert _is_pair(x), (key, layer)
            # a pair carries ~16 significant bits: few values are plain bf16
            assert _bf16_fraction(x) < 0.05, (key, layer, _bf16_fraction(x))
    assert _is_pair(tr["final_in"])
    # the exact mode stores fp64 values: the same checks fail there
    ex = _trace(workload.TINY_GQA_BF16, "exact")
    assert not _is_f32(ex["gate"][0]) and not _is_pair(ex["act"][0])


def test_dropped_fp32_rounding_is_caught(monkeypatch):
    monkeypatch.setattr(oracle._Rounding, "f32", lambda self, x: x)
    tr = _trace(workload.TINY_GQA_BF16)
    assert not all(_is_f32(x) for key in RESULTS for x in tr[key])


def test_fp32_contract_stores_fp32():
    tr = _trace(workload.TINY)
    for key in RESULTS + OPERANDS:
        for x in tr[key]:
            assert _is_f32(x), key


def test_split_matches_torch_and_its_bound():
    rng = np.random.default_rng(3)
    x = np.concatenate([rng.standard_normal(50000) * 10.0 ** rng.integers(-8, 8, 50000),
                        [0.0, -0.0, 1.0, 1.0 + 2.0 ** -9, 3.0 + 2.0 ** -20]])
    x32 = torch.from_numpy(x).to(torch.float32)
    hi = x32.to(torch.bfloat16)
    lo = (x32 - hi.to(torch.float32)).to(torch.bfloat16)
    ref = hi.double().numpy() + lo.double().numpy()
    got = oracle.split_bf16(x)
    np.testing.assert_array_equal(got, ref)
    # hi carries 8 significant bits and lo the next 8 (rounded): the pair is
    # within 2^-17 of the fp32 value, relative, for normal numbers
    xf = x32.double().numpy()
    big = np.abs(xf) > 1e-30
    assert (np.abs(got - xf)[big] <= 2.0 ** -17 * np.abs(xf)[big]).all()


def test_rope_table_is_correctly_rounded_fp32():
    shape = workload.LLAMA8B
    rnd = oracle._Rounding(shape, "contract")
    pos = np.array([0, 1, 2, 1023, 1053, 4124, 8234])
    cos, sin = oracle.rope_table(shape, pos, rnd)
    i = np.arange(shape.head_dim // 2)
    ang = pos[:, None] * shape.rope_base ** (-2.0 * i / shape.head_dim)
    for tab, ref in ((cos, np.cos(ang)), (sin, np.sin(ang))):
        assert _is_f32(tab)
        # within half an fp32 ulp of the fp64 value (correct rounding)
        ulp = np.spacing(np.abs(tab).astype(np.float32)).astype(np.float64)
        assert (np.abs(tab - ref) <= 0.5 * ulp + 1e-300).all()


@pytest.mark.parametrize("shape", [workload.TINY, workload.TINY_GQA_BF16], ids=lambda s: s.name)
def test_temperature_divides_the_fused_logits(shape):
    hist = [int(t) for t in workload.random_ids(shape.vocab, 40, 13, 0)]
    drafts = [int(t) for t in workload.random_ids(shape.vocab, 3, 13, 1)]
    probe = workload.random_ids(shape.vocab, 4, 13, 2)
    past = oracle.prefix_kv(shape, 1, hist[:-1])
    base = oracle.verify(shape, 1, hist, drafts, probe, 0.3, 2, past=past)
    z = base["z"]
    assert _is_f32(z)
    for T, scale in ((0.5, 2.0), (0.25, 4.0)):  # powers of two divide exactly
        got = oracle.verify(shape, 1, hist, drafts, probe, 0.3, 2, temperature=T, past=past)
        np.testing.assert_array_equal(got["z"], z * scale)
        assert (got["accept_len"], got["next_id"]) == (base["accept_len"], base["next_id"])
    got = oracle.verify(shape, 1, hist, drafts, probe, 0.3, 2, temperature=0.8, past=past)
    zt = got["z"]
    assert _is_f32(zt)
    ulp = np.spacing(np.abs(zt).astype(np.float32)).astype(np.float64)
    assert (np.abs(zt - z / np.float64(np.float32(0.8))) <= 0.5 * ulp).all()
    # greedy decisions do not depend on the temperature
    assert (got["accept_len"], got["next_id"]) == (base["accept_len"], base["next_id"])


@pytest.mark.parametrize("shape", [workload.TINY, workload.TINY_GQA_BF16], ids=lambda s: s.name)
@pytest.mark.parametrize("mode", ["contract", "exact"])
def test_prefix_kv_reuse_equals_recomputation(shape, mode):
    hist = [int(t) for t in workload.random_ids(shape.vocab, 57, 14, 0)]
    drafts = [int(t) for t in workload.random_ids(shape.vocab, 4, 14, 1)]
    probe = workload.random_ids(shape.vocab, 6, 14, 2)
    past = oracle.prefix_kv(shape, 2, hist[:-1], mode)
    assert past[0].shape == (shape.n_layers, len(hist) - 1, shape.n_kv_heads, shape.head_dim)
    a = oracle.verify(shape, 2, hist, drafts, probe, 0.3, 4, mode=mode)
    b = oracle.verify(shape, 2, hist, drafts, probe, 0.3, 4, mode=mode, past=past)
    for key in ("o", "r", "z"):
        assert _rel(b[key], a[key]) <= 1e-12, key
    assert (a["accept_len"], a["next_id"]) == (b["accept_len"], b["next_id"])
    g1 = oracle.greedy_continuation(shape, 2, hist, 4, mode)
    g2 = oracle.greedy_continuation(shape, 2, hist, 4, mode, past=past)
    assert g1 == g2
    # the K/V a later verify attends equal those of a longer prefix
    ks, vs = oracle.prefix_kv(shape, 2, hist, mode)
    np.testing.assert_allclose(ks[:, :len(hist) - 1], past[0], rtol=0, atol=1e-12 * np.abs(ks).max())
    np.testing.assert_allclose(vs[:, :len(hist) - 1], past[1], rtol=0, atol=1e-12 * np.abs(vs).max())
