"""Pins of the CPU oracle against things other than itself (CPU only).

* the weight generator against the published splitmix64 stream and the
  moments of the Irwin-Hall(4) distribution;
* the bf16 rounding against torch's float32 -> bfloat16 conversion;
* the decoder forward against a library implementation of the same
  architecture (transformers' LlamaForCausalLM, fp64), and a planted mistake
  in the oracle must break that agreement;
* closed forms of RMSNorm and rotary embedding.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workload


def test_splitmix64_published_stream():
    # First outputs of splitmix64 started at seed 0 (reference implementation
    # of Steele, Lea and Flood's generator).
    assert oracle.splitmix64_stream(0, 3) == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


@pytest.mark.parametrize("shape", [workload.TINY, workload.TINY_GQA_BF16])
def test_weight_moments(shape):
    w = oracle.weight(shape, 0, 0, "gate").ravel()
    n = w.size
    assert abs(w.mean()) < 5 * 0.02 / math.sqrt(n)
    assert abs(w.std() / 0.02 - 1.0) < 0.01
    # Irwin-Hall(4) support: |s| <= 2*65535, i.e. 2 * sqrt(3) sigma
    assert np.abs(w).max() <= 2 * math.sqrt(3) * 0.02 * 1.0001
    # different tensors and seeds give different values
    assert not np.array_equal(w[:64], oracle.weight(shape, 0, 0, "up").ravel()[:64])
    assert not np.array_equal(w[:64], oracle.weight(shape, 1, 0, "gate").ravel()[:64])


def test_weight_bits_match_values():
    s = workload.TINY_GQA_BF16
    idx = np.array([0, 1, 17, 4095, 12345], dtype=np.uint64)
    bits = oracle.weight_bits(s, 5, 1, "v", idx)
    vals = oracle.fill(s, 5, oracle.tensor_index(s, 1, "v"), 0, 12346)[idx.astype(np.int64)]
    as_f = (bits.astype(np.uint32) << 16).view(np.float32)
    np.testing.assert_array_equal(as_f.astype(np.float64), vals)


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(20000) * 10.0 ** rng.integers(-6, 6, 20000),
        # exact halfway cases between adjacent bf16 values
        np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -(2.0 + 2.0 ** -7), 3.0 + 2.0 ** -7]),
    ]).astype(np.float32).astype(np.float64)
    ref = torch.from_numpy(x).to(torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(oracle.round_bf16(x), ref)


# ------------------------------------------------------------------ decoder

def hf_llama(shape, seed):
    from transformers import LlamaConfig, LlamaForCausalLM
    cfg = LlamaConfig(
        vocab_size=shape.vocab, hidden_size=shape.d_model, intermediate_size=shape.ffn_dim,
        num_hidden_layers=shape.n_layers, num_attention_heads=shape.n_heads,
        num_key_value_heads=shape.n_kv_heads, head_dim=shape.head_dim, rms_norm_eps=shape.rms_eps,
        max_position_embeddings=4096, rope_parameters={"rope_type": "default", "rope_theta": shape.rope_base},
        tie_word_embeddings=False, attention_bias=False, mlp_bias=False)
    cfg._attn_implementation = "eager"
    model = LlamaForCausalLM(cfg).to(torch.float64).eval()
    names = {"q": "self_attn.q_proj", "k": "self_attn.k_proj", "v": "self_attn.v_proj", "o": "self_attn.o_proj",
             "gate": "mlp.gate_proj", "up": "mlp.up_proj", "down": "mlp.down_proj"}
    sd = {"model.embed_tokens.weight": oracle.weight(shape, seed, None, "embed"),
          "lm_head.weight": oracle.weight(shape, seed, None, "lm_head")}
    for l in range(shape.n_layers):
        for nm, key in names.items():
            sd[f"model.layers.{l}.{key}.weight"] = oracle.weight(shape, seed, l, nm)
    with torch.no_grad():
        for key, param in model.state_dict().items():
            if key in sd:
                param.copy_(torch.from_numpy(sd[key]))
            else:
                assert key.endswith("norm.weight"), key
                param.fill_(1.0)
    return model


def hf_logits(model, tokens):
    with torch.no_grad():
        return model(torch.tensor([list(tokens)])).logits[0].numpy()


PIN_SHAPES = [workload.TINY, workload.TINY_GQA_BF16]


@pytest.mark.parametrize("shape", PIN_SHAPES, ids=lambda s: s.name)
def test_forward_matches_library_llama(shape):
    tokens = workload.random_ids(shape.vocab, 33, 7, 1)
    model = hf_llama(shape, 3)
    ref = hf_logits(model, tokens)
    got = oracle.forward(shape, 3, tokens, list(range(len(tokens))), mode="exact")
    # the library keeps RMSNorm and the rotary angles in fp32 internally
    assert np.abs(got - ref).max() < 1e-5 * np.abs(ref).max()


@pytest.mark.parametrize("shape", PIN_SHAPES, ids=lambda s: s.name)
def test_forward_at_scattered_rows_matches_library(monkeypatch, shape):
    """The last layer runs only on the requested rows (the causal mask makes
    each row's output independent of later rows): logits at a scattered,
    unordered subset equal the library's logits at those positions."""
    tokens = workload.random_ids(shape.vocab, 33, 7, 1)
    ref = hf_logits(hf_llama(shape, 3), tokens)
    rows = [32, 0, 17, 5, 31]
    got = oracle.forward(shape, 3, tokens, rows, mode="exact")
    assert np.abs(got - ref[rows]).max() < 1e-5 * np.abs(ref).max()
    # a query masked as if it sat at the first rows' positions is caught
    real = oracle.causal_attention
    monkeypatch.setattr(oracle, "causal_attention", lambda q, k, v, q_pos=None: real(q, k, v, None))
    bad = oracle.forward(shape, 3, tokens, rows, mode="exact")
    assert np.abs(bad - ref[rows]).max() > 1e-3 * np.abs(ref).max()


def _wrong_rope(x, cos, sin):
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([x1 * c + x2 * s, x2 * c - x1 * s], axis=-1)  # sign flipped


def _wrong_norm(h, eps):
    return h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True))  # epsilon dropped


@pytest.mark.parametrize("mistake", ["rope_sign", "gqa_group", "silu_as_relu", "causal_off", "norm_eps_dropped"])
def test_planted_mistakes_break_the_pin(monkeypatch, mistake):
    shape = workload.TINY_GQA_BF16
    tokens = workload.random_ids(shape.vocab, 17, 7, 2)
    ref = hf_logits(hf_llama(shape, 3), tokens)
    if mistake == "rope_sign":
        monkeypatch.setattr(oracle, "rope", _wrong_rope)
    elif mistake == "gqa_group":
        real = oracle.causal_attention

        def interleaved(q, k, v, q_pos=None):  # q head h -> kv head h % Hkv instead of h // G
            n, Hq, hd = q.shape
            Hkv = k.shape[1]
            kk = np.stack([k[:, h % Hkv] for h in range(Hq)], axis=1)
            vv = np.stack([v[:, h % Hkv] for h in range(Hq)], axis=1)
            return real(q, kk, vv, q_pos)
        monkeypatch.setattr(oracle, "causal_attention", interleaved)
    elif mistake == "norm_eps_dropped":
        monkeypatch.setattr(oracle, "rms_norm", _wrong_norm)
    elif mistake == "silu_as_relu":
        monkeypatch.setattr(oracle, "silu", lambda x: np.maximum(x, 0.0))
    elif mistake == "causal_off":
        def full(q, k, v, q_pos=None):
            n, Hq, hd = q.shape
            G = Hq // k.shape[1]
            out = np.empty_like(q)
            for h in range(Hq):
                s = q[:, h] @ k[:, h // G].T / np.sqrt(hd)
                p = np.exp(s - s.max(1, keepdims=True))
                out[:, h] = (p / p.sum(1, keepdims=True)) @ v[:, h // G]
            return out
        monkeypatch.setattr(oracle, "causal_attention", full)
    got = oracle.forward(shape, 3, tokens, list(range(len(tokens))), mode="exact")
    assert np.abs(got - ref).max() > 1e-3 * np.abs(ref).max()


def test_rms_norm_closed_form():
    # constant vector c: y = c / sqrt(c^2 + eps) in every component
    for c in (0.5, -3.0, 1e-3):
        h = np.full((1, 64), c)
        y = oracle.rms_norm(h, 1e-5)
        np.testing.assert_allclose(y, c / math.sqrt(c * c + 1e-5), rtol=1e-14)


def test_rope_closed_form_and_relative_position():
    shape = workload.TINY  # hd = 64
    rnd = oracle._Rounding(shape, "exact")
    pos = np.arange(40)
    cos, sin = oracle.rope_table(shape, pos, rnd)
    hd = shape.head_dim
    # unit vector on dim i rotates in the (i, i + hd/2) plane by p * theta_i
    for i in (0, 5, hd // 2 - 1):
        x = np.zeros((len(pos), 1, hd))
        x[:, 0, i] = 1.0
        y = oracle.rope(x, cos, sin)[:, 0]
        theta = shape.rope_base ** (-2.0 * i / hd)
        np.testing.assert_allclose(y[:, i], np.cos(pos * theta), atol=1e-14)
        np.testing.assert_allclose(y[:, i + hd // 2], np.sin(pos * theta), atol=1e-14)
    # q(m) . k(n) depends only on m - n
    rng = np.random.default_rng(1)
    q = rng.standard_normal(hd)
    k = rng.standard_normal(hd)
    Q = oracle.rope(np.tile(q, (len(pos), 1, 1)), cos, sin)[:, 0]
    K = oracle.rope(np.tile(k, (len(pos), 1, 1)), cos, sin)[:, 0]
    d1 = Q[10] @ K[3]
    d2 = Q[30] @ K[23]
    assert abs(d1 - d2) < 1e-10 * abs(d1)


def test_contract_mode_is_a_small_perturbation():
    shape = workload.TINY_GQA_BF16
    tokens = workload.random_ids(shape.vocab, 25, 7, 3)
    ex = oracle.forward(shape, 4, tokens, [24], mode="exact")
    ct = oracle.forward(shape, 4, tokens, [24], mode="contract")
    rel = np.abs(ex - ct).max() / np.abs(ex).max()
    assert 0 < rel < 2e-2
