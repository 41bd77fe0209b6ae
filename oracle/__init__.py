"""CPU oracle for the Reflective Verification verify pass -- TEST INFRASTRUCTURE.

Only tests/, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. It shares no code with the GPU library
and never imports it.

What it computes (arXiv 2505.18629):
  * Section 3.1, Eq. 1 and Algorithm 1: the reflective draft is
    [x_1..x_g, template, x_1..x_g] with template = probe || prefix-position
    tokens, scored in one causal forward pass after the prefix.
  * Algorithm 1: original logits o_1..o_{g+1} and reflective logits
    o_m..o_{m+g} with m = g + |template| + 1.
  * Section 3.2, Eq. 2: p_i = softmax((1 - alpha) * o_i + alpha * r_i).
  * Appendix A, Algorithm 2 (exact-match verification), at temperature 0.
  * Appendix A, Algorithm 3 (entropy-thresholded "typical" acceptance) with
    a greedy bonus token.
  * Algorithm 1 (speculative sampling): uniform acceptance tests against
    p_i / q_i and a draw from norm(max(0, p - q)), with the random numbers
    taken from Philox4x64-10 (Salmon et al., SC 2011) under a fixed counter
    layout, so that the GPU library can draw the same ones.

Because one causal pass produces exactly the next-token logits at every block
position, the oracle is that definition written out: a plain Llama-style
decoder run from scratch over prefix || block (no KV cache), then the rows
Algorithm 1 names are picked out, fused and verified.

Precision modes:
  "exact"    -- fp64 everywhere (used to pin the decoder against a library
                implementation);
  "contract" -- fp64 arithmetic, but values are rounded where the GPU library
                stores them: fp32 for every matmul result and the residual
                stream; and every computed value that is stored for a later
                matmul -- norm outputs, rotated q, the K/V cache, attention
                output, SwiGLU output -- to its operand form.  For bf16
                models the operand form of an fp32 value x is the pair
                hi = bf16(x), lo = bf16(x - hi), about 16 significant bits;
                for fp32 models it is fp32.  The weights are the only bf16
                values.  The remaining GPU-vs-oracle differences are fp32
                accumulation order and the dropped lo*lo products of the
                attention matmuls (relative 2^-16).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, List, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle_weights.so")
_lib = None


def build() -> str:
    """Compile the weight generator (plain C, OpenMP)."""
    src = os.path.join(_HERE, "weights.c")
    cmd = ["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11", src, "-o", _LIB_PATH, "-lm"]
    subprocess.run(cmd, check=True)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        u64, i64, dbl = ctypes.c_uint64, ctypes.c_int64, ctypes.c_double
        vp = ctypes.c_void_p
        lib.orc_fill.argtypes = [u64, u64, u64, u64, ctypes.c_int, dbl, vp]
        lib.orc_fill.restype = None
        lib.orc_bits_at.argtypes = [u64, u64, vp, i64, ctypes.c_int, dbl, vp]
        lib.orc_bits_at.restype = None
        lib.orc_splitmix64_stream.argtypes = [u64, ctypes.c_int, vp]
        lib.orc_splitmix64_stream.restype = None
        lib.orc_round_bf16.argtypes = [vp, vp, i64]
        lib.orc_round_bf16.restype = None
        lib.orc_scale.argtypes = [dbl]
        lib.orc_scale.restype = ctypes.c_float
        _lib = lib
    return _lib


# ---------------------------------------------------------------- weights

TENSOR_NAMES = ("q", "k", "v", "o", "gate", "up", "down")


def tensor_index(shape, layer: int | None, name: str) -> int:
    """Generator tensor numbering: 0 embedding, 1 + 7l + j per layer matrix,
    1 + 7L the LM head."""
    if name == "embed":
        return 0
    if name == "lm_head":
        return 1 + 7 * shape.n_layers
    return 1 + 7 * layer + TENSOR_NAMES.index(name)


def tensor_dims(shape, name: str):
    """Logical [out][in] dims of a weight matrix (y = x @ W.T)."""
    d, hd, F, V = shape.d_model, shape.head_dim, shape.ffn_dim, shape.vocab
    qd, kvd = shape.n_heads * hd, shape.n_kv_heads * hd
    return {
        "embed": (V, d), "lm_head": (V, d),
        "q": (qd, d), "k": (kvd, d), "v": (kvd, d), "o": (d, qd),
        "gate": (F, d), "up": (F, d), "down": (d, F),
    }[name]


def _is_bf16(shape) -> int:
    return 1 if shape.dtype == "bf16" else 0


def fill(shape, seed: int, t: int, start: int, count: int) -> np.ndarray:
    out = np.empty(count, dtype=np.float64)
    _load().orc_fill(seed, t, start, count, _is_bf16(shape), shape.init_std,
                     out.ctypes.data_as(ctypes.c_void_p))
    return out


def weight(shape, seed: int, layer: int | None, name: str, row0: int = 0, nrows: int | None = None) -> np.ndarray:
    """Rows [row0, row0 + nrows) of a logical weight matrix, as fp64."""
    n_out, n_in = tensor_dims(shape, name)
    if nrows is None:
        nrows = n_out - row0
    t = tensor_index(shape, layer, name)
    return fill(shape, seed, t, row0 * n_in, nrows * n_in).reshape(nrows, n_in)


def weight_bits(shape, seed: int, layer: int | None, name: str, flat_idx: np.ndarray) -> np.ndarray:
    """Stored bit patterns (bf16 in the low 16 bits, or fp32) at flat logical indices."""
    idx = np.ascontiguousarray(flat_idx, dtype=np.uint64)
    out = np.empty(len(idx), dtype=np.uint32)
    _load().orc_bits_at(seed, tensor_index(shape, layer, name), idx.ctypes.data_as(ctypes.c_void_p),
                        len(idx), _is_bf16(shape), shape.init_std, out.ctypes.data_as(ctypes.c_void_p))
    return out


def embedding_rows(shape, seed: int, tokens: Sequence[int]) -> np.ndarray:
    d = shape.d_model
    out = np.empty((len(tokens), d), dtype=np.float64)
    cache: Dict[int, np.ndarray] = {}
    for j, tok in enumerate(tokens):
        tok = int(tok)
        if tok not in cache:
            cache[tok] = fill(shape, seed, 0, tok * d, d)
        out[j] = cache[tok]
    return out


def splitmix64_stream(seed: int, n: int) -> List[int]:
    out = np.empty(n, dtype=np.uint64)
    _load().orc_splitmix64_stream(seed, n, out.ctypes.data_as(ctypes.c_void_p))
    return [int(v) for v in out]


# ---------------------------------------------------------------- rounding

def round_f32(x: np.ndarray) -> np.ndarray:
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round through fp32 to bf16, nearest-even at each step."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty_like(x)
    _load().orc_round_bf16(x.ctypes.data_as(ctypes.c_void_p), out.ctypes.data_as(ctypes.c_void_p), x.size)
    return out


def split_bf16(x: np.ndarray) -> np.ndarray:
    """hi + lo with x32 = fp32(x), hi = bf16(x32), lo = bf16(x32 - hi).
    x32 - hi is exact in fp32, so the pair is a function of x32 alone."""
    x32 = round_f32(x)
    hi = round_bf16(x32)
    return hi + round_bf16(x32 - hi)


class _Rounding:
    def __init__(self, shape, mode: str):
        if mode not in ("exact", "contract"):
            raise ValueError(mode)
        self.exact = mode == "exact"
        self.bf16 = shape.dtype == "bf16"

    def f32(self, x):
        return x if self.exact else round_f32(x)

    def kv(self, x):
        """K/V cache storage: the operand form (bf16 hi/lo pair, or fp32)."""
        return self.operand(x)

    def operand(self, x):
        """Matmul operand form of an activation: bf16 hi/lo pair or fp32."""
        if self.exact:
            return x
        return split_bf16(x) if self.bf16 else round_f32(x)


# ---------------------------------------------------------------- decoder

def rms_norm(h: np.ndarray, eps: float) -> np.ndarray:
    """y = h / sqrt(mean(h^2) + eps) * g, with gains g = 1 at init."""
    return h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + eps)


def rope_table(shape, positions: np.ndarray, rnd: _Rounding):
    """cos/sin of p * base^(-2i/hd), i < hd/2, evaluated in fp64; the contract
    stores the table in fp32."""
    hd = shape.head_dim
    i = np.arange(hd // 2, dtype=np.float64)
    theta = shape.rope_base ** (-2.0 * i / hd)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * theta[None, :]
    return rnd.f32(np.cos(ang)), rnd.f32(np.sin(ang))


def rope(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """Rotate-half rotary embedding: dims (i, i + hd/2) rotate by angle_i.
    x is [n][heads][hd]; cos/sin are [n][hd/2]."""
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, q_pos=None, rows_per_chunk: int = 1024) -> np.ndarray:
    """Softmax(q k^T / sqrt(hd)) v where the query at position j attends keys
    0..j; q head h reads kv head h // (Hq / Hkv).  q [m][Hq][hd] holds the
    queries at positions q_pos (default 0..m-1), k/v [n][Hkv][hd] the keys at
    positions 0..n-1.  Queries are taken rows_per_chunk at a time (each
    query's softmax is independent of the others), and a chunk only forms
    scores against the keys its latest query may see; the mask then removes
    the later keys of the chunk's earlier queries."""
    m, Hq, hd = q.shape
    group = Hq // k.shape[1]
    q_pos = np.arange(m) if q_pos is None else np.asarray(q_pos, dtype=np.int64)
    out = np.empty_like(q)
    for r0 in range(0, m, rows_per_chunk):
        r1 = min(m, r0 + rows_per_chunk)
        qp = q_pos[r0:r1]
        nk = int(qp.max()) + 1
        mask = np.arange(nk)[None, :] > qp[:, None]
        for h in range(Hq):
            kv = h // group
            s = (q[r0:r1, h, :] @ k[:nk, kv, :].T) / np.sqrt(hd)
            s[mask] = -np.inf
            s -= s.max(axis=1, keepdims=True)
            np.exp(s, out=s)
            s /= s.sum(axis=1, keepdims=True)
            out[r0:r1, h, :] = s @ v[:nk, kv, :]
    return out


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def _matmul_wT(shape, seed, layer, name, a, rnd: _Rounding, chunk_rows: int = 16384):
    """a @ W.T, W generated in row chunks to bound memory; fp32-rounded in the contract."""
    n_out, _ = tensor_dims(shape, name)
    if a.shape[0] == 0:
        return np.zeros((0, n_out))
    if n_out <= chunk_rows:
        return rnd.f32(a @ weight(shape, seed, layer, name).T)
    parts = []
    for r0 in range(0, n_out, chunk_rows):
        nr = min(chunk_rows, n_out - r0)
        parts.append(a @ weight(shape, seed, layer, name, r0, nr).T)
    return rnd.f32(np.concatenate(parts, axis=1))


def forward(shape, seed: int, tokens: Sequence[int], rows: Sequence[int], mode: str = "contract",
            return_kv: bool = False, past=None, trace=None):
    """Next-token logits at the given rows of `tokens`.

    Without `past` the tokens sit at positions 0..n-1 and everything is
    computed from scratch.  With past = (ks, vs), the per-layer K and V of the
    tokens at positions 0..p-1 as returned by an earlier call, the tokens sit
    at positions p..p+n-1 and attend those cached keys and values before their
    own (the same causal computation, with the earlier positions' K and V
    taken from where they were first computed).

    Returns logits [len(rows)][V] (fp64 holding fp32 values in the contract
    mode) and, if asked, the per-layer K and V of `tokens` [L][n][Hkv][hd] as
    the GPU stores them (post-rotary, storage form).  `trace`, if a dict,
    receives each layer's stored intermediates (for tests of the rounding
    contract)."""
    rnd = _Rounding(shape, mode)
    tokens = np.asarray(tokens, dtype=np.int64)
    n = len(tokens)
    p0 = 0 if past is None else past[0].shape[1]
    Hq, Hkv, hd = shape.n_heads, shape.n_kv_heads, shape.head_dim
    cos, sin = rope_table(shape, p0 + np.arange(n), rnd)
    h = embedding_rows(shape, seed, tokens)
    rows = np.asarray(rows, dtype=np.int64)
    ks, vs = [], []
    for l in range(shape.n_layers):
        # Only `rows` of the last layer's output are read, and under the causal
        # mask a row's output depends on its own query and the keys and values
        # at or before it; so that layer projects K and V for every token and
        # runs the rest (query, attention, o-proj, MLP) on `rows` alone.
        sel = rows if l == shape.n_layers - 1 else np.arange(n)
        a = rnd.operand(rms_norm(h, shape.rms_eps))
        q = _matmul_wT(shape, seed, l, "q", a[sel], rnd).reshape(len(sel), Hq, hd)
        k = _matmul_wT(shape, seed, l, "k", a, rnd).reshape(n, Hkv, hd)
        v = _matmul_wT(shape, seed, l, "v", a, rnd).reshape(n, Hkv, hd)
        q = rnd.operand(rope(q, cos[sel], sin[sel]))
        k = rnd.kv(rope(k, cos, sin))
        v = rnd.kv(v)
        if return_kv:
            ks.append(k)
            vs.append(v)
        kk = k if past is None else np.concatenate([past[0][l], k])
        vv = v if past is None else np.concatenate([past[1][l], v])
        att = rnd.operand(causal_attention(q, kk, vv, p0 + sel).reshape(len(sel), Hq * hd))
        if trace is not None:
            trace.setdefault("norm_in", []).append(a)
            trace.setdefault("q", []).append(q)
            trace.setdefault("k", []).append(k)
            trace.setdefault("v", []).append(v)
            trace.setdefault("att", []).append(att)
        o = _matmul_wT(shape, seed, l, "o", att, rnd)
        h = rnd.f32(h[sel] + o)
        a = rnd.operand(rms_norm(h, shape.rms_eps))
        g = _matmul_wT(shape, seed, l, "gate", a, rnd)
        u = _matmul_wT(shape, seed, l, "up", a, rnd)
        act = rnd.operand(silu(g) * u)
        dn = _matmul_wT(shape, seed, l, "down", act, rnd)
        if trace is not None:
            trace.setdefault("o_proj", []).append(o)
            trace.setdefault("resid_mid", []).append(h)
            trace.setdefault("ffn_in", []).append(a)
            trace.setdefault("gate", []).append(g)
            trace.setdefault("up", []).append(u)
            trace.setdefault("act", []).append(act)
            trace.setdefault("down", []).append(dn)
        h = rnd.f32(h + dn)
        if trace is not None:
            trace.setdefault("resid", []).append(h)
    if shape.n_layers == 0:
        h = h[rows]
    a = rnd.operand(rms_norm(h, shape.rms_eps))
    logits = _matmul_wT(shape, seed, None, "lm_head", a, rnd)
    if trace is not None:
        trace["final_in"] = a
        trace["logits"] = logits
    if return_kv:
        return logits, np.stack(ks), np.stack(vs)
    return logits


def prefix_kv(shape, seed: int, tokens: Sequence[int], mode: str = "contract"):
    """Per-layer K and V of `tokens` at positions 0..n-1 (the cache a verify
    of the next block attends), computed from scratch."""
    _, ks, vs = forward(shape, seed, tokens, [], mode, return_kv=True)
    return ks, vs


def extend_kv(past, ks, vs):
    """past (K, V at positions 0..p-1) followed by K, V of the next tokens."""
    if past is None:
        return ks, vs
    return np.concatenate([past[0], ks], axis=1), np.concatenate([past[1], vs], axis=1)


# ---------------------------------------------------------------- the method

def reflective_block(history: Sequence[int], drafts: Sequence[int], probe: Sequence[int], prefix_pos: int):
    """Block scored by one verify pass (Eq. 1; Algorithm 1).

    Row 0 is the last committed token c = history[-1], whose KV is not cached
    yet (it was emitted as the previous step's bonus token); it yields o_1.
    The reflective draft [x, probe, history[-P:], x] follows.  shift is the
    number of tokens of the probe, the prefix-position part and the first draft
    copy (Eq. 2's shift_len), so r_i sits at block row shift + i - 1.
    """
    L, k, P = len(history), len(drafts), prefix_pos
    if P > L:
        raise ValueError("prefix_pos exceeds the committed length")
    template = list(probe) + (list(history[L - P:]) if P > 0 else [])
    block = [int(history[-1])] + list(drafts) + template + list(drafts)
    shift = k + len(template)
    orig_rows = list(range(k + 1))
    refl_rows = [shift + i for i in range(k + 1)]
    return [int(t) for t in block], shift, orig_rows, refl_rows


def fuse(o: np.ndarray, r: np.ndarray, alpha: float) -> np.ndarray:
    """Eq. 2's fused logits, in fp32: (1 - alpha) * o + alpha * r."""
    a = np.float32(alpha)
    return (np.float32(1.0) - a) * np.asarray(o, np.float32) + a * np.asarray(r, np.float32)


def log_softmax(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    m = x.max(axis=-1, keepdims=True)
    return x - (m + np.log(np.exp(x - m).sum(axis=-1, keepdims=True)))


def accept_greedy(z: np.ndarray, drafts: Sequence[int]):
    """Algorithm 2 at temperature 0: x_hat_i = argmax p_i (lowest id on ties);
    n = number of leading drafts equal to x_hat; t = argmax p_{n+1}."""
    k = len(drafts)
    xhat = np.argmax(z, axis=-1)
    n = k
    for i in range(k):
        if int(xhat[i]) != int(drafts[i]):
            n = i
            break
    return n, int(xhat[n])


def decision_margins(z: np.ndarray, drafts: Sequence[int], n: int, tie_eps: float = 1e-3):
    """Distance of each decision on the accept path from its boundary, in
    fused-logit units: z_i[x_i] - max_{v != x_i} z_i[v] for the drafts that
    were tested, and top1 - top2 of z_{n+1} for the bonus token."""
    k = len(drafts)
    ms = []
    for i in range(min(n + 1, k)):
        zi = np.asarray(z[i], dtype=np.float64)
        x = int(drafts[i])
        others = np.delete(zi, x)
        ms.append(float(zi[x] - others.max()))
    top = np.sort(np.asarray(z[n], dtype=np.float64))[-2:]
    gap = float(top[1] - top[0])
    near = any(abs(m) < tie_eps for m in ms) or gap < tie_eps
    return ms, gap, near


def entropy(logits: np.ndarray) -> np.ndarray:
    """Shannon entropy in nats of softmax(logits) per row, fp64:
    H = -sum_v p_v log p_v, with 0 log 0 = 0 (ids whose logit is -inf)."""
    lp = log_softmax(logits)
    p = np.exp(lp)
    with np.errstate(invalid="ignore"):
        return -np.where(p > 0, p * lp, 0.0).sum(-1)


def accept_typical(z: np.ndarray, o: np.ndarray, drafts: Sequence[int], eps: float, delta: float,
                   entropy_of: str = "fused"):
    """Entropy-thresholded acceptance of Algorithm 3 with a greedy bonus token.

    p_i = softmax(z_i) is the fused distribution (Eq. 2).  The threshold is
    min(eps, delta * exp(-H)), with H the entropy of p_i (entropy_of="fused")
    or of the original target distribution softmax(o_i) ("original").  Draft
    i is accepted while p_i(x_i) exceeds its threshold (the printed rejection
    set has the comparison reversed; acceptance of the tokens the target finds
    plausible is what the rule is for); n counts the leading accepted drafts
    and t = argmax z_{n+1} (lowest id on ties).  Compared in the log domain:
    log p_i(x_i) > min(log eps, log delta - H), which keeps eps = inf and
    delta = 0 exact.  Returns n, t and the log-domain margins of the tested
    drafts."""
    k = len(drafts)
    lpz = log_softmax(z)
    H = entropy(z if entropy_of == "fused" else o)
    with np.errstate(divide="ignore"):
        log_eps, log_delta = np.log(np.float64(eps)), np.log(np.float64(delta))
    n, margins = k, []
    for i in range(k):
        thr = min(log_eps, log_delta - H[i])
        m = float(lpz[i][int(drafts[i])] - thr)
        margins.append(m)
        if not m > 0:
            n = i
            break
    t = int(np.argmax(z[n]))
    return n, t, margins


# ------------------------------------------------------------ randomness
# Philox4x64-10: a 10-round counter-based generator; each round multiplies
# counter words 0 and 2 by fixed odd constants (full 128-bit products), mixes
# the high halves with the other words and the key, and the key is advanced by
# two Weyl constants between rounds.
_PHILOX_M = (0xD2E7470EE14C6C93, 0xCA5A826395121157)
_PHILOX_W = (0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B)
_M64 = (1 << 64) - 1


def philox4x64(counter: Sequence[int], key: Sequence[int]) -> List[int]:
    c = [int(x) & _M64 for x in counter]
    k0, k1 = int(key[0]) & _M64, int(key[1]) & _M64
    for rnd in range(10):
        p0, p1 = _PHILOX_M[0] * c[0], _PHILOX_M[1] * c[2]
        c = [((p1 >> 64) ^ c[1] ^ k0) & _M64, p1 & _M64, ((p0 >> 64) ^ c[3] ^ k1) & _M64, p0 & _M64]
        if rnd < 9:
            k0, k1 = (k0 + _PHILOX_W[0]) & _M64, (k1 + _PHILOX_W[1]) & _M64
    return c


def uniform24(word: int) -> float:
    """The top 23 bits of a 64-bit word as a uniform in (0, 1): (w >> 41) + 1/2
    over 2^23, whose odd 24-bit numerator makes it exact in fp32 and fp64."""
    return ((int(word) >> 41) + 0.5) / float(1 << 23)


def acceptance_uniform(seed: int, seq: int, i: int) -> float:
    """r_i of sequence slot `seq` (Algorithm 1): word 0 of Philox at counter
    (i, seq, 0, 0), key (seed, 0)."""
    return uniform24(philox4x64((i, seq, 0, 0), (seed, 0))[0])


def gumbel_uniforms(seed: int, seq: int, V: int) -> np.ndarray:
    """One uniform per vocabulary id v for the bonus-token draw: word v % 4 of
    Philox at counter (v // 4, seq, 1, 0), key (seed, 0)."""
    u = np.empty(V, dtype=np.float64)
    for blk in range((V + 3) // 4):
        words = philox4x64((blk, seq, 1, 0), (seed, 0))
        for j in range(4):
            if 4 * blk + j < V:
                u[4 * blk + j] = uniform24(words[j])
    return u


def accept_sampling(z: np.ndarray, q: np.ndarray, drafts: Sequence[int], seed: int, seq: int,
                    tie_eps: float = 1e-3):
    """Algorithm 1's speculative-sampling rule on the fused distribution
    p_i = softmax(z_i) (z already divided by the temperature).

    Draft i is rejected when r_i > p_i(x_i) / q_i(x_i), compared as
    r_i * q_i(x_i) > p_i(x_i); n = leading accepted drafts.  The bonus token
    is drawn from norm(max(0, p_{n+1} - q_{n+1})) if n < k, else from
    p_{k+1}, as argmax_v (log w_v + G_v) with w the unnormalised weights and
    G_v = -log(-log(u_v)) Gumbel noise (the Gumbel-max form of a categorical
    draw; normalisation does not change the argmax).  Returns n, t, the
    log-domain acceptance margins log p - log(r q) of the tested drafts,
    the top-1 minus top-2 gap of the perturbed scores, and a near-tie flag."""
    k = len(drafts)
    lp = log_softmax(z)
    n, margins = k, []
    for i in range(k):
        x = int(drafts[i])
        r = acceptance_uniform(seed, seq, i)
        p_x, q_x = float(np.exp(lp[i][x])), float(q[i][x])
        m = np.inf if q_x <= 0 else float(np.log(p_x) - np.log(r * q_x))
        margins.append(m)
        if r * q_x > p_x:
            n = i
            break
    if n < k:
        w = np.exp(lp[n]) - np.asarray(q[n], dtype=np.float64)
        with np.errstate(divide="ignore"):
            score = np.where(w > 0, np.log(np.maximum(w, 1e-300)), -np.inf)
    else:
        score = lp[k]
    u = gumbel_uniforms(seed, seq, z.shape[-1])
    s = score - np.log(-np.log(u))
    t = int(np.argmax(s))
    top = np.sort(s)[-2:]
    gap = float(top[1] - top[0])
    near = any(abs(m) < tie_eps for m in margins) or gap < tie_eps
    return n, t, margins, gap, near


def verify(shape, seed: int, history: Sequence[int], drafts: Sequence[int], probe: Sequence[int],
           alpha: float, prefix_pos: int, mode: str = "contract", rule: str = "greedy", eps: float = 0.09,
           delta: float = 0.3, entropy_of: str = "fused", tie_eps: float = 1e-3, temperature: float = 1.0,
           q: np.ndarray | None = None, rng_seed: int = 0, slot: int = 0, past=None) -> Dict:
    """One verify step for one sequence: Algorithm 1's block with Algorithm
    2's rule (rule="greedy"), Algorithm 3's (rule="typical") or Algorithm 1's
    speculative sampling (rule="sampling", draft distributions q [k][V],
    random numbers from (rng_seed, batch slot `slot`)).  The fused logits are divided by
    the temperature (fp32) before any rule.  `past`, if given, is
    prefix_kv(history[:-1]): the block then attends it instead of the prefix
    being recomputed."""
    history = [int(t) for t in history]
    drafts = [int(t) for t in drafts]
    block, shift, orig_rows, refl_rows = reflective_block(history, drafts, probe, prefix_pos)
    base = len(history) - 1
    if past is None:
        seq = history[:-1] + block
        rows = [base + j for j in orig_rows] + [base + j for j in refl_rows]
        logits = forward(shape, seed, seq, rows, mode)
    else:
        if past[0].shape[1] != base:
            raise ValueError("past must hold the K/V of history[:-1]")
        logits = forward(shape, seed, block, orig_rows + refl_rows, mode, past=past)
    k = len(drafts)
    o, r = logits[: k + 1], logits[k + 1:]
    z = fuse(o, r, alpha)
    if temperature != 1.0:
        z = (z.astype(np.float32) / np.float32(temperature)).astype(np.float32)
    if rule == "sampling":
        n, t, ms, gap, near = accept_sampling(z.astype(np.float64), q, drafts, rng_seed, slot, tie_eps)
    elif rule == "greedy":
        n, t = accept_greedy(z, drafts)
        ms, gap, near = decision_margins(z, drafts, n, tie_eps)
    elif rule == "typical":
        n, t, ms = accept_typical(z, o, drafts, eps, delta, entropy_of)
        top = np.sort(np.asarray(z[n], dtype=np.float64))[-2:]
        gap = float(top[1] - top[0])
        near = any(abs(m) < tie_eps for m in ms) or gap < tie_eps
    else:
        raise ValueError(f"unknown rule {rule}")
    return {
        "block": block, "shift": shift, "o": o, "r": r, "z": z.astype(np.float64),
        "lp_o": log_softmax(o), "lp_r": log_softmax(r), "lp_z": log_softmax(z),
        "h_z": entropy(z), "h_o": entropy(o),
        "accept_len": n, "next_id": t, "margins": ms, "gap": gap, "near_tie": near,
    }


def greedy_continuation(shape, seed: int, history: Sequence[int], n_tokens: int, mode: str = "contract",
                        past=None) -> List[int]:
    """Target's own greedy continuation (used to build realistic drafts).
    Without `past` every token is recomputed from scratch over the whole
    sequence; with past = prefix_kv(history[:-1]) each step runs one token on
    top of the growing K/V of the earlier ones."""
    seq = [int(t) for t in history]
    out = []
    for _ in range(n_tokens):
        if past is None:
            logits = forward(shape, seed, seq, [len(seq) - 1], mode)
        else:
            logits, ks, vs = forward(shape, seed, seq[-1:], [0], mode, return_kv=True, past=past)
            past = extend_kv(past, ks, vs)
        t = int(np.argmax(logits[0]))
        out.append(t)
        seq.append(t)
    return out
