"""Seeded synthetic workloads: model shapes and token-id inputs.

This module holds no arithmetic of the method. It only describes model shapes
and draws token ids, prefix lengths and replacement masks from seeded numpy
generators, so that the GPU library and the CPU oracle receive identical
inputs. The paper evaluates trained Llama-3 targets on MT-Bench, GSM8K and
HumanEval (Section 4.1); none of those are available, so random-init models
of the same shapes and uniform-random token ids stand in for them. The verify
pass costs the same for any token contents, so the stand-in is faithful for
timing; parity is checked on these same inputs.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import List, Sequence

import numpy as np


@dataclass(frozen=True)
class ModelShape:
    """Llama-style decoder shape (pre-norm RMSNorm, rotary, GQA, SwiGLU,
    untied LM head). dtype is the storage type of weights and KV cache."""

    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    dtype: str  # "f32" or "bf16"
    rms_eps: float = 1e-5
    rope_base: float = 10000.0
    init_std: float = 0.02

    def with_layers(self, n_layers: int) -> "ModelShape":
        return replace(self, name=f"{self.name}-{n_layers}L", n_layers=n_layers)


TINY = ModelShape("tiny", 2, 256, 4, 4, 64, 1024, 4096, "f32")
LLAMA8B = ModelShape("llama3-8b", 32, 4096, 32, 8, 128, 14336, 128256, "bf16")
# the 1B draft paired with the 8B target (Section 4.1): Llama-3.2-1B's shape
LLAMA1B = ModelShape("llama3-1b", 16, 2048, 32, 8, 64, 8192, 128256, "bf16")
QWEN14B = ModelShape("14b", 48, 5120, 40, 8, 128, 13824, 152064, "bf16")
LLAMA70B = ModelShape("llama3-70b", 80, 8192, 64, 8, 128, 28672, 128256, "bf16")
# small bf16 shape with GQA for quick parity cases
TINY_GQA_BF16 = ModelShape("tiny-gqa-bf16", 2, 256, 8, 2, 32, 768, 4096, "bf16")


@dataclass(frozen=True)
class Workload:
    """One benchmark/parity configuration of the verify pass."""

    name: str
    index: int              # seed namespace
    shape: ModelShape
    batch: int
    prefix_lo: int          # prefix length L_b drawn uniformly in [lo, hi]
    prefix_hi: int
    k: int                  # draft length (gamma)
    n_probe: int            # reflective-probe length |R|
    p_lo: float             # per-sequence replacement probability in [p_lo, p_hi]
    p_hi: float
    alpha: float = 0.3      # Table 5
    prefix_pos: int = 4     # Table 5 "Prefix Len"
    weight_seed: int = 0

    @property
    def rows_per_seq(self) -> int:
        return 1 + 2 * self.k + self.n_probe + self.prefix_pos


WORKLOADS = {
    w.name: w
    for w in [
        Workload("tiny-f32-b1", 0, TINY, 1, 128, 128, 4, 8, 0.3, 0.3),
        Workload("8b-bf16-b1", 1, LLAMA8B, 1, 1024, 1024, 5, 16, 0.3, 0.3),
        Workload("8b-bf16-b16-ragged", 2, LLAMA8B, 16, 512, 4096, 5, 16, 0.1, 0.5),
        Workload("14b-bf16-b4", 3, QWEN14B, 4, 2048, 2048, 7, 24, 0.3, 0.3),
        Workload("70b-bf16-b8", 4, LLAMA70B, 8, 8192, 8192, 8, 24, 0.3, 0.3),
    ]
}


def rng(*key: int) -> np.random.Generator:
    return np.random.default_rng(list(key))


def probe_ids(w: Workload) -> np.ndarray:
    """Fixed random reflective-probe ids for a workload (stands in for a
    tokenised reflection prompt, Table 2)."""
    return rng(w.index, 0xBEEF).integers(0, w.shape.vocab, size=w.n_probe, dtype=np.int64).astype(np.int32)


def prefix_lengths(w: Workload, case: int = 0) -> np.ndarray:
    g = rng(w.index, case, 1)
    return g.integers(w.prefix_lo, w.prefix_hi + 1, size=w.batch).astype(np.int32)


def prefix_ids(w: Workload, lengths: Sequence[int], case: int = 0) -> List[np.ndarray]:
    g = rng(w.index, case, 2)
    return [g.integers(0, w.shape.vocab, size=int(L)).astype(np.int32) for L in lengths]


def replace_probs(w: Workload, case: int = 0) -> np.ndarray:
    g = rng(w.index, case, 3)
    return g.uniform(w.p_lo, w.p_hi, size=w.batch)


def corrupt(tokens: Sequence[int], p: float, vocab: int, g: np.random.Generator) -> np.ndarray:
    """Replace each token independently with probability p by a uniform id."""
    t = np.asarray(tokens, dtype=np.int32).copy()
    mask = g.random(len(t)) < p
    t[mask] = g.integers(0, vocab, size=int(mask.sum())).astype(np.int32)
    return t


def draft_rng(w: Workload, case: int, b: int) -> np.random.Generator:
    return rng(w.index, case, 4, b)


def random_ids(vocab: int, n: int, *key: int) -> np.ndarray:
    return rng(*key).integers(0, vocab, size=n).astype(np.int32)
