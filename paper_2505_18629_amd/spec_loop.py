"""Speculative decoding loop over the C ABI.

A draft model proposes k tokens, one decode step each; the target scores
them in one reflective verification pass (Eq. 1) and keeps the accepted
prefix plus one token, under the rule of Algorithm 2 (greedy), 3 (typical)
or 1 (speculative sampling).  Both models are `Verifier` handles of this
package (seeded random-init weights).

A draft decode step is a verify call on the draft cache with k = 0, no
probe and P = 0: its single block row scores the last committed token and
the returned token is the draft's next proposal (its argmax, or with the
sampling rule a draw from its distribution, whose probabilities become
q_i).  Each draft step writes the KV of its block row, i.e. of the
token before its proposal, so after k steps the draft cache holds KV up to
x_{k-1}.  If a sequence accepts all k drafts, one more draft step at length
L + k computes the KV of x_k (its proposal is discarded).  Then
rv_commit_tokens writes the target's emitted token into the draft history
at L + n; the draft KV below that position holds the accepted tokens, and
later calls overwrite the rest.  One host synchronisation per round reads n (prefix lengths are host
inputs of every call).
"""
from __future__ import annotations

import time
from typing import List, Sequence

import numpy as np


class SpeculativeLoop:
    def __init__(self, rv, target, draft, k: int, probe: Sequence[int], alpha: float, prefix_pos: int,
                 rule: str = "greedy", temperature: float = 1.0, seed: int = 0, epsilon: float = 0.09,
                 delta: float = 0.3, entropy_src: int = 0):
        import torch
        if target.batch != draft.batch or target.shape.vocab != draft.shape.vocab:
            raise ValueError("target and draft need the same batch and vocabulary")
        if rule not in ("greedy", "typical", "sampling"):
            raise ValueError(f"unknown rule {rule}")
        self.rv, self.torch = rv, torch
        self.target, self.draft = target, draft
        self.k, self.alpha, self.P = k, alpha, prefix_pos
        self.rule, self.T, self.seed = rule, temperature, seed
        self.eps, self.delta, self.entropy_src = epsilon, delta, entropy_src
        self.probe = np.asarray(probe, dtype=np.int32)
        self.d_probe = torch.from_numpy(self.probe).cuda() if len(self.probe) else None
        B, V = target.batch, target.shape.vocab
        self.d_drafts = torch.zeros((B, max(k, 1)), dtype=torch.int32, device="cuda")
        self.d_q = torch.zeros((B, max(k, 1), V), dtype=torch.float32, device="cuda") if rule == "sampling" else None
        self.d_p = torch.empty((B, V), dtype=torch.float32, device="cuda") if rule == "sampling" else None
        self.rounds = 0
        self.accepted: List[int] = []

    def prefill(self, prefixes: Sequence[Sequence[int]]):
        self.lens = self.target.prefill(prefixes)
        self.draft.prefill(prefixes)
        self.tokens = [list(map(int, p)) for p in prefixes]
        return self.lens

    def _round_seed(self, j: int) -> int:
        return ((self.seed & 0xFFFFFFFF) << 32) | ((self.rounds * (self.k + 1) + j) & 0xFFFFFFFF)

    def round(self) -> np.ndarray:
        """One draft-then-verify round; returns the accepted draft count per sequence."""
        rv, torch, dr, tg = self.rv, self.torch, self.draft, self.target
        k = self.k
        lens_d = list(self.lens)
        for j in range(k):
            if self.rule == "sampling":
                rv.rv_verify_sampled(dr.cache, lens_d, None, 0, None, None, 0, 0.0, 0, self._round_seed(j),
                                     dr.accept_len, dr.next_id, temperature=self.T)
                # the draft's distribution of its proposal, p = softmax(z), as the library emits it
                rv.rv_debug_output(dr.cache, rv.RV_OUT_PROB_FUSED, self.d_p)
                self.d_q[:, j].copy_(self.d_p)
            else:
                rv.rv_verify(dr.cache, lens_d, None, 0, None, 0, 0.0, 0, dr.accept_len, dr.next_id,
                             temperature=self.T)
            self.d_drafts[:, j].copy_(dr.next_id)
            lens_d = [x + 1 for x in lens_d]
        drafts = self.d_drafts[:, :k].contiguous()
        if self.rule == "sampling":
            rv.rv_verify_sampled(tg.cache, self.lens, drafts, k, self.d_q[:, :k].contiguous(), self.d_probe,
                                 len(self.probe), self.alpha, self.P, self._round_seed(k), tg.accept_len,
                                 tg.next_id, temperature=self.T)
        else:
            rule = rv.RV_RULE_GREEDY if self.rule == "greedy" else rv.RV_RULE_TYPICAL
            rv.rv_verify(tg.cache, self.lens, drafts, k, self.d_probe, len(self.probe), self.alpha, self.P,
                         tg.accept_len, tg.next_id, rule=rule, epsilon=self.eps, delta=self.delta,
                         entropy_src=self.entropy_src, temperature=self.T)
        n = tg.accept_len.cpu().numpy().astype(np.int64)
        if (n < 0).any():
            raise RuntimeError("out-of-range token id in a verify block")
        if k > 0 and (n == k).any():
            # KV of x_k in the draft cache (harmless past the accepted prefix elsewhere)
            rv.rv_verify(dr.cache, lens_d, None, 0, None, 0, 0.0, 0, dr.accept_len, dr.next_id,
                         temperature=self.T)
        # the draft history takes the target's emitted token at L + n
        rv.rv_commit_tokens(dr.cache, [int(L + m) for L, m in zip(self.lens, n)], tg.next_id)
        t = tg.next_id.cpu().numpy()
        d = drafts.cpu().numpy()
        for b in range(tg.batch):
            self.tokens[b] += [int(x) for x in d[b, :n[b]]] + [int(t[b])]
            self.lens[b] += int(n[b]) + 1
        self.rounds += 1
        self.accepted += n.tolist()
        return n

    def generate(self, n_tokens: int):
        """Rounds until every sequence has n_tokens new tokens; returns the
        new tokens per sequence and the wall time."""
        start = [len(t) for t in self.tokens]
        t0 = time.perf_counter()
        while min(len(t) - s for t, s in zip(self.tokens, start)) < n_tokens:
            self.round()
        self.torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        return [t[s:s + n_tokens] for t, s in zip(self.tokens, start)], wall
