"""The speculative decoding loop (draft proposes, target verifies) over the C ABI."""
import numpy as np
import pytest

import oracle
import workload

pytestmark = pytest.mark.gpu


def make_loop(rv, draft_seed, rule="greedy", alpha=0.0, k=4, seed=0, T=1.0, batch=1):
    from paper_2505_18629_amd.spec_loop import SpeculativeLoop
    shape = workload.TINY
    tgt = rv.Verifier(shape, 0, batch, 200, max_block=32, max_drafts=k)
    drf = rv.Verifier(shape, draft_seed, batch, 200, max_block=32, max_drafts=k)
    probe = workload.random_ids(shape.vocab, 5, 8, 0xBEEF)
    return SpeculativeLoop(rv, tgt, drf, k, probe, alpha, 4, rule=rule, temperature=T, seed=seed), tgt, drf


def test_greedy_loop_is_lossless(rv, gpu):
    """At alpha = 0 the greedy rule keeps exactly the target's greedy
    decoding, whatever the draft proposes."""
    loop, tgt, drf = make_loop(rv, draft_seed=5)
    prefix = [int(t) for t in workload.random_ids(workload.TINY.vocab, 40, 8, 1)]
    loop.prefill([prefix])
    toks, _ = loop.generate(20)
    ref = oracle.greedy_continuation(workload.TINY, 0, prefix, 20)
    assert toks[0] == ref
    tgt.close(), drf.close()


def test_self_draft_accepts_every_draft(rv, gpu):
    import torch
    loop, tgt, drf = make_loop(rv, draft_seed=0, k=3, batch=2)
    prefixes = [[int(t) for t in workload.random_ids(workload.TINY.vocab, L, 8, 2 + L)] for L in (30, 44)]
    loop.prefill(prefixes)
    for _ in range(4):
        n = loop.round()
        assert (n == 3).all()
    # the draft history holds what the target committed
    for b in range(2):
        L = loop.lens[b]
        a = torch.empty(L, dtype=torch.int32, device="cuda")
        c = torch.empty(L, dtype=torch.int32, device="cuda")
        rv.rv_debug_export_ids(tgt.cache, b, 0, L, a)
        rv.rv_debug_export_ids(drf.cache, b, 0, L, c)
        torch.cuda.synchronize()
        assert a.cpu().tolist() == c.cpu().tolist() == loop.tokens[b]
    tgt.close(), drf.close()


@pytest.mark.parametrize("rule", ["sampling", "typical"])
def test_loop_is_a_function_of_its_seed(rv, gpu, rule):
    prefix = [int(t) for t in workload.random_ids(workload.TINY.vocab, 33, 8, 3)]
    outs = []
    for _ in range(2):
        loop, tgt, drf = make_loop(rv, draft_seed=9, rule=rule, alpha=0.3, seed=42, T=0.7)
        loop.prefill([prefix])
        toks, _ = loop.generate(12)
        assert all(0 <= t < workload.TINY.vocab for t in toks[0])
        outs.append(toks[0])
        tgt.close(), drf.close()
    assert outs[0] == outs[1]
