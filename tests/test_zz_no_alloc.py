"""rv_fuse_accept_noalloc (the no-allocation variant of rv_debug_fuse_accept)
against rv_debug_fuse_accept through the C ABI (GPU): the same accept_len
and next_id, bit for bit, on two calls in a row, the second smaller than the
first, and on the rule and edge cases the variant keeps (ties, typical rule,
out-of-range drafts).  Its limits are enforced before anything runs."""
import numpy as np
import pytest

import workload

pytestmark = pytest.mark.gpu

SHAPE = workload.ModelShape("head-v8192", 1, 128, 4, 4, 32, 128, 8192, "f32")


@pytest.fixture(scope="module")
def ref(rv, gpu):
    v = rv.Verifier(SHAPE, 0, 4, 64, max_block=8, max_drafts=8)
    yield v
    v.close()


def logits_for(B, k, seed):
    rng = np.random.default_rng(seed)
    o = (rng.standard_normal((B, k + 1, SHAPE.vocab)) * 2).astype(np.float32)
    r = (rng.standard_normal((B, k + 1, SHAPE.vocab)) * 2).astype(np.float32)
    drafts = rng.integers(0, SHAPE.vocab, (B, k)).astype(np.int32)
    # sequence 0 drafts its original argmaxes (accepted at alpha = 0), and a
    # tie across vocabulary chunks decides its bonus token
    drafts[0] = np.argmax(o[0][:k], -1)
    o[0, k, [5000, 300]] = 20.0
    return o, r, drafts


def run_both(rv, v, o, r, drafts, alpha, **kw):
    import torch
    B, k1, V = o.shape
    logits = torch.from_numpy(np.ascontiguousarray(np.concatenate([o, r], axis=1))).cuda()
    d = torch.from_numpy(np.ascontiguousarray(drafts)).cuda() if k1 > 1 else None
    n1 = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    t1 = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    rv.rv_fuse_accept_noalloc(logits, k1 - 1, d, alpha, n1, t1, **kw)
    torch.cuda.synchronize()
    got = (n1.cpu().numpy().copy(), t1.cpu().numpy().copy())
    # the existing entry point on the same logits (its cache holds 4 sequences)
    n2 = torch.zeros(4, dtype=torch.int32, device="cuda")
    t2 = torch.zeros(4, dtype=torch.int32, device="cuda")
    pad = 4 - B
    if pad:
        logits = torch.cat([logits, logits[:1].expand(pad, -1, -1)], 0).contiguous()
        d = torch.cat([d, d[:1].expand(pad, -1)], 0).contiguous() if d is not None else None
    rv.rv_debug_fuse_accept(v.cache, logits, [10] * 4, d, k1 - 1, alpha, n2, t2, **kw)
    torch.cuda.synchronize()
    want = (n2.cpu().numpy()[:B].copy(), t2.cpu().numpy()[:B].copy())
    return got, want


@pytest.mark.parametrize("alpha", [0.0, 0.3])
def test_two_calls_in_a_row_match_the_cache_entry_point(rv, ref, alpha):
    o, r, drafts = logits_for(4, 6, 1)
    got, want = run_both(rv, ref, o, r, drafts, alpha)
    np.testing.assert_array_equal(got[0], want[0])
    np.testing.assert_array_equal(got[1], want[1])
    if alpha == 0.0:
        assert (int(got[0][0]), int(got[1][0])) == (6, 300)
    # second call, smaller (fewer sequences, fewer drafts, other values): the
    # statistics left by the first call must not leak into it
    o, r, drafts = logits_for(2, 3, 2)
    got, want = run_both(rv, ref, o, r, drafts, alpha)
    np.testing.assert_array_equal(got[0], want[0])
    np.testing.assert_array_equal(got[1], want[1])


def test_typical_rule_and_out_of_range_drafts(rv, ref):
    o, r, drafts = logits_for(3, 4, 3)
    drafts[2, 1] = SHAPE.vocab + 3
    kw = dict(rule=rv.RV_RULE_TYPICAL, epsilon=0.2, delta=0.5)
    got, want = run_both(rv, ref, o, r, drafts, 0.3, **kw)
    np.testing.assert_array_equal(got[0], want[0])
    np.testing.assert_array_equal(got[1], want[1])
    assert (int(got[0][2]), int(got[1][2])) == (-1, -1)
    # k = 0: one decode decision
    got, want = run_both(rv, ref, o[:, :1], r[:, :1], drafts[:, :0], 0.5)
    np.testing.assert_array_equal(got[1], want[1])


def test_limits_are_checked_before_any_work(rv, ref):
    import torch
    n = torch.zeros(256, dtype=torch.int32, device="cuda")
    t = torch.zeros(256, dtype=torch.int32, device="cuda")
    # 256 x 33 rows x 63 chunks exceeds the scratch: rejected, outputs untouched
    big = torch.zeros((256, 2, 128256), dtype=torch.float32, device="cuda")
    d = torch.zeros((256, 32), dtype=torch.int32, device="cuda")
    with pytest.raises(rv.RVError) as e:
        rv._check(rv._lib.rv_fuse_accept_noalloc(big.data_ptr(), 256, 32, 128256, d.data_ptr(),
                                                 rv.ctypes.byref(rv.rv_fusion(0.3, 0, 0, 0.1, 0.1, 0, 1.0)),
                                                 n.data_ptr(), t.data_ptr(), None))
    assert e.value.name == "RV_E_CAPACITY"
    with pytest.raises(rv.RVError) as e:
        rv.rv_fuse_accept_noalloc(big[:2], 0, None, 0.3, n, t, rule=rv.RV_RULE_SAMPLING)
    assert e.value.name == "RV_E_ARG"
    torch.cuda.synchronize()
    assert int(n.abs().sum()) == 0 and int(t.abs().sum()) == 0
