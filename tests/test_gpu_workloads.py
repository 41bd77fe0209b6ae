"""The four bf16 workloads at their real sizes, one decoder layer deep.

Each case builds the workload's model shape with a single decoder layer (full
widths, head layout and vocabulary), prefills the workload's own prefixes (its
batch and prefix lengths, ragged where the workload is) and verifies with its
draft count, probe length, prefix-position count and alpha.  The rows of the
pass and the prefix lengths are those of the full-depth pass, so every matrix,
attention and combine launch has the shape, k-split and key split that the
timed pass uses in each of its layers.  The oracle recomputes sampled
sequences of the batch from scratch (its last layer runs only on the rows it
returns, which keeps a one-layer model at an 8192-token prefix to seconds).

The matrix kernels of the 14B and 70B shapes are also checked on their own,
at the row counts of those workloads, on sampled output columns.
"""
import numpy as np
import pytest

import oracle
import workload
from decisions import greedy_allowed

pytestmark = pytest.mark.gpu

# sequences of each batch that the oracle recomputes
CHECKED = {
    "8b-bf16-b1": lambda lens: [0],
    "8b-bf16-b16-ragged": lambda lens: sorted({int(np.argmin(lens)), int(np.argmax(lens))}),
    "14b-bf16-b4": lambda lens: [2],
    "70b-bf16-b8": lambda lens: [5],
}

OUTS = ("o", "r", "z")


@pytest.mark.parametrize("name,case", [(n, 0) for n in CHECKED] + [("8b-bf16-b1", 1), ("8b-bf16-b16-ragged", 1)])
def test_workload_one_layer_matches_oracle(rv, gpu, name, case):
    import torch
    w = workload.WORKLOADS[name]
    shape = w.shape.with_layers(1)
    lens = [int(x) for x in workload.prefix_lengths(w, case)]
    prefixes = [[int(t) for t in p] for p in workload.prefix_ids(w, lens, case)]
    check = CHECKED[name](lens)
    S = w.rows_per_seq
    print(f"\n{name} case {case}: batch {w.batch}, prefixes {min(lens)}..{max(lens)}, {S} rows per sequence, "
          f"oracle on sequences {check}", flush=True)
    # random drafts; each checked sequence's first draft is the oracle's
    # greedy token after its prefix, so that alpha = 0 accepts it
    drafts = np.stack([workload.random_ids(shape.vocab, w.k, w.index, 7, case, b) for b in range(w.batch)])
    for b in check:
        drafts[b, 0] = int(np.argmax(oracle.forward(shape, w.weight_seed, prefixes[b], [lens[b] - 1])[0]))
    probe = workload.probe_ids(w)

    v = rv.Verifier(shape, w.weight_seed, w.batch, max(lens) + S + 8, max_block=max(64, S),
                    max_drafts=max(16, w.k))
    got = {}
    try:
        v.prefill(prefixes)
        for alpha in (w.alpha, 0.0):
            acc, nxt = v.verify(lens, drafts, probe, alpha, w.prefix_pos)
            torch.cuda.synchronize()
            outs = {key: v.output(wh).cpu().numpy()[check]
                    for key, wh in (("o", rv.RV_OUT_ORIG), ("r", rv.RV_OUT_REFL), ("z", rv.RV_OUT_FUSED),
                                    ("lp_z", rv.RV_OUT_LOGP_FUSED))}
            got[alpha] = (acc.cpu().numpy()[check], nxt.cpu().numpy()[check], outs)
    finally:
        v.close()

    for i, b in enumerate(check):
        ref = oracle.verify(shape, w.weight_seed, prefixes[b], drafts[b], probe, w.alpha, w.prefix_pos)
        # alpha = 0 from the same logits: Eq. 2 reduces to the original distribution
        z0 = oracle.fuse(ref["o"], ref["r"], 0.0).astype(np.float64)
        n0, t0 = oracle.accept_greedy(z0, drafts[b])
        near0 = oracle.decision_margins(z0, drafts[b], n0)[2]
        refs = {w.alpha: (ref["z"], ref["lp_z"], ref["accept_len"], ref["next_id"], ref["near_tie"]),
                0.0: (z0, oracle.log_softmax(z0), n0, t0, near0)}
        for alpha, (z_ref, lp_ref, n_ref, t_ref, near) in refs.items():
            acc, nxt, outs = got[alpha]
            want = {"o": ref["o"], "r": ref["r"], "z": z_ref}
            for key in OUTS:
                err = np.abs(outs[key][i] - want[key])
                rel = (err.max(-1) / np.abs(want[key]).max(-1)).max()
                assert rel <= 2e-2, (name, b, alpha, key, rel)
                # the hi/lo operand contract keeps GPU and oracle far closer than the bar
                assert err.max() < 1e-3, (name, b, alpha, key, float(err.max()))
            assert np.abs(outs["lp_z"][i] - lp_ref).max() < 2e-3, (name, b, alpha)
            if not near:
                assert (int(acc[i]), int(nxt[i])) == (n_ref, t_ref), (name, b, alpha)
            else:
                assert greedy_allowed(z_ref, drafts[b], int(acc[i]), int(nxt[i])), (name, b, alpha)
            if alpha == 0.0 and not near:
                assert int(acc[i]) >= 1, (name, b)


def split_planes(x):
    """bf16 hi/lo planes [2][M][K] of an fp32 matrix, and their exact sum."""
    import torch
    x32 = torch.from_numpy(np.asarray(x, dtype=np.float32))
    hi = x32.to(torch.bfloat16)
    lo = (x32 - hi.float()).to(torch.bfloat16)
    planes = torch.stack([hi, lo]).contiguous()
    exact = hi.double().numpy() + lo.double().numpy()
    return planes, exact


@pytest.fixture(scope="module", params=["14b-bf16-b4", "70b-bf16-b8"])
def wide_model(request, rv, gpu):
    w = workload.WORKLOADS[request.param]
    v = rv.Verifier(w.shape.with_layers(1), 0, w.batch, 128, max_block=64, max_drafts=16)
    yield w, v
    v.close()


@pytest.mark.parametrize("matrix", ["qkv", "o", "gateup", "down", "lm_head"])
def test_matrix_kernel_wide_shapes(rv, wide_model, matrix):
    """Every matrix of the 14B and 70B shapes, at one sequence's block rows
    and at the workload's batch of blocks: 48 sampled output columns against
    the oracle's fp64 dot products with its own weight rows."""
    import torch
    w, v = wide_model
    shape = v.shape
    mat = {"qkv": rv.RV_MAT_QKV, "o": rv.RV_MAT_O, "gateup": rv.RV_MAT_GATEUP, "down": rv.RV_MAT_DOWN,
           "lm_head": rv.RV_MAT_LM_HEAD}[matrix]
    parts = {"qkv": ["q", "k", "v"], "o": ["o"], "gateup": ["gate", "up"], "down": ["down"],
             "lm_head": ["lm_head"]}[matrix]
    K = oracle.tensor_dims(shape, parts[0])[1]
    sizes = [oracle.tensor_dims(shape, p)[0] for p in parts]
    N = sum(sizes)
    for M in (w.rows_per_seq, w.batch * w.rows_per_seq):
        rng = np.random.default_rng([M, K, N])
        x = rng.standard_normal((M, K)).astype(np.float32)
        planes, xe = split_planes(x)
        y = torch.empty((M, N), dtype=torch.float32, device="cuda")
        rv.rv_debug_linear(v.cache, 0, mat, planes.cuda(), y)
        torch.cuda.synchronize()
        got = y.cpu().numpy()
        cols = set(rng.integers(0, N, 40).tolist())
        off = 0
        for p, n in zip(parts, sizes):
            cols.update([off, off + n - 1])
            off += n
        for col in sorted(cols):
            off = 0
            for p, n in zip(parts, sizes):
                if col < off + n:
                    wrow = oracle.weight(shape, 0, 0 if p != "lm_head" else None, p, col - off, 1)[0]
                    break
                off += n
            ref = xe @ wrow
            scale = np.sqrt((xe * xe).sum(1) * (wrow * wrow).sum())
            err = np.abs(got[:, col] - ref)
            assert (err <= 2e-6 * scale + 1e-6).all(), (w.name, matrix, M, col, float((err / scale).max()))
