"""Every benchmark workload at its full depth against the CPU oracle (GPU).

The bf16 workloads (8B at batch 1 and batch 16 ragged, 14B at batch 4, 70B
at batch 8) are compared with the oracle's results stored in
tests/golden/fulldepth_<workload>.json, which tests/golden/make_fulldepth.py
writes from the oracle alone (the 70B pass takes the oracle hours, too long
to repeat here).  The model, prefixes, probe and drafts are the workload's
own (the drafts of the checked sequences are the oracle's greedy
continuation with the workload's random replacements; the other sequences'
drafts are random ids that only complete the batch).  The GPU pass is the
one bench.py times: the whole model, the whole batch.

Checked for each stored sequence, at alpha = 0.3 and at alpha = 0 (the
latter decided from the same o and r rows, where Eq. 2 gives z = o):
* o, r and z at the stored ids (a fixed sample plus the drafts): per row,
  max |diff| / max |ref| <= 2e-2, and the measured max |diff| is printed;
* log-softmax of z at those ids, the entropies, the decision margins;
* accept_len and next_id equal to the oracle's; where the oracle flags a
  near-tie (a margin within 1e-3), the GPU's decision must be one the
  oracle's fused rows allow: every accepted draft within 1e-3 of its row's
  maximum, a rejected draft not more than 1e-3 above every other id, and
  next_id within 1e-3 of its row's maximum.

The tiny fp32 workload is compared with the oracle live, every logit.
"""
import glob
import json
import os

import numpy as np
import pytest

import oracle
import workload

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
FIXTURES = sorted(glob.glob(os.path.join(HERE, "golden", "fulldepth_*.json")),
                  key=lambda p: ["8b-bf16-b1", "8b-bf16-b16-ragged", "14b-bf16-b4", "70b-bf16-b8"].index(
                      json.load(open(p))["workload"]))
BF16_REL = 2e-2
TIE = 1e-3


def _value(row, key, v):
    """Oracle value of id v in a stored row (sampled ids, drafts, top list)."""
    ids = row["ids"]
    j = np.searchsorted(ids, v)
    if j < len(ids) and ids[j] == v:
        return row[key][j]
    top_ids, top_vals = row["top_" + key]
    if v in top_ids:
        return top_vals[top_ids.index(v)]
    return None


def decision_allowed(rows, key, drafts, n, t):
    """Whether (n, t) is a correct decision for some fused rows within TIE of
    the oracle's (key "z", or "o" at alpha = 0)."""
    k = len(drafts)
    if not 0 <= n <= k:
        return False
    for i in range(n):
        top1 = rows[i]["top_" + key][1][0]
        if _value(rows[i], key, drafts[i]) < top1 - TIE:
            return False
    if n < k:
        x = drafts[n]
        zx = _value(rows[n], key, x)
        others = [val for tid, val in zip(*rows[n]["top_" + key]) if tid != x]
        if max(others) < zx - TIE or t == x:
            return False
    zt = _value(rows[n], key, t)
    return zt is not None and zt >= rows[n]["top_" + key][1][0] - TIE


def _free(v):
    """Closes the handles and drops the device buffers (the 70B model holds
    141 GB), so the next model fits."""
    import torch
    v.close()
    v.model_buf = v.cache_buf = v._keep = v._keep2 = None
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("path", FIXTURES, ids=lambda p: os.path.basename(p)[10:-5])
def test_full_depth_matches_oracle(rv, gpu, path):
    import torch
    with open(path) as f:
        fx = json.load(f)
    w = workload.WORKLOADS[fx["workload"]]
    shape = w.shape
    assert fx["layers"] == shape.n_layers and fx["k"] == w.k and fx["n_probe"] == w.n_probe
    probe = workload.probe_ids(w)
    S = w.rows_per_seq
    max_len = max(max(c["prefix_len"]) for c in fx["cases"]) + S + 8
    v = rv.Verifier(shape, w.weight_seed, w.batch, max_len, max_block=max(64, S), max_drafts=max(16, w.k))
    report = []
    try:
        for case in fx["cases"]:
            lens = [int(x) for x in workload.prefix_lengths(w, case["case"])]
            assert lens == case["prefix_len"]
            prefixes = [[int(t) for t in p] for p in workload.prefix_ids(w, lens, case["case"])]
            drafts = np.array(case["drafts"], dtype=np.int32)
            print(f"\n{w.name} case {case['case']}: {shape.n_layers} layers, batch {w.batch}, prefixes "
                  f"{min(lens)}..{max(lens)}, sequences {[s['seq'] for s in case['sequences']]}", flush=True)
            v.prefill(prefixes)
            got = {}
            for alpha in (w.alpha, 0.0):
                acc, nxt = v.verify(lens, drafts, probe, alpha, w.prefix_pos)
                torch.cuda.synchronize()
                got[alpha] = (acc.cpu().numpy().copy(), nxt.cpu().numpy().copy(),
                              {wh: v.output(wh).cpu().numpy() for wh in range(8)})
            for sq in case["sequences"]:
                b = sq["seq"]
                for alpha, dec_key, key in ((w.alpha, "alpha", "z"), (0.0, "alpha0", "o")):
                    acc, nxt, out = got[alpha]
                    dec = sq[dec_key]
                    worst = {}
                    for i, row in enumerate(sq["rows"]):
                        ids = row["ids"]
                        for name, wh in (("o", rv.RV_OUT_ORIG), ("r", rv.RV_OUT_REFL), ("z", rv.RV_OUT_FUSED)):
                            ref = np.asarray(row[name if (name != "z" or alpha != 0.0) else "o"])
                            err = float(np.abs(out[wh][b][i][ids] - ref).max())
                            scale = row["max_abs"][name if (name != "z" or alpha != 0.0) else "o"]
                            assert err <= BF16_REL * scale, (w.name, b, alpha, name, i, err, scale)
                            worst[name] = max(worst.get(name, 0.0), err)
                        if alpha != 0.0:
                            err = float(np.abs(out[rv.RV_OUT_LOGP_FUSED][b][i][ids] - np.asarray(row["lp_z"])).max())
                            assert err <= BF16_REL * row["max_abs"]["z"], (w.name, b, "lp_z", i, err)
                            worst["lp_z"] = max(worst.get("lp_z", 0.0), err)
                            for j, hk in ((0, "h_z"), (1, "h_o")):
                                assert abs(out[rv.RV_OUT_ENTROPY][j][b][i] - row[hk]) <= BF16_REL * max(1, row[hk])
                    n, t = int(acc[b]), int(nxt[b])
                    if not dec["near_tie"]:
                        assert (n, t) == (dec["accept_len"], dec["next_id"]), (w.name, b, alpha, dec)
                        mg = out[rv.RV_OUT_MARGINS][b]
                        np.testing.assert_allclose(mg[:len(dec["margins"])], dec["margins"], atol=5e-2)
                    assert decision_allowed(sq["rows"], key, sq["drafts"], n, t), (w.name, b, alpha, n, t, dec)
                    report.append(f"{w.name} case {case['case']} seq {b} alpha {alpha}: n={n} t={t} "
                                  f"(oracle {dec['accept_len']}, {dec['next_id']}, near-tie {dec['near_tie']}) "
                                  + " ".join(f"max|d{kk}|={vv:.2e}" for kk, vv in worst.items()))
                # the greedy drafts up to the first replacement are accepted at alpha = 0
                lead = next((i for i, (g, x) in enumerate(zip(sq["greedy"], sq["drafts"])) if g != x), w.k)
                if not sq["alpha0"]["near_tie"]:
                    assert int(got[0.0][0][b]) == min(lead, w.k)
    finally:
        _free(v)
    print("\n" + "\n".join(report), flush=True)


def test_tiny_workload_matches_oracle(rv, gpu):
    """The tiny fp32 workload as bench.py builds it: every logit (1e-4) and
    the decisions."""
    import torch
    w = workload.WORKLOADS["tiny-f32-b1"]
    shape = w.shape
    lens = [int(x) for x in workload.prefix_lengths(w)]
    prefix = [int(t) for t in workload.prefix_ids(w, lens)[0]]
    greedy = oracle.greedy_continuation(shape, w.weight_seed, prefix, w.k)
    ps = workload.replace_probs(w)
    drafts = [int(t) for t in workload.corrupt(greedy, ps[0], shape.vocab, workload.draft_rng(w, 0, 0))]
    probe = workload.probe_ids(w)
    v = rv.Verifier(shape, w.weight_seed, 1, lens[0] + w.rows_per_seq + 8, max_block=64, max_drafts=16)
    v.prefill([prefix])
    for alpha in (w.alpha, 0.0):
        acc, nxt = v.verify(lens, np.array([drafts]), probe, alpha, w.prefix_pos)
        torch.cuda.synchronize()
        ref = oracle.verify(shape, w.weight_seed, prefix, drafts, probe, alpha, w.prefix_pos)
        for key, wh in (("o", rv.RV_OUT_ORIG), ("r", rv.RV_OUT_REFL), ("z", rv.RV_OUT_FUSED)):
            assert np.abs(v.output(wh).cpu().numpy()[0] - ref[key]).max() <= 1e-4, (alpha, key)
        if not ref["near_tie"]:
            assert (int(acc[0]), int(nxt[0])) == (ref["accept_len"], ref["next_id"]), alpha
    _free(v)
