#!/usr/bin/env python3
"""Writes tests/golden/fulldepth_<workload>.json: the CPU oracle's results
for verify passes of the benchmark workloads at their full depth.

Only the oracle (oracle/) and the seeded input generators (workload/) are
used; nothing here touches the GPU library.  For each checked sequence the
oracle computes the prefix K/V from scratch (oracle.prefix_kv), the model's
own greedy continuation of k tokens on top of it, replaces each token with
probability p by a uniform id (the drafts of the workload, Section 4.1 /
Table 5 settings), and runs one verify (Eq. 1 block, Algorithm 1 rows,
Eq. 2 fusion, Algorithm 2 at temperature 0).  Sequences that are not
checked get uniform-random drafts; they only complete the batch.

A full row of the vocabulary is too large to store for every case, so each
row keeps: the largest |value| of o, r and z; o, r, z and log-softmax(z) at
a fixed sample of ids (the same ids for every row of the file) plus the
draft ids; the 16 largest fused logits (and original logits, for the alpha
= 0 decision) with their ids; the entropies; the decisions and margins.

Usage: python tests/golden/make_fulldepth.py [--only-missing] [--ckpt DIR] [WORKLOAD ...]
(--ckpt: compute each prefix in chunks kept in DIR, so that an interrupted run
resumes; the 70B prefix takes hours on a few host cores)
"""
from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import workload  # noqa: E402

# (case, checked sequences, drafts) per workload: "workload" drafts are the
# greedy continuation with the workload's random replacements, "greedy" ones
# the continuation itself (every draft acceptable at alpha = 0).  The tiny
# fp32 workload is checked live against the oracle instead (it takes a
# second).
PLAN = {
    "8b-bf16-b1": [(0, "all", "workload"), (1, "all", "workload"), (0, "all", "greedy")],
    "8b-bf16-b16-ragged": [(0, "short+long", "workload"), (0, [8], "greedy")],
    "14b-bf16-b4": [(0, [0, 3], "workload"), (0, [0], "greedy")],
    "70b-bf16-b8": [(0, [5], "workload"), (0, [5], "greedy")],
}
N_SAMPLE = 512
TOP = 16


def f9(x):
    return [float(f"{v:.9g}") for v in np.asarray(x, dtype=np.float64).ravel()]


def checked_sequences(spec, lens):
    if spec == "all":
        return list(range(len(lens)))
    if spec == "short+long":
        return sorted({int(np.argmin(lens)), int(np.argmax(lens))})
    return list(spec)


def top_list(row, n=TOP):
    row = np.asarray(row, dtype=np.float64)
    idx = np.argsort(-row, kind="stable")[:n]
    return [int(i) for i in idx], f9(row[idx])


CHUNK = 1024


def prefix_kv(shape, seed, tokens, ckpt_dir=None, tag=""):
    """The oracle's prefix K/V.  With ckpt_dir the prefix is computed in
    chunks of CHUNK tokens, each chunk attending the K/V of those before it
    (oracle.forward with past: the same causal computation), and every
    chunk's K/V is kept in ckpt_dir, so an interrupted run resumes at the
    first chunk not on disk."""
    if not ckpt_dir:
        return oracle.prefix_kv(shape, seed, tokens)
    os.makedirs(ckpt_dir, exist_ok=True)
    past = None
    for c0 in range(0, len(tokens), CHUNK):
        path = os.path.join(ckpt_dir, f"{tag}_{c0}_{len(tokens)}.npz")
        if os.path.exists(path):
            with np.load(path) as z:
                ks, vs = z["k"], z["v"]
        else:
            _, ks, vs = oracle.forward(shape, seed, tokens[c0:c0 + CHUNK], [], return_kv=True, past=past)
            np.savez(path + ".tmp.npz", k=ks, v=vs)
            os.replace(path + ".tmp.npz", path)
        past = oracle.extend_kv(past, ks, vs)
        print(f"    prefix chunk {c0}..{min(c0 + CHUNK, len(tokens)) - 1} of {len(tokens)}", flush=True)
    return past


def run_case(w, case, spec, rule, cols, ckpt_dir=None):
    shape = w.shape
    lens = [int(x) for x in workload.prefix_lengths(w, case)]
    prefixes = [[int(t) for t in p] for p in workload.prefix_ids(w, lens, case)]
    probe = workload.probe_ids(w)
    ps = workload.replace_probs(w, case)
    check = checked_sequences(spec, lens)
    drafts = [[int(t) for t in workload.random_ids(shape.vocab, w.k, w.index, 7, case, b)] for b in range(w.batch)]
    seqs = []
    for b in check:
        t0 = time.time()
        past = prefix_kv(shape, w.weight_seed, prefixes[b][:-1], ckpt_dir, f"{w.name}_c{case}_s{b}")
        t1 = time.time()
        greedy = oracle.greedy_continuation(shape, w.weight_seed, prefixes[b], w.k, past=past)
        if rule == "greedy":
            drafts[b] = [int(t) for t in greedy]
        else:
            drafts[b] = [int(t) for t in workload.corrupt(greedy, ps[b], shape.vocab,
                                                          workload.draft_rng(w, case, b))]
        ref = oracle.verify(shape, w.weight_seed, prefixes[b], drafts[b], probe, w.alpha, w.prefix_pos, past=past)
        t2 = time.time()
        # alpha = 0 from the same rows: Eq. 2 reduces to the original logits
        z0 = oracle.fuse(ref["o"], ref["r"], 0.0).astype(np.float64)
        n0, t0_ = oracle.accept_greedy(z0, drafts[b])
        m0, g0, near0 = oracle.decision_margins(z0, drafts[b], n0)
        rows = []
        for i in range(w.k + 1):
            ids = sorted(set(cols) | set(drafts[b]))
            rows.append({
                "ids": ids,
                "o": f9(ref["o"][i][ids]), "r": f9(ref["r"][i][ids]), "z": f9(ref["z"][i][ids]),
                "lp_z": f9(ref["lp_z"][i][ids]),
                "max_abs": {key: float(np.abs(ref[key][i]).max()) for key in ("o", "r", "z")},
                "top_z": top_list(ref["z"][i]), "top_o": top_list(ref["o"][i]),
                "h_z": float(ref["h_z"][i]), "h_o": float(ref["h_o"][i]),
            })
        seqs.append({
            "seq": b, "prefix_len": lens[b], "greedy": greedy, "drafts": drafts[b], "rows": rows,
            "alpha": {"accept_len": ref["accept_len"], "next_id": ref["next_id"], "margins": ref["margins"],
                      "gap": ref["gap"], "near_tie": bool(ref["near_tie"])},
            "alpha0": {"accept_len": n0, "next_id": t0_, "margins": m0, "gap": g0, "near_tie": bool(near0)},
            "oracle_seconds": {"prefix": round(t1 - t0, 1), "greedy_and_verify": round(t2 - t1, 1)},
        })
        print(f"  {w.name} case {case} seq {b}: L={lens[b]} n={ref['accept_len']} t={ref['next_id']} "
              f"alpha0 n={n0} near={ref['near_tie']}/{near0} ({t1 - t0:.0f}+{t2 - t1:.0f} s)", flush=True)
    return {"case": case, "drafts_rule": rule, "prefix_len": lens, "drafts": drafts, "sequences": seqs}


def main(names, only_missing=False, ckpt_dir=None):
    """Writes each workload's file; with only_missing, keeps the cases an
    existing file already holds and computes the others."""
    for name in names:
        w = workload.WORKLOADS[name]
        cols = sorted(set(np.random.default_rng([w.index, 0x5EED]).integers(0, w.shape.vocab, N_SAMPLE).tolist()))
        path = os.path.join(os.path.dirname(os.path.abspath(__file__)), f"fulldepth_{name}.json")
        have = {}
        if only_missing and os.path.exists(path):
            with open(path) as f:
                have = {(c["case"], c.get("drafts_rule", "workload")): c for c in json.load(f)["cases"]}
        out = {
            "source": ("CPU oracle (oracle/), contract mode, full depth; inputs from workload/ with the seeds "
                       "named by workload and case. Written by tests/golden/make_fulldepth.py."),
            "workload": name, "layers": w.shape.n_layers, "alpha": w.alpha, "prefix_pos": w.prefix_pos,
            "k": w.k, "n_probe": w.n_probe, "cases": [],
        }
        for case, spec, rule in PLAN[name]:
            if (case, rule) in have:
                c = have[(case, rule)]
                c["drafts_rule"] = rule
                out["cases"].append(c)
            else:
                out["cases"].append(run_case(w, case, spec, rule, cols, ckpt_dir))
        with open(path, "w") as f:
            json.dump(out, f, separators=(",", ":"))
        print(f"wrote {path} ({os.path.getsize(path) / 1e3:.0f} kB)", flush=True)


if __name__ == "__main__":
    args = sys.argv[1:]
    missing = "--only-missing" in args
    ckpt = None
    if "--ckpt" in args:
        i = args.index("--ckpt")
        ckpt = args[i + 1]
        del args[i:i + 2]
    args = [a for a in args if a != "--only-missing"]
    main(args or list(PLAN), missing, ckpt)
