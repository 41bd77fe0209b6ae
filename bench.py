#!/usr/bin/env python3
"""Throughput of the Reflective Verification verify pass on one MI355X.

One step = one rv_verify call: the whole pass (block assembly, all decoder
layers over the block against the KV cache, LM head on the 2(k+1) rows per
sequence, fusion, log-softmax, accept and commit).  Inputs and the cache are
resident in HBM before the timed region; repeated calls are idempotent, so
the same step is timed K times.

Default workload: the 8B-shaped bf16 model (32 layers, d 4096, 32/8 heads x
128, FFN 14336, vocab 128256), batch 1, prefix 1024, k = 5 drafts from the
model's own greedy continuation with random replacement p = 0.3, probe of 16
ids, prefix-position length 4, alpha = 0.3.  Weights are seeded random-init
(the paper's trained targets are not available); cost depends only on shapes.

Prints one JSON line.  See --help for options.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def traffic_model(shape, lens, S, k):
    """Bytes one verify step must move.  Algorithmic (what the method needs,
    the weights in their storage type and the KV cache at one element of that
    type): every layer matrix and the LM head streamed once, the KV of the
    prefix read once, the block's KV written.  This library also stores a lo
    plane beside every bf16 KV element and matmul operand (the hi/lo
    precision contract); those extra bytes are reported beside it."""
    d, hd, F, V, L = shape.d_model, shape.head_dim, shape.ffn_dim, shape.vocab, shape.n_layers
    qd, kvd = shape.n_heads * hd, shape.n_kv_heads * hd
    w = 2 if shape.dtype == "bf16" else 4
    layer_w = (d * (qd + 2 * kvd) + qd * d + 2 * F * d + F * d) * w
    weights = L * layer_w + V * d * w
    kv_row = 2 * kvd * w * L
    kv_read = sum(int(x) - 1 for x in lens) * kv_row
    kv_write = len(lens) * S * kv_row
    M = len(lens) * S
    # matmul operands written and read once per layer (norm outputs twice, q,
    # attention output, SwiGLU output), LM-head operands
    act_elems = L * M * (2 * d + 2 * qd + F) + len(lens) * 2 * (k + 1) * d
    lo = 2 if shape.dtype == "bf16" else 0
    return {"algorithmic": weights + kv_read + kv_write, "weights": weights, "kv_read": kv_read,
            "kv_write": kv_write, "kv_lo_planes": (kv_read + kv_write) * lo // w if lo else 0,
            "operands": act_elems * 4}


def algorithmic_bytes(shape, lens, S, k):
    return traffic_model(shape, lens, S, k)["algorithmic"]


def algorithmic_flops(shape, lens, S, k):
    """Matmul flops of the layers over B*S rows, the LM head over the 2(k+1)
    rows per sequence, and attention (QK^T and PV) over the cached prefix
    plus the causal block."""
    d, hd, F, V, L = shape.d_model, shape.head_dim, shape.ffn_dim, shape.vocab, shape.n_layers
    qd, kvd = shape.n_heads * hd, shape.n_kv_heads * hd
    layer_params = d * (qd + 2 * kvd) + qd * d + 3 * F * d
    B = len(lens)
    flops = 2 * layer_params * B * S * L + 2 * V * d * B * 2 * (k + 1)
    flops += sum(4 * S * qd * ((int(x) - 1) + (S + 1) / 2) for x in lens) * L
    return flops


def gateup_bytes(shape, M):
    """Algorithmic bytes of one gate/up launch: its weights, streamed once
    (the few-kB activations are not counted, as in the step's bytes)."""
    d, F = shape.d_model, shape.ffn_dim
    return 2 * F * d * (2 if shape.dtype == "bf16" else 4)


MFMA_PEAK_TFLOPS = 2500.0  # dense bf16
RIDGE_FLOP_PER_BYTE = MFMA_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)


def gateup_flops(shape, M):
    """Algorithmic flops of one gate/up launch (2 per multiply-add)."""
    return 2 * M * 2 * shape.ffn_dim * shape.d_model


def calibrate_copy(nbytes=1 << 30, reps=3):
    """A plain device copy of known size, for scaling rocprofv3's FETCH_SIZE
    and WRITE_SIZE counters to bytes (run under the profiler)."""
    import torch
    x = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    x.fill_(1)
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    for _ in range(reps):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"calibration_copy_bytes": nbytes, "reps": reps}), flush=True)


def e2e_bench(args):
    """End-to-end speculative decoding (the loop in paper_2505_18629_amd.spec_loop):
    the 1B-shaped draft proposes k tokens one decode step at a time, the 8B target
    verifies them in one reflective pass.  Both are random-init, so the draft
    rarely matches the target: the figure is a timing of the loop, not of the
    paper's acceptance rates (those need trained weights)."""
    import torch
    import paper_2505_18629_amd as rv
    import workload as wl
    from paper_2505_18629_amd.spec_loop import SpeculativeLoop
    w = wl.WORKLOADS["8b-bf16-b1"]
    lens = wl.prefix_lengths(w)
    prefix = [int(t) for t in wl.prefix_ids(w, lens)[0]]
    max_len = len(prefix) + (args.steps + args.warmup + 2) * (w.k + 1) + w.rows_per_seq + 8
    tgt = rv.Verifier(w.shape, w.weight_seed, 1, max_len, max_block=max(64, w.rows_per_seq), max_drafts=w.k)
    drf = rv.Verifier(wl.LLAMA1B, 1, 1, max_len, max_block=8, max_drafts=w.k)
    loop = SpeculativeLoop(rv, tgt, drf, w.k, wl.probe_ids(w), w.alpha, w.prefix_pos)
    loop.prefill([prefix])
    for _ in range(args.warmup):
        loop.round()
    torch.cuda.synchronize()
    n0, r0 = len(loop.tokens[0]), loop.rounds
    t0 = time.perf_counter()
    for _ in range(args.steps):
        loop.round()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    toks = len(loop.tokens[0]) - n0
    print(json.dumps({
        "metric": "end-to-end tokens/s (speculative loop, 1B-shaped draft + 8B-shaped target)",
        "value": toks / wall, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_round": wall * 1e3 / args.steps, "higher_is_better": True, "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded random-init weights and token ids)",
        "config": {"workload": "8b-bf16-b1 target + llama3-1b-shaped draft", "k": w.k, "alpha": w.alpha,
                   "rule": "greedy", "prefix_len": len(prefix)},
        "mean_accepted": float(np.mean(loop.accepted[r0:])), "tokens": toks,
    }), flush=True)
    tgt.close()
    drf.close()


def source_hash(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def traffic_from_profiles(kernel_src):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if
    it was taken on the current kernel source; else None."""
    p = os.path.join(ROOT, "profiles", "gateup_8b_b1_counters.json")
    if not os.path.exists(p):
        return None
    try:
        rec = json.load(open(p))
    except Exception:
        return None
    if rec.get("kernel_source_sha256_16") != source_hash(kernel_src):
        return None
    return rec.get("hbm_bytes_per_launch")


def stored_parity(rv, v, w, lens, drafts):
    """The timed step's decisions and sampled logits against the oracle's
    stored results for the same inputs (tests/golden/fulldepth_<workload>.json,
    written by tests/golden/make_fulldepth.py from the oracle alone), when the
    file exists and holds these drafts: the GPU's greedy continuation and the
    oracle's agree unless a near-tie decided one of them differently."""
    path = os.path.join(ROOT, "tests", "golden", f"fulldepth_{w.name}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        fx = json.load(f)
    case = next((c for c in fx["cases"] if c["case"] == 0 and c.get("drafts_rule", "workload") == "workload"), None)
    if case is None or case["prefix_len"] != list(lens):
        return None
    acc = v.accept_len.cpu().numpy()
    nxt = v.next_id.cpu().numpy()
    z = v.output(rv.RV_OUT_FUSED).cpu().numpy()
    checked, equal, near, worst = 0, 0, 0, 0.0
    for sq in case["sequences"]:
        b = sq["seq"]
        if [int(x) for x in drafts[b]] != sq["drafts"]:
            continue
        checked += 1
        dec = sq["alpha"]
        near += bool(dec["near_tie"])
        equal += (int(acc[b]), int(nxt[b])) == (dec["accept_len"], dec["next_id"])
        for i, row in enumerate(sq["rows"]):
            worst = max(worst, float(np.abs(z[b][i][row["ids"]] - np.asarray(row["z"])).max()))
    return {"reference": os.path.relpath(path, ROOT), "sequences_checked": checked,
            "decisions_equal": equal, "oracle_near_ties": near, "max_abs_dz_sampled": worst}


def build_state(rv, w, case=0):
    import torch
    import workload as wl
    shape = w.shape
    lens = wl.prefix_lengths(w, case)
    prefixes = wl.prefix_ids(w, lens, case)
    S = w.rows_per_seq
    max_len = int(max(lens)) + S + w.k + 8
    v = rv.Verifier(shape, w.weight_seed, w.batch, max_len, max_block=max(64, S), max_drafts=max(16, w.k))
    v.prefill([list(map(int, p)) for p in prefixes])
    # the target's own greedy continuation, one single-row verify per token
    greedy = np.zeros((w.batch, w.k), dtype=np.int32)
    cur = [int(x) for x in lens]
    empty = np.zeros((w.batch, 0), dtype=np.int32)
    for j in range(w.k):
        _, nxt = v.verify(cur, empty, [], 0.0, 0)
        greedy[:, j] = nxt.cpu().numpy()
        cur = [c + 1 for c in cur]
    ps = wl.replace_probs(w, case)
    drafts = np.stack([wl.corrupt(greedy[b], ps[b], shape.vocab, wl.draft_rng(w, case, b)) for b in range(w.batch)])
    probe = wl.probe_ids(w)
    torch.cuda.synchronize()
    return v, [int(x) for x in lens], drafts, probe


def cpu_baseline(w, lens, drafts, probe, layers=12):
    """The CPU oracle on a bounded sample of the same step: the from-scratch
    forward over prefix + block for `layers` of the model's layers plus the LM
    head on the 2(k+1) rows, fusion and accept, for sequence 0; the layer time
    is scaled to the full depth."""
    import oracle
    import workload as wl
    shape = w.shape
    sample = shape.with_layers(layers)
    prefix = [int(t) for t in wl.prefix_ids(w, lens, 0)[0]]
    t0 = time.perf_counter()
    oracle.verify(sample, w.weight_seed, prefix, drafts[0], probe, w.alpha, w.prefix_pos)
    t_sample = time.perf_counter() - t0
    # a second run with one layer: the oracle runs every layer but the last
    # over all rows, the last (like the LM head) only on the block rows it
    # returns, so L layers cost t_one + (L - 1) * (t_sample - t_one) / (layers - 1)
    one = shape.with_layers(1)
    t0 = time.perf_counter()
    oracle.verify(one, w.weight_seed, prefix, drafts[0], probe, w.alpha, w.prefix_pos)
    t_one = time.perf_counter() - t0
    per_layer = max(t_sample - t_one, 1e-9) / (layers - 1)
    t_step = t_one + per_layer * (shape.n_layers - 1)
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    try:
        from threadpoolctl import threadpool_info
        info = threadpool_info()
        if info:
            threads = max(i.get("num_threads", 0) for i in info)
    except Exception:
        pass
    return {
        "value": 1.0 / (t_step * w.batch),  # the oracle verifies one sequence at a time
        "unit": "verify steps/s",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"sequence 0 of the workload: from-scratch fp64 forward over its {lens[0]}-token prefix + "
                   f"{w.rows_per_seq}-row block with {layers} and 1 of {shape.n_layers} layers plus LM head, fusion "
                   f"and accept; per-layer time scaled to {shape.n_layers} layers (measured {t_sample + t_one:.1f} s)"),
        "seconds_per_step_est": t_step,
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="8b-bf16-b1")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-steps", type=int, default=5)
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a 1 GiB device copy (counter calibration under rocprofv3)")
    ap.add_argument("--e2e", action="store_true",
                    help="time the end-to-end speculative loop (1B-shaped draft + 8B-shaped target) instead")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (the verify pass would shard by "
              "sequence across data-parallel replicas, with no communication inside a pass). Run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.e2e:
        e2e_bench(args)
        return

    import torch
    import paper_2505_18629_amd as rv
    import workload as wl

    w = wl.WORKLOADS[args.workload]
    shape = w.shape
    print(f"[bench] workload {w.name}: building model and cache", file=sys.stderr, flush=True)
    v, lens, drafts, probe = build_state(rv, w)
    S = w.rows_per_seq
    d_dr = torch.from_numpy(np.ascontiguousarray(drafts.astype(np.int32))).cuda()
    d_pr = torch.from_numpy(probe.astype(np.int32)).cuda() if len(probe) else None
    stream = torch.cuda.current_stream()

    def step():
        rv.rv_verify(v.cache, lens, d_dr, w.k, d_pr, len(probe), w.alpha, w.prefix_pos, v.accept_len, v.next_id,
                     stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print(f"[bench] warmup done ({args.warmup} steps)", file=sys.stderr, flush=True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms = e0.elapsed_time(e1) / args.steps
    print(f"[bench] timed {args.steps} steps: {ms:.3f} ms/step", file=sys.stderr, flush=True)
    accept = v.accept_len.cpu().numpy().tolist()

    # per-kernel-class durations from HIP events on the same stream
    rv.rv_debug_profile(v.cache, True)
    for _ in range(args.profile_steps):
        step()
    torch.cuda.synchronize()
    per_class = {}
    for i, name in enumerate(rv.PROF_CLASSES):
        tot, n = rv.rv_debug_profile_read(v.cache, i)
        per_class[name] = {"ms_per_launch": tot / n if n else None, "launches_per_step": n // args.profile_steps,
                           "ms_per_step": tot / args.profile_steps}
    rv.rv_debug_profile(v.cache, False)
    # the outputs of the last (timed-shape) step, before anything reuses the workspace
    v.k, v.kb = w.k, None  # the timed calls bypassed Verifier.verify
    parity = stored_parity(rv, v, w, lens, drafts)

    tm = traffic_model(shape, lens, S, w.k)
    step_bytes = tm["algorithmic"]
    step_flops = algorithmic_flops(shape, lens, S, w.k)
    steps_per_s = 1000.0 / ms
    gbs = step_bytes / (ms * 1e-3) / 1e9
    M = w.batch * S
    gu_bytes = gateup_bytes(shape, M)
    gu_flops = gateup_flops(shape, M)
    # the dominant kernel's average duration: the production kernel in the
    # pass's launch shape, launched back to back over every layer's weights
    # on the pass's stream, HIP events around the batch.  (This agrees with
    # rocprofv3's in-pass average of the kernel to about 1%; the event pairs
    # the library attaches to single launches in the profiled steps add about
    # 1.7 us to each, so that figure is reported beside it, not used.)
    gu_ms = rv.rv_debug_time_matrix(v.cache, rv.RV_MAT_GATEUP, M, 4 * shape.n_layers, stream=stream)
    gu_inpass_ms = per_class["gateup"]["ms_per_launch"]
    gu_gbs = gu_bytes / (gu_ms * 1e-3) / 1e9 if gu_ms else None
    # bf16 weights: M flops per weight byte; above the ridge the kernel is MFMA-bound
    mfma_bound = shape.dtype == "bf16" and M > RIDGE_FLOP_PER_BYTE
    if mfma_bound:
        achieved = gu_flops / (gu_ms * 1e-3) / 1e12 if gu_ms else None
        roofline = {"kernel": "gate/up matmul + SwiGLU", "bound": "mfma", "achieved": achieved,
                    "peak": MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": (achieved / MFMA_PEAK_TFLOPS) if achieved else None,
                    "algorithmic_flops_per_launch": gu_flops, "ms_per_launch": gu_ms,
                    "in_pass_event_ms_per_launch": gu_inpass_ms, "traffic": None, "hbm_gbs": gu_gbs}
    else:
        roofline = {"kernel": "gate/up matmul + SwiGLU", "bound": "hbm", "achieved": gu_gbs, "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": (gu_gbs / HBM_PEAK_GBS) if gu_gbs else None,
                    "algorithmic_bytes_per_launch": gu_bytes, "ms_per_launch": gu_ms,
                    "in_pass_event_ms_per_launch": gu_inpass_ms, "traffic": None}
    pass_line = {"bound": "mfma" if mfma_bound else "hbm", "algorithmic_bytes": step_bytes,
                 "achieved_gbs": gbs, "frac_of_8tbs": gbs / HBM_PEAK_GBS,
                 "achieved_tflops": step_flops / (ms * 1e-3) / 1e12,
                 "frac_of_2_5pf": step_flops / (ms * 1e-3) / 1e12 / MFMA_PEAK_TFLOPS,
                 "bytes_beyond_algorithmic": {k_: tm[k_] for k_ in ("kv_lo_planes", "operands")}}
    kernel_src = os.path.join(ROOT, "paper_2505_18629_amd", "csrc", "k_gemm.hip")
    if w.name == "8b-bf16-b1":
        roofline["traffic"] = traffic_from_profiles(kernel_src)

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a bounded sample", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, lens, drafts, probe)

    out = {
        "metric": "verify steps/s (+ draft tokens verified/s, HBM GB/s)",
        "value": steps_per_s,
        "unit": "verify steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": shape.dtype,
        "data": "synthetic (seeded random-init weights and token ids)",
        "config": {"workload": w.name, "layers": shape.n_layers, "d_model": shape.d_model,
                   "heads": f"{shape.n_heads}/{shape.n_kv_heads}x{shape.head_dim}", "ffn": shape.ffn_dim,
                   "vocab": shape.vocab, "batch": w.batch, "prefix_len": lens if w.batch <= 4 else
                   [int(min(lens)), int(max(lens))], "k": w.k, "n_probe": w.n_probe, "prefix_pos": w.prefix_pos,
                   "alpha": w.alpha, "block_rows_per_seq": S, "parallelism": "single GPU"},
        "draft_tokens_per_s": steps_per_s * w.batch * w.k,
        "hbm_gbs": gbs,
        "hbm_frac": gbs / HBM_PEAK_GBS,
        "algorithmic_bytes_per_step": step_bytes,
        "tflops": step_flops / (ms * 1e-3) / 1e12,
        "mfma_frac": step_flops / (ms * 1e-3) / 1e12 / MFMA_PEAK_TFLOPS,
        "algorithmic_flops_per_step": step_flops,
        "wall_s_timed": t_wall,
        "accept_len": accept,
        "accept_len_hist": {str(n): accept.count(n) for n in sorted(set(accept))},
        "roofline": roofline,
        "pass": pass_line,
        "parity": parity,
        "kernel_ms_per_step": {k: round(v_["ms_per_step"], 4) for k, v_ in per_class.items()},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    v.close()


if __name__ == "__main__":
    main()
