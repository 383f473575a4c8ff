#!/usr/bin/env python3
"""Decode-step throughput of the SpeContext hot path on one MI355X.

One step = retrieval scoring over every cached token + exact top-k + sparse
GQA attention over the selected K/V rows of every layer (spec_step, one call
on torch's current stream).  Inputs are seeded synthetic tensors already
resident in HBM when the timed region starts.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

Prints ONE JSON line (see the fields below).  Single-GPU build: --gpus N with
N > 1 exits with a message.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode steps/s of retrieve+top-k+sparse attn; achieved HBM GB/s vs peak"
PEAK_HBM_GBPS = 8000.0  # MI355X published HBM3E bandwidth
CSRC = os.path.join(ROOT, "paper_2512_00722_amd", "csrc")
ATTN_SOURCES = ("attn.hip", "device_common.h", "internal.h")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_traffic.json")
FRONT_SOURCES = ("frontend.hip", "device_common.h", "internal.h")
FRONT_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "frontend_traffic.json")
MLA_SOURCES = ("mla.hip", "device_common.h", "internal.h")
MLA_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "mla_traffic.json")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--attn-iters", type=int, default=20)
    ap.add_argument("--head-level", action="store_true",
                    help="one token set per KV head (the group maximum of the retrieval "
                         "heads' weights) instead of one per sequence")
    ap.add_argument("--variants", action="store_true",
                    help="also time the secondary schedules: steps with a 1 GiB cache flush "
                         "before each, per-layer attention launches, and the unfused "
                         "score / top-k / gather / compact-attention sequence")
    ap.add_argument("--frontend", action="store_true",
                    help="time only the retrieval head's front end for the new token "
                         "(embedding row, Q/K projection, YaRN rotary embedding, K_r append): "
                         "--steps calls, replayed from HIP graphs of 20 calls")
    ap.add_argument("--offload", type=int, default=0, metavar="N",
                    help="ragged elastic workload only: keep the last N layers' KV in pinned "
                         "host memory (spec_step_offload: elastic loads over the host link on a "
                         "second stream, one event per layer)")
    ap.add_argument("--headline-only", action="store_true",
                    help="time only the benchmark workload (by default the other four "
                         "decode-step workloads follow it, under \"configs\")")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run three 1 GiB device-to-device copies (known HBM bytes) so "
                         "that PMC byte counters can be scaled")
    return ap.parse_args()


def attn_bytes(w, counts):
    """Algorithmic bytes of one attention launch: selected K and V rows of
    every layer, the bf16 queries and the fp32 outputs."""
    kb = sum(int(c) for c in counts)
    return w.n_layers * (kb * w.H_kv * w.d * 2 * 2 + w.B * w.H_q * w.d * 2 + w.B * w.H_q * w.d * 4)


def attn_source_digest(sources=ATTN_SOURCES):
    """sha256 of a kernel's sources (default: the attention's) with comments
    and blank lines removed: it changes when the code does, not when a
    comment does."""
    import re
    h = hashlib.sha256()
    for name in sources:
        txt = open(os.path.join(CSRC, name)).read()
        txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
        txt = re.sub(r"//[^\n]*", "", txt)
        lines = [ln.rstrip() for ln in txt.splitlines() if ln.strip()]
        h.update(("\n".join(lines) + "\n").encode())
    return h.hexdigest()


def stored_traffic(workload, path=TRAFFIC_FILE, sources=ATTN_SOURCES):
    """Per-launch HBM bytes of a kernel (default: the attention) on
    `workload`, measured with rocprofv3 PMC counters; valid only for the code
    they were taken on."""
    try:
        with open(path) as f:
            t = json.load(f)
        if t.get("attn_code_sha256", t.get("code_sha256")) != attn_source_digest(sources):
            return None
        return t.get("workloads", {}).get(workload, {}).get("bytes_per_launch")
    except (OSError, ValueError):
        return None


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def host_blas():
    """(threads, description) of the BLAS numpy runs the oracle's products on."""
    import numpy as np
    np.ones((64, 64)) @ np.ones((64, 64))   # the BLAS is loaded on first use
    try:
        from threadpoolctl import threadpool_info
        info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if info:
            i = info[0]
            return (int(i.get("num_threads", 1)),
                    f"{i.get('internal_api')} {i.get('version')} ({i.get('threading_layer')}, "
                    f"{i.get('architecture')})")
    except Exception:
        pass
    return len(os.sched_getaffinity(0)), "unknown"


def cpu_baseline(w, x, res, budget_s=20.0):
    """Time the fp64 oracle on a bounded sample of the same step on the host
    cores: every sequence's scoring + top-k, and attention for as many
    layers as fit the budget (selected rows copied to the host untimed);
    the per-step time is scaled to all layers."""
    import numpy as np
    import torch

    import oracle

    threads, blas = host_blas()

    def f64(t):
        return t.float().cpu().numpy().astype(np.float64)

    seq = x["seq_lens"].cpu().numpy()
    ks = x["ks"].cpu().numpy()
    # host copies of the inputs, made outside the timed calls
    qr_h = [f64(x["q_r"][b]) for b in range(w.B)]
    kr_h = [f64(x["K_r"][b, :int(seq[b])]) for b in range(w.B)]
    per_steps, layers_done, spent = [], 0, 0.0
    for rep in range(3):
        t_score = 0.0
        idxs = []
        for b in range(w.B):
            t0 = time.perf_counter()
            s = oracle.retrieval_scores(qr_h[b], kr_h[b], int(seq[b]))
            idx = oracle.topk_indices(s, int(ks[b]))
            t_score += time.perf_counter() - t0
            idxs.append(idx)
        t_attn = 0.0
        layers_done = 0
        for layer in range(w.n_layers):
            for b in range(w.B):
                sel = torch.as_tensor(idxs[b], device=x["K"].device)
                Ks = f64(x["K"][layer, b, sel])
                Vs = f64(x["V"][layer, b, sel])
                qn = f64(x["q"][layer, b])
                t0 = time.perf_counter()
                oracle.sparse_gqa_attention(qn, Ks, Vs, np.arange(len(idxs[b])))
                t_attn += time.perf_counter() - t0
            layers_done += 1
            if t_score + t_attn > budget_s:
                break
        per_steps.append(t_score + t_attn * w.n_layers / layers_done)
        spent += t_score + t_attn
        if spent > budget_s:
            break
    per_step = statistics.median(per_steps)
    return {
        "value": 1.0 / per_step,
        "unit": "steps/s",
        "cores": int(threads),
        "cpu_model": cpu_model(),
        "blas": blas,
        "kind": "oracle",
        "sample": (f"fp64 numpy oracle on the same workload, median of {len(per_steps)} "
                   f"step(s): scoring + top-k for all {w.B} sequences, attention for "
                   f"{layers_done} of {w.n_layers} layers (selected rows copied to host "
                   f"untimed), scaled to {w.n_layers} layers; {spent:.1f} s of CPU work"),
    }


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: the library runs on one GPU; --gpus {args.gpus} is not supported "
              "(the decode step would shard by sequence with no exchange; that path is not built)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2512_00722_amd as spec
    from workloads import BENCH_WORKLOAD, WORKLOADS, algorithmic_bytes, elastic_sequence, generate

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    spec.load_library()
    dev = torch.device("cuda:0")
    name = args.workload or BENCH_WORKLOAD
    w = WORKLOADS[name]
    t_gen = time.perf_counter()
    if w.mla and not args.frontend:
        from workloads import generate_mla
        x = generate_mla(w, seed=args.seed, device=dev)
    else:
        x = generate(w, seed=args.seed, device=dev, with_kv=not args.frontend and not w.mla)
    torch.cuda.synchronize()
    t_gen = time.perf_counter() - t_gen
    print(f"[bench] workload {name} generated in {t_gen:.1f}s", file=sys.stderr, flush=True)

    if args.frontend:
        print(json.dumps(run_frontend(args, spec, w, x)), flush=True)
        return
    if w.mla:
        if args.head_level:
            print("bench.py: the MLA workload keeps one token set per sequence", file=sys.stderr)
            sys.exit(2)
        print(json.dumps(run_mla(args, spec, w, x)), flush=True)
        return
    if w.steps > 1 and args.head_level:
        print("bench.py: elastic loading keeps one token set per sequence; --head-level does "
              "not apply to this workload", file=sys.stderr)
        sys.exit(2)
    if args.offload:
        if w.steps <= 1:
            print("bench.py: --offload applies to the ragged elastic workload", file=sys.stderr)
            sys.exit(2)
        line = run_offload(args, spec, w, x, elastic_sequence(w, x, seed=args.seed, device=dev),
                           args.offload)
        print(json.dumps(line), flush=True)
        return
    if w.steps > 1:
        line = run_elastic(args, spec, w, x, elastic_sequence(w, x, seed=args.seed, device=dev),
                           algorithmic_bytes)
        print(json.dumps(line), flush=True)
        return

    line = run_fixed(args, spec, w, x, name)
    if args.workload is None and not args.headline_only:
        # the other decode-step workloads, each generated, measured and freed in turn
        del x
        torch.cuda.empty_cache()
        line["configs"] = other_configs(args, spec, WORKLOADS, dev)
    print(json.dumps(line), flush=True)


def run_fixed(args, spec, w, x, name):
    """The fused step on a fixed-length workload: exactly args.steps steps
    timed between two device synchronisations (the headline), per-step HIP
    events over as many steps again (median, p10, p90), per-op times from
    graph replays, the attention kernel against the HBM roofline."""
    import torch
    from workloads import algorithmic_bytes

    dev = x["q"].device
    call = dict(q_r=x["q_r"], K_r=x["K_r"], seq_lens=x["seq_lens"], ks=x["ks"], q=x["q"],
                K=x["K"], V=x["V"], k_max=w.k, head_level=args.head_level)
    outputs = {}
    res = spec.step(**call, outputs=outputs)
    torch.cuda.synchronize()
    ws = torch.zeros(spec.workspace_size(_dims_of(spec, w, x, args.head_level), spec.OP_STEP),
                     dtype=torch.uint8, device=dev)

    for _ in range(args.warmup):
        spec.step(**call, outputs=outputs, ws=ws)
    torch.cuda.synchronize()

    # ---- timed region: exactly K steps between two device synchronisations
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record()
    for i in range(args.steps):
        spec.step(**call, outputs=outputs, ws=ws)
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps
    ev_ms_per_step = ev0.elapsed_time(ev1) / args.steps
    print(f"[bench] {args.steps} steps in {wall:.3f}s", file=sys.stderr, flush=True)
    per_step = per_step_events(lambda: spec.step(**call, outputs=outputs, ws=ws),
                               max(args.steps, 50))

    # ---- per-op times (same inputs, same stream), HIP events
    counts = outputs["counts"].cpu().tolist()
    seq = x["seq_lens"].cpu().tolist()
    n_it = args.attn_iters
    attn_out = torch.empty_like(outputs["out"])
    dims_a = _dims_attn(spec, w, x, outputs)
    ws_attn = torch.zeros(max(16, spec.workspace_size(dims_a, spec.OP_ATTN)), dtype=torch.uint8,
                          device=dev)
    n_sets = w.H_kv if args.head_level else 1
    sets = (n_sets,) if args.head_level else ()
    scores = torch.empty((w.B,) + sets + (w.L_cap,), dtype=torch.float32, device=dev)
    # Each op is timed over n_it back-to-back launches captured in a HIP
    # graph and replayed between two events on the launch stream, so that the
    # figure is the GPU's, not the Python launch path's (the standalone
    # scoring call takes about as long to launch from Python as to run).
    def timed(fn):
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(n_it):
                fn()
        graph.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        graph.replay()
        e1.record()
        torch.cuda.synchronize()
        del graph
        return e0.elapsed_time(e1) * 1e3 / n_it

    dims_hl = _dims_of(spec, w, x, args.head_level)
    ws_score = torch.zeros(spec.workspace_size(dims_hl, spec.OP_SCORE), dtype=torch.uint8,
                           device=dev)
    ws_topk = torch.zeros(max(16, spec.workspace_size(dims_hl, spec.OP_TOPK)),
                          dtype=torch.uint8, device=dev)
    op_us = {
        "score": timed(lambda: spec.score(x["q_r"], x["K_r"], x["seq_lens"], out=scores,
                                          ws=ws_score, n_sets=n_sets)),
        "topk": timed(lambda: spec.topk(scores, x["seq_lens"], x["ks"], w.k, idx=outputs["idx"],
                                        counts=outputs["counts"], ws=ws_topk)),
        "attn": timed(lambda: spec.sparse_decode_attn(x["q"], x["K"], x["V"], outputs["counts"],
                                                      idx=outputs["idx"], out=attn_out,
                                                      with_lse=False, ws=ws_attn)),
    }

    step_bytes = algorithmic_bytes(w, seq, x["ks"].cpu().tolist())
    a_bytes = attn_bytes(w, counts)
    attn_s = op_us["attn"] * 1e-6
    achieved = a_bytes / attn_s / 1e9
    # the stored counters were taken with one token set per sequence
    traffic = None if args.head_level else stored_traffic(name)
    value = args.steps / wall
    line = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": name, "B": w.B, "L": w.L, "H_r": w.H_r, "d_r": w.d_r,
                   "n_layers": w.n_layers, "H_q": w.H_q, "H_kv": w.H_kv, "d": w.d, "k": w.k,
                   "token_sets": "per_kv_head" if args.head_level else "per_sequence"},
        "roofline": {
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": PEAK_HBM_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBPS, 4),
            "traffic": traffic,
            # the partials workspace exists only when selections are split (then a
            # second kernel merges them)
            "kernel": "sparse GQA decode attention (attn_split_kernel"
                      + (" + attn_combine_kernel)" if spec.workspace_size(dims_a, spec.OP_ATTN) > 0
                         else ")"),
            "bytes_per_launch": a_bytes,
            "avg_launch_us": round(op_us["attn"], 2),
        },
        "step_hbm_gbps": round(step_bytes * value / 1e9, 1),
        "step_frac_of_peak": round(step_bytes * value / 1e9 / PEAK_HBM_GBPS, 4),
        "step_algorithmic_bytes": step_bytes,
        "step_ms_events": round(ev_ms_per_step, 4),
        "step_us": per_step,
        "op_us": {k: round(v, 2) for k, v in op_us.items()},
    }
    if args.variants:
        line["variants"] = run_variants(args, spec, w, x, call, outputs, ws, step_bytes, n_sets)
    if args.copy_calibration:
        copy_calibration(dev)
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a bounded sample", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(w, x, res)
    return line


def _spread(t):
    t = sorted(t)
    q = lambda f: t[min(len(t) - 1, int(f * len(t)))]
    return {"n": len(t), "median": round(statistics.median(t), 2), "p10": round(q(0.1), 2),
            "p90": round(q(0.9), 2), "mean": round(statistics.mean(t), 2)}


def per_step_events(fn, n):
    """Median, p10, p90 and mean of n single steps, each between two HIP
    events on the launch stream (eager launches, as in the timed loop)."""
    import torch
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(n)]
    for e0, e1 in evs:
        e0.record()
        fn()
        e1.record()
    torch.cuda.synchronize()
    return _spread([e0.elapsed_time(e1) * 1e3 for e0, e1 in evs])


def other_configs(args, spec, workloads, dev):
    """The other decode-step workloads of the benchmark, one after another
    (each generated on the GPU, measured, then freed): steps/s, per-step
    spread, the step's algorithmic bytes against peak, and the attention
    kernel against the roofline with its stored PMC traffic."""
    import copy

    import torch
    from workloads import BENCH_WORKLOAD, algorithmic_bytes, elastic_sequence, generate

    res = {}
    for name in ("b1_l4096_k512_1layer", "b32_l16384_k1024_hr16", "b1_l131072_k4096_g8",
                 "b64_ragged_l2k_16k_elastic"):
        if name == BENCH_WORKLOAD:
            continue
        w = workloads[name]
        a = copy.copy(args)
        a.no_cpu_baseline, a.variants, a.copy_calibration = True, False, False
        t0 = time.perf_counter()
        x = generate(w, seed=args.seed, device=dev)
        torch.cuda.synchronize()
        print(f"[bench] config {name} generated in {time.perf_counter() - t0:.1f}s",
              file=sys.stderr, flush=True)
        if w.steps > 1:
            a.steps, a.warmup = 3 * w.steps, w.steps     # three 16-step passes
            ln = run_elastic(a, spec, w, x, elastic_sequence(w, x, seed=args.seed, device=dev),
                             algorithmic_bytes)
        else:
            ln = run_fixed(a, spec, w, x, name)
        keep = ("value", "ms_per_step", "step_us", "step_frac_of_peak", "step_hbm_gbps",
                "step_algorithmic_bytes", "op_us", "first_step_us", "later_steps_us_mean")
        r = {k: ln[k] for k in keep if k in ln}
        r["steps"] = a.steps
        r["roofline"] = {k: ln["roofline"][k] for k in ("achieved", "frac", "traffic",
                                                         "bytes_per_launch", "avg_launch_us",
                                                         "kernel")}
        res[name] = r
        if w.steps > 1:   # the same workload with its last 4 layers' KV in host memory
            a.offload = 4
            ln = run_offload(a, spec, w, x, elastic_sequence(w, x, seed=args.seed, device=dev), 4)
            res[name + "_offload4"] = {k: ln[k] for k in ("value", "ms_per_step", "step_us",
                                                          "first_step_us", "host_link",
                                                          "host_bytes_per_step")}
            res[name + "_offload4"]["steps"] = a.steps
        del x, ln
        torch.cuda.empty_cache()
    return res


def run_elastic(args, spec, w, x, e, algorithmic_bytes):
    """The appended-token workload: decode steps run through the w.steps-step
    sequence cyclically; the elastic state is reset at the start of each pass
    (its first step is a full load).  Exactly args.steps steps are timed."""
    import torch

    dev = x["K"].device
    S = w.steps
    st = spec.ElasticState(w.n_layers, w.B, w.k, w.H_kv, w.d, dev)
    outputs = {}
    ws = torch.zeros(spec.workspace_size(_dims_of(spec, w, x), spec.OP_STEP), dtype=torch.uint8,
                     device=dev)

    def one(i):
        s = i % S
        if s == 0:
            st.reset()
        spec.step(q_r=e["q_r"][s], K_r=x["K_r"], seq_lens=e["seq_lens"][s], ks=x["ks"],
                  q=e["q"][s], K=x["K"], V=x["V"], k_max=w.k, elastic=st, outputs=outputs, ws=ws)

    for i in range(args.warmup):
        one(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        one(i)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    value = args.steps / wall
    print(f"[bench] {args.steps} elastic steps in {wall:.3f}s", file=sys.stderr, flush=True)

    # Untimed passes with per-step events and readback: rows loaded per step,
    # per-step times, and the algorithmic bytes of the timed steps.  The
    # first pass only warms up the readback path (its first use initialises
    # host-side work that would land inside the first step's events).
    ks = x["ks"].cpu().tolist()
    for _ in range(2):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * S)]
        deltas, step_bytes = [], []
        for s in range(S):
            ev[2 * s].record()
            one(s)
            ev[2 * s + 1].record()
            torch.cuda.synchronize()
            deltas.append(int(st.n_changed.sum()))
            step_bytes.append(algorithmic_bytes(w, e["seq_lens"][s].cpu().tolist(), ks,
                                                delta_rows=deltas[-1]))
        step_us = [ev[2 * s].elapsed_time(ev[2 * s + 1]) * 1e3 for s in range(S)]
    timed_bytes = sum(step_bytes[i % S] for i in range(args.steps))
    k_total = sum(min(k, int(L)) for k, L in zip(ks, e["seq_lens"][0].cpu().tolist()))

    # The dominant kernel, timed back to back between HIP events on the
    # launch stream: the step's attention over the slots.  On a steady
    # update (a fifth of the rows new) the step copies the new rows first
    # and the attention only reads the slots, which the compact attention
    # over the slot buffers reproduces.  With SPEC_ELASTIC_PATH=fused the
    # attention loads every update's rows itself: then the kernel timed is
    # that attention with the last update's slot sources (rerunning it
    # rewrites the same rows).
    counts = outputs["counts"]
    attn_out = torch.empty_like(outputs["out"])
    q_last = e["q"][S - 1]
    copy_path = os.environ.get("SPEC_ELASTIC_PATH") != "fused"
    dims_a = spec.Dims.make(B=w.B, L_cap=w.k, L_max=w.k, k_max=w.k, n_layers=w.n_layers,
                            H_q=w.H_q, H_kv=w.H_kv, d=w.d)
    ws_attn = torch.zeros(max(16, spec.workspace_size(dims_a, spec.OP_ATTN),
                              spec.workspace_size(_dims_of(spec, w, x), spec.OP_ATTN)),
                          dtype=torch.uint8, device=dev)
    if copy_path:
        fn = lambda: spec.sparse_decode_attn(q_last, st.kbuf, st.vbuf, counts, idx=None,
                                             out=attn_out, with_lse=False, ws=ws_attn)
    else:
        fn = lambda: spec.sparse_decode_attn_elastic(q_last, x["K"], x["V"], st, counts,
                                                     out=attn_out, with_lse=False, ws=ws_attn)
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.attn_iters):
        fn()
    e1.record()
    torch.cuda.synchronize()
    attn_us = e0.elapsed_time(e1) * 1e3 / args.attn_iters
    kb = sum(int(c) for c in counts.cpu().tolist())
    a_bytes = w.n_layers * (kb * w.H_kv * w.d * 2 * 2 + w.B * w.H_q * w.d * 2 + w.B * w.H_q * w.d * 4)
    if not copy_path:  # plus the rows written into their slots
        a_bytes += w.n_layers * int(st.n_changed.sum()) * w.H_kv * w.d * 2 * 2
    achieved = a_bytes / (attn_us * 1e-6) / 1e9
    if args.copy_calibration:
        copy_calibration(dev)
    return {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "L0": [w.ragged_min, w.L], "H_r": w.H_r,
                   "d_r": w.d_r, "n_layers": w.n_layers, "H_q": w.H_q, "H_kv": w.H_kv, "d": w.d,
                   "k": w.k, "steps_per_pass": S, "elastic": True},
        "roofline": {
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": PEAK_HBM_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBPS, 4),
            "traffic": stored_traffic(w.name),
            "kernel": ("sparse GQA decode attention over the slot buffers (attn_split_kernel)"
                       if copy_path else "sparse GQA decode attention over the slots, loading "
                       "the update's rows (attn_split_kernel)"),
            "bytes_per_launch": a_bytes,
            "avg_launch_us": round(attn_us, 2),
        },
        "step_hbm_gbps": round(timed_bytes / wall / 1e9, 1),
        "step_frac_of_peak": round(timed_bytes / wall / 1e9 / PEAK_HBM_GBPS, 4),
        "step_algorithmic_bytes": round(timed_bytes / args.steps),
        "rows_loaded_per_step": deltas,
        "selected_rows": k_total,
        "step_us": _spread(step_us),
        "first_step_us": round(step_us[0], 1),
        "later_steps_us_mean": round(statistics.mean(step_us[1:]), 1) if S > 1 else None,
    }


PCIE5_X16_GBPS = 64.0  # MI355X host link, PCIe 5.0 x16, one direction (published)


def host_link_gbps(dev, nbytes=1 << 30):
    """Host-to-device bandwidth of a plain copy from pinned memory (the
    reference the elastic loads are compared with): median of 3 copies."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    dst = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    ts = []
    for _ in range(4):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src, non_blocking=True)
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1) * 1e-3)
    del src, dst
    return nbytes / statistics.median(ts[1:]) / 1e9


def run_offload(args, spec, w, x, e, n_off):
    """The ragged elastic workload with the KV of its last n_off layers in
    pinned host memory (spec_step_offload): per step the retrieval and top-k,
    the elastic plan, the host-to-device loads of S_now - S_last for each
    offloaded layer on a second stream, the attention of the device layers
    meanwhile, then each offloaded layer's attention after its own rows.  The
    16-step sequence runs cyclically; each pass starts from an empty slot
    state (a full load).  Reports steps/s, the bytes each step moved over the
    host link against a full reload of the same selection, and the loads'
    host-link bandwidth (measured alone) against a plain pinned copy."""
    import torch

    dev = x["K"].device
    S = w.steps
    n_dev = w.n_layers - n_off
    t0 = time.perf_counter()
    host_k = torch.empty((n_off,) + tuple(x["K"].shape[1:]), dtype=torch.bfloat16,
                         pin_memory=True)
    host_v = torch.empty_like(host_k, pin_memory=True)
    host_k.copy_(x["K"][n_dev:])
    host_v.copy_(x["V"][n_dev:])
    print(f"[bench] {n_off} layers ({2 * host_k.numel() * 2 / 1e9:.1f} GB) in pinned host memory "
          f"in {time.perf_counter() - t0:.1f}s", file=sys.stderr, flush=True)
    K_dev, V_dev = (x["K"][:n_dev], x["V"][:n_dev]) if n_dev else (None, None)
    st = spec.ElasticState(n_off, w.B, w.k, w.H_kv, w.d, dev)
    copy = torch.cuda.Stream()
    events = spec.OffloadEvents(n_off, dev)
    outputs = {}
    dims = spec.Dims.make(B=w.B, L_cap=w.L_cap, L_max=w.L_cap, k_max=w.k, H_r=w.H_r, d_r=w.d_r,
                          n_layers=w.n_layers, H_q=w.H_q, H_kv=w.H_kv, d=w.d,
                          kr_stride_b=x["K_r"].stride(0), kv_stride_layer=x["K"].stride(0),
                          kv_stride_b=x["K"].stride(1))
    ws = torch.zeros(spec.workspace_size(dims, spec.OP_OFFLOAD), dtype=torch.uint8, device=dev)

    def one(i):
        s = i % S
        if s == 0:
            st.reset()
        spec.step_offload(e["q_r"][s], x["K_r"], e["seq_lens"][s], x["ks"], e["q"][s], K_dev,
                          V_dev, host_k, host_v, w.k, st, copy_stream=copy, events=events,
                          ws=ws, outputs=outputs)

    for i in range(args.warmup):
        one(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        one(i)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    value = args.steps / wall
    print(f"[bench] {args.steps} offloaded steps in {wall:.3f}s", file=sys.stderr, flush=True)

    # One more pass with per-step events and the rows each step loaded.
    row_bytes = 2 * w.H_kv * w.d * 2          # K and V of one token in one layer
    step_us, rows = [], []
    for s in range(S):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        one(s)
        e1.record()
        torch.cuda.synchronize()
        step_us.append(e0.elapsed_time(e1) * 1e3)
        rows.append(int(st.n_changed.sum()))
    k_total = int(outputs["counts"].sum())
    host_bytes = [r * n_off * row_bytes for r in rows]
    full_bytes = k_total * n_off * row_bytes

    # The loads alone (plan + host copies, one stream) on the same selections:
    # the host-link bandwidth they reach, later steps of a pass.
    idx_seq = []
    for s in range(S):
        r = spec.step(e["q_r"][s], x["K_r"], e["seq_lens"][s], x["ks"], e["q"][s], x["K"],
                      x["V"], k_max=w.k)
        idx_seq.append((r["idx"].clone(), r["counts"].clone()))
    st2 = spec.ElasticState(n_off, w.B, w.k, w.H_kv, w.d, dev)
    load_us = []
    for s in range(S):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        spec.offload_load(idx_seq[s][0], idx_seq[s][1], host_k, host_v, st2)
        e1.record()
        torch.cuda.synchronize()
        load_us.append(e0.elapsed_time(e1) * 1e3)
    link = host_link_gbps(dev)
    later = range(1, S)
    load_gbps = statistics.median(host_bytes[s] / (load_us[s] * 1e-6) / 1e9 for s in later)
    full_gbps = host_bytes[0] / (load_us[0] * 1e-6) / 1e9
    med_bytes = statistics.median(host_bytes[s] for s in later)
    del host_k, host_v
    return {
        "metric": "decode steps/s of retrieve+top-k+sparse attn with the last layers' KV in "
                  "host memory (elastic loading over the host link)",
        "value": round(value, 3), "unit": "steps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(wall * 1e3 / args.steps, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "L0": [w.ragged_min, w.L], "n_layers": w.n_layers,
                   "layers_in_host_memory": n_off, "H_q": w.H_q, "H_kv": w.H_kv, "d": w.d,
                   "k": w.k, "steps_per_pass": S},
        "step_us": _spread(step_us[1:]),
        "first_step_us": round(step_us[0], 1),
        "host_link": {
            "bound": "host_link",
            "elastic_load_gbps": round(load_gbps, 1),
            "full_load_gbps": round(full_gbps, 1),
            "plain_copy_gbps": round(link, 1),
            "frac_of_plain_copy": round(load_gbps / link, 3),
            "peak_gbps": PCIE5_X16_GBPS,
            "load_us_median": round(statistics.median(load_us[s] for s in later), 1),
        },
        "host_bytes_per_step": {
            "elastic_median": int(med_bytes),
            "full_reload": int(full_bytes),
            "reduction": round(1.0 - med_bytes / full_bytes, 4),
            "rows_loaded_per_step": rows,
            "selected_rows": k_total,
        },
    }


def copy_calibration(dev):
    """Three 1 GiB device-to-device copies (known HBM bytes) whose PMC byte
    counts scale the counters of the kernels."""
    import torch
    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def run_frontend(args, spec, w, x):
    """The retrieval head's front end alone: --steps calls on the workload's
    synthetic weights (the whole embedding table), timed over graph replays
    with HIP events on the launch stream."""
    import torch
    from workloads import frontend_bytes, frontend_inputs

    dev = x["K_r"].device
    fe = frontend_inputs(w, x["seq_lens"], seed=args.seed, device=dev)
    q_r = torch.empty_like(x["q_r"])
    dims = _dims_of_retrieval(spec, w, x)
    ws = torch.zeros(spec.workspace_size(dims, spec.OP_FRONTEND), dtype=torch.uint8, device=dev)

    def front():
        spec.retrieval_qk(fe["tokens"], fe["pos"], fe["emb"], fe["w_q"], fe["w_k"], x["K_r"],
                          rope_base=w.rope_base, yarn_scale=w.yarn_scale,
                          yarn_orig_ctx=w.orig_ctx, q_r=q_r, ws=ws)

    reps = 20
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(max(args.warmup, 1)):
            front()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(reps):
            front()
    graph.replay()
    torch.cuda.synchronize()
    n_rep = max(1, (args.steps + reps - 1) // reps)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(n_rep):
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    calls = n_rep * reps
    us = e0.elapsed_time(e1) * 1e3 / calls
    fb = frontend_bytes(w)
    achieved = fb / (us * 1e-6) / 1e9
    kernels = ("qk_gemv_kernel" if w.B <= 16 else
               "qk_full_kernel" if w.B <= 64 else "qk_partial_kernel + qk_finish_kernel")
    line = {
        "metric": "retrieval head front-end calls/s (embedding, Q/K projection, YaRN RoPE, "
                  "K_r append)",
        "value": round(calls / wall, 1),
        "unit": "calls/s",
        "n_gpus": 1, "steps": calls, "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / calls, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H_r": w.H_r, "d_r": w.d_r,
                   "hidden": w.hidden, "vocab": w.vocab, "rope_base": w.rope_base,
                   "yarn_scale": w.yarn_scale, "orig_ctx": w.orig_ctx},
        "roofline": {
            "bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS,
            "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBPS, 4),
            "traffic": stored_traffic(w.name, FRONT_TRAFFIC_FILE, FRONT_SOURCES),
            "kernel": kernels, "bytes_per_launch": fb, "avg_launch_us": round(us, 3),
        },
    }
    del graph, fe
    if args.copy_calibration:
        copy_calibration(dev)
    return line


def run_mla(args, spec, w, x):
    """A decode step of an MLA model: retrieval scores, top-k, then the MLA
    sparse attention of every layer over the selected latent rows.  Timed
    over --steps eager steps between two device synchronisations (HIP
    events on the launch stream); the roofline is that of the MLA entry
    point (absorption, latent attention, output projection) with its
    algorithmic bytes: selected latent rows, queries, up-projection weights
    and outputs of every layer."""
    import numpy as np
    import torch
    from workloads import mla_attn_bytes, mla_bytes

    dev = x["K_r"].device
    dims_s = _dims_of_retrieval(spec, w, x)
    scores = torch.empty((w.B, w.L_cap), dtype=torch.float32, device=dev)
    idx = torch.empty((w.B, w.k), dtype=torch.int32, device=dev)
    counts = torch.empty((w.B,), dtype=torch.int32, device=dev)
    ws_s = torch.zeros(spec.workspace_size(dims_s, spec.OP_SCORE), dtype=torch.uint8, device=dev)
    dims_t = spec.Dims.make(B=w.B, L_cap=w.L_cap, L_max=w.L_cap, k_max=w.k, H_q=1, H_kv=1)
    ws_t = torch.zeros(max(16, spec.workspace_size(dims_t, spec.OP_TOPK)), dtype=torch.uint8,
                       device=dev)
    dims_m = spec.MlaDims.make(B=w.B, L_cap=w.L_cap, k_max=w.k, n_layers=w.n_layers, H=w.H_q,
                               ckv_stride_layer=x["ckv"].stride(0),
                               ckv_stride_b=x["ckv"].stride(1))
    ws_m = torch.zeros(spec.mla_workspace_size(dims_m), dtype=torch.uint8, device=dev)
    out = torch.empty((w.n_layers, w.B, w.H_q, w.d_v), dtype=torch.float32, device=dev)

    def mla():
        spec.mla_sparse_decode_attn(x["q_mla"], x["ckv"], x["w_uk"], x["w_uv"], idx, counts,
                                    out=out, with_lse=False, ws=ws_m)

    def step():
        spec.score(x["q_r"], x["K_r"], x["seq_lens"], out=scores, ws=ws_s)
        spec.topk(scores, x["seq_lens"], x["ks"], w.k, idx=idx, counts=counts, ws=ws_t)
        mla()

    for _ in range(max(args.warmup, 1)):
        step()
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record()
    for _ in range(args.steps):
        step()
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    print(f"[bench] {args.steps} MLA steps in {wall:.3f}s", file=sys.stderr, flush=True)

    n_it = args.attn_iters
    mla()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(n_it):
        mla()
    e1.record()
    torch.cuda.synchronize()
    mla_us = e0.elapsed_time(e1) * 1e3 / n_it
    seq = x["seq_lens"].cpu().tolist()
    ks = x["ks"].cpu().tolist()
    m_bytes = mla_attn_bytes(w, seq, ks)
    s_bytes = mla_bytes(w, seq, ks)
    achieved = m_bytes / (mla_us * 1e-6) / 1e9
    value = args.steps / wall
    line = {
        "metric": "decode steps/s of retrieve + top-k + MLA sparse attention (latent cache); "
                  "achieved HBM GB/s vs peak",
        "value": round(value, 3), "unit": "steps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(wall * 1e3 / args.steps, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "L": w.L, "H_r": w.H_r, "d_r": w.d_r,
                   "n_layers": w.n_layers, "H": w.H_q, "d_c": w.d_c, "d_rope": w.d_rope,
                   "d_nope": w.d_nope, "d_v": w.d_v, "k": w.k},
        "roofline": {
            "bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS,
            "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBPS, 4),
            "traffic": stored_traffic(w.name, MLA_TRAFFIC_FILE, MLA_SOURCES),
            "kernel": "MLA sparse attention (mla_absorb_kernel + mla_attn_kernel + "
                      "mla_out_kernel)",
            "bytes_per_launch": m_bytes, "avg_launch_us": round(mla_us, 2),
        },
        "step_hbm_gbps": round(s_bytes * value / 1e9, 1),
        "step_frac_of_peak": round(s_bytes * value / 1e9 / PEAK_HBM_GBPS, 4),
        "step_algorithmic_bytes": s_bytes,
        "step_ms_events": round(ev0.elapsed_time(ev1) / args.steps, 4),
    }
    if args.copy_calibration:
        copy_calibration(dev)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = mla_cpu_baseline(w, x, idx, counts)
    return line


def mla_cpu_baseline(w, x, idx, counts, budget_s=20.0):
    """The fp64 oracle on a bounded sample of the MLA step: one sequence's
    scoring + top-k and its MLA attention over as many (layer) units as fit
    the budget, scaled to all sequences and layers."""
    import numpy as np
    import oracle

    threads, blas = host_blas()

    def f64(t):
        return t.float().cpu().numpy().astype(np.float64)

    L = int(x["seq_lens"][0])
    qr, kr = f64(x["q_r"][0]), f64(x["K_r"][0, :L])
    t0 = time.perf_counter()
    sel = oracle.topk_indices(oracle.retrieval_scores(qr, kr, L), int(x["ks"][0]))
    t_score = time.perf_counter() - t0
    t_attn, done = 0.0, 0
    for layer in range(w.n_layers):
        q = f64(x["q_mla"][layer, 0])
        ckv = f64(x["ckv"][layer, 0])
        wuk, wuv = f64(x["w_uk"][layer]), f64(x["w_uv"][layer])
        t0 = time.perf_counter()
        oracle.mla_sparse_attention(q[:, :w.d_nope], q[:, w.d_nope:], ckv[:, :w.d_c],
                                    ckv[:, w.d_c:], wuk, wuv, sel)
        t_attn += time.perf_counter() - t0
        done += 1
        if t_score + t_attn > budget_s:
            break
    per_step = w.B * (t_score + t_attn * w.n_layers / done)
    return {"value": 1.0 / per_step, "unit": "steps/s", "cores": int(threads),
            "cpu_model": cpu_model(), "blas": blas, "kind": "oracle",
            "sample": (f"fp64 numpy oracle: scoring + top-k and MLA attention (per-head keys "
                       f"and values raised from the selected latents) of sequence 0 for "
                       f"{done} of {w.n_layers} layers, scaled to {w.n_layers} layers and "
                       f"{w.B} sequences; {t_score + t_attn:.1f} s of CPU work")}


def _dims_of_retrieval(spec, w, x):
    return spec.Dims.make(B=w.B, L_cap=w.L_cap, L_max=w.L_cap, k_max=1, H_r=w.H_r, d_r=w.d_r,
                          n_layers=1, H_q=1, H_kv=1, d=128, kr_stride_b=x["K_r"].stride(0))


def run_variants(args, spec, w, x, call, outputs, ws, step_bytes, n_sets=1):
    """Secondary schedules of the same step (µs per step, HIP events on the
    launch stream).

    flushed_step: each step alone, after a 1 GiB write that evicts the L2 and
    the 256 MB last-level cache (outside the events): median, p10, p90.
    per_layer_attention: score, top-k, then one attention launch per layer
    (the schedule of a model that attends layer by layer).
    unfused: score, top-k, materialised gather of the selected rows of every
    layer, attention over the compact rows.
    fused_step_graph: the fused step, replayed from a HIP graph.
    retrieval_frontend: the retrieval head's front end for the new token
    (per call, 20 calls per graph); frontend_then_step_graph: the front end
    followed by the step on the q_r it produced.
    These are captured in HIP graphs and replayed.
    """
    import torch

    dev = x["K"].device
    n = max(args.steps // 2, 5)

    def ev_loop(fn, iters):
        """µs per call of fn, captured once in a HIP graph and replayed
        (the many small launches of these schedules would otherwise time the
        Python launch path, not the GPU)."""
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for _ in range(3):
                fn()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            fn()
        graph.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(iters):
            graph.replay()
        e1.record()
        torch.cuda.synchronize()
        del graph
        return e0.elapsed_time(e1) * 1e3 / iters

    res = {}
    flush = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    times = []
    for i in range(n):
        flush.fill_(i & 255)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        spec.step(**call, outputs=outputs, ws=ws)
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1) * 1e3)
    del flush
    times.sort()
    med = statistics.median(times)
    res["flushed_step"] = {"median_us": round(med, 1), "p10_us": round(times[len(times) // 10], 1),
                           "p90_us": round(times[(9 * len(times)) // 10], 1),
                           "steps_per_s": round(1e6 / med, 1),
                           "frac_of_peak": round(step_bytes / (med * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4)}

    sets = (n_sets,) if n_sets > 1 else ()
    scores = torch.empty((w.B,) + sets + (w.L_cap,), dtype=torch.float32, device=dev)
    idx, counts = outputs["idx"], outputs["counts"]
    dims_s = _dims_of(spec, w, x, n_sets > 1)
    ws_s = torch.zeros(spec.workspace_size(dims_s, spec.OP_SCORE), dtype=torch.uint8, device=dev)
    ws_t = torch.zeros(max(16, spec.workspace_size(dims_s, spec.OP_TOPK)), dtype=torch.uint8,
                       device=dev)
    out = torch.empty_like(outputs["out"])

    def score_topk():
        spec.score(x["q_r"], x["K_r"], x["seq_lens"], out=scores, ws=ws_s, n_sets=n_sets)
        spec.topk(scores, x["seq_lens"], x["ks"], w.k, idx=idx, counts=counts, ws=ws_t)

    dims_l = spec.Dims.make(B=w.B, L_cap=w.L_cap, L_max=w.L_cap, k_max=w.k, n_layers=1,
                            H_q=w.H_q, H_kv=w.H_kv, d=w.d, kv_stride_layer=x["K"].stride(0),
                            kv_stride_b=x["K"].stride(1))
    ws_l = torch.zeros(max(16, spec.workspace_size(dims_l, spec.OP_ATTN)), dtype=torch.uint8,
                       device=dev)

    def per_layer():
        score_topk()
        for layer in range(w.n_layers):
            spec.sparse_decode_attn(x["q"][layer:layer + 1], x["K"][layer:layer + 1],
                                    x["V"][layer:layer + 1], counts, idx=idx,
                                    out=out[layer:layer + 1], with_lse=False, ws=ws_l)

    us = ev_loop(per_layer, n)
    res["per_layer_attention"] = {"us_per_step": round(us, 1), "steps_per_s": round(1e6 / us, 1)}

    ks = torch.empty((w.n_layers, w.B, w.k, w.H_kv, w.d), dtype=torch.bfloat16, device=dev)
    vs = torch.empty_like(ks)
    dims_c = spec.Dims.make(B=w.B, L_cap=w.k, L_max=w.k, k_max=w.k, n_layers=w.n_layers,
                            H_q=w.H_q, H_kv=w.H_kv, d=w.d)
    ws_c = torch.zeros(max(16, spec.workspace_size(dims_c, spec.OP_ATTN)), dtype=torch.uint8,
                       device=dev)

    def unfused():
        score_topk()
        spec.gather(x["K"], x["V"], idx, counts, out=(ks, vs))
        spec.sparse_decode_attn(x["q"], ks, vs, counts, out=out, with_lse=False, ws=ws_c)

    us = ev_loop(unfused, n)
    res["unfused_with_gather"] = {"us_per_step": round(us, 1), "steps_per_s": round(1e6 / us, 1)}
    us = ev_loop(lambda: spec.step(**call, outputs=outputs, ws=ws), n)
    res["fused_step_graph"] = {"us_per_step": round(us, 1), "steps_per_s": round(1e6 / us, 1)}
    del ks, vs

    # The retrieval head's front end for the new token (embedding row, Q/K
    # projection, YaRN rotary embedding, append to K_r), alone and ahead of
    # the step.  It writes the new key over each sequence's last cached row.
    from workloads import frontend_bytes, frontend_inputs
    fe = frontend_inputs(w, x["seq_lens"], seed=0, device=dev)
    q_r_new = torch.empty_like(x["q_r"])
    ws_f = torch.zeros(spec.workspace_size(dims_s, spec.OP_FRONTEND), dtype=torch.uint8,
                       device=dev)

    def front():
        spec.retrieval_qk(fe["tokens"], fe["pos"], fe["emb"], fe["w_q"], fe["w_k"], x["K_r"],
                          rope_base=w.rope_base, yarn_scale=w.yarn_scale,
                          yarn_orig_ctx=w.orig_ctx, q_r=q_r_new, ws=ws_f)

    reps = 20

    def front_rep():
        for _ in range(reps):
            front()

    us = ev_loop(front_rep, n) / reps
    fb = frontend_bytes(w)
    res["retrieval_frontend"] = {
        "us_per_call": round(us, 2), "algorithmic_bytes": fb,
        "GBps": round(fb / (us * 1e-6) / 1e9, 1),
        "frac_of_peak": round(fb / (us * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4),
        "vocab": w.vocab, "hidden": w.hidden, "yarn_scale": w.yarn_scale}
    call_fe = dict(call)
    call_fe["q_r"] = q_r_new

    def front_step():
        front()
        spec.step(**call_fe, outputs=outputs, ws=ws)

    us = ev_loop(front_step, n)
    res["frontend_then_step_graph"] = {"us_per_step": round(us, 1),
                                       "steps_per_s": round(1e6 / us, 1)}
    del fe
    torch.cuda.empty_cache()
    return res


def _dims_of(spec, w, x, head_level=False):
    return spec.Dims.make(B=w.B, L_cap=w.L_cap, L_max=w.L_cap, k_max=w.k, H_r=w.H_r, d_r=w.d_r,
                          n_layers=w.n_layers, H_q=w.H_q, H_kv=w.H_kv, d=w.d,
                          kr_stride_b=x["K_r"].stride(0), kv_stride_layer=x["K"].stride(0),
                          kv_stride_b=x["K"].stride(1), n_sets=w.H_kv if head_level else 1)


def _dims_attn(spec, w, x, outputs):
    return spec.Dims.make(B=w.B, L_cap=w.L_cap, L_max=w.L_cap, k_max=w.k, n_layers=w.n_layers,
                          H_q=w.H_q, H_kv=w.H_kv, d=w.d, kv_stride_layer=x["K"].stride(0),
                          kv_stride_b=x["K"].stride(1))


if __name__ == "__main__":
    main()
