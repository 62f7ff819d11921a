#!/usr/bin/env python3
"""Benchmark of the batched cGRU-attention scoring step on one MI355X.

One step = one nmt_score_batch call over the whole batch: the forward step
(H_i, P_i) <- NMT(H_{i-1}, E_i) of the paper's Section 5.1 for B
hypothesis rows, returning log p of one requested word per row over the full
target vocabulary plus the new states.  The default workload is the en->ru
shape: V = 100,000, E = 500, H = A = 1024, B = 2,000 rows over 20 source
sentences of length U{10..50} (padded to 50), fp32, seeded synthetic weights.

Prints ONE JSON line.  ``value`` is scored hypothesis-words per second
(rows / step time) with every input already resident in device memory.
``roofline`` reports the vocabulary-projection kernel (75% of the step's
flops) against the fp32 MFMA peak, from its own HIP-event duration measured
inside the timed region.  ``cpu_baseline`` times the fp64 oracle on a
bounded row sample on the host cores.

  python bench.py [--steps K] [--warmup W] [--config NAME] [--no-cpu-baseline]
  python bench.py --copy-probe BYTES   # plain copy kernel for counter calibration
  python bench.py --forest             # ScoreBatch over a prefix-tree forest (separate line)
  python bench.py --ensemble K         # K models per step and their parameter average (separate line)
  python bench.py --rescore            # stack rescoring of one sentence's synthetic stacks (separate line)
  python bench.py --library-gemms      # the vendor GEMM library on the step's shapes (context, separate line)
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

METRIC = "scored hypothesis-words/sec at V=100k, H=1024, B=2000; MFMA util %"
UNIT = "scored hypothesis-words/s"
PEAK_TFLOPS = {"f32": 157.3, "bf16": 2516.6}   # MI355X dense MFMA
PEAK_HBM_GBS = 8000.0
KERNEL_HEADERS = ("paper_1605_04809_amd/csrc/device.hpp", "paper_1605_04809_amd/csrc/internal.hpp")
KERNEL_FILE = "paper_1605_04809_amd/csrc/kernels.hip"
VOCAB_SECTION = ("// ------------------------------------------------ vocabulary projection",
                 "// ---------------------------------------------------- partials combine")
TRAFFIC_FILE = "profiles/vocab_lse_{workload}_traffic.txt"


def kernel_source_hash() -> str:
    """Hash of the vocabulary kernel's source section and the shared headers."""
    h = hashlib.sha256()
    for f in KERNEL_HEADERS:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    text = open(os.path.join(ROOT, KERNEL_FILE)).read()
    a, b = text.index(VOCAB_SECTION[0]), text.index(VOCAB_SECTION[1])
    h.update(text[a:b].encode())
    return h.hexdigest()[:16]


def step_flops(cfg, src_len, sent_id):
    """Flops one step computes (padding and never-stored logits excluded).
    With fp32 weights the products of the previous word's embedding with the
    first GRU's input weights (2 E 3H per row) and the readout's word weights
    (2 E E) are rows of per-word tables built with the model, and the
    products of the context with the second GRU's input weights (2 C 3H) and
    the readout's context weights (2 C E) are mixed by the attention from
    per-position projections of the annotations (2 L (3H + E) per row instead
    of the context's 2 L C): only what the step computes is counted."""
    E, H, A, C, V = cfg.E, cfg.H, cfg.A, cfg.C, cfg.V
    L = src_len[sent_id].astype(np.float64)
    pre = cfg.wtype == "f32"
    xe, xc = (0, 0) if pre else (E, C)      # the embedding's and the context's shares of K in the step
    per_row = (2 * (xe + H) * 3 * H         # first GRU
               + 2 * H * A                  # attention query
               + 2 * (H + xc) * 3 * H       # second GRU
               + 2 * (H + xe + xc) * E      # readout
               + 2 * E * V)                 # vocabulary projection
    mixed = 3 * H + E if pre else C         # columns the attention mixes per position
    attention = float(np.sum(3 * L * A + 2 * L * mixed))
    vocab = 2.0 * E * V * len(sent_id)
    return per_row * len(sent_id) + attention, vocab


def read_traffic(workload: str):
    """HBM bytes per vocab-kernel launch from the committed counter summary,
    or None if it is missing or was taken on different kernel sources."""
    path = os.path.join(ROOT, TRAFFIC_FILE.format(workload=workload))
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line:
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("kernel_source_sha256") != kernel_source_hash():
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(wl, min_seconds=10.0, max_seconds=30.0):
    """The fp64 oracle as it stands, on a bounded sample of rows of the workload:
    chunks of consecutive rows (wrapping round the batch) until at least
    min_seconds of scoring, sized to stay under max_seconds."""
    import oracle
    m = oracle.Model.from_workload(wl)
    ctx, pctx, _ = oracle.encode(m, wl.src_ids, wl.src_len)   # source initialisation, not timed
    B = len(wl.y_prev)
    threads = oracle.num_threads()
    done, elapsed, chunk, start_row = 0, 0.0, max(threads, 8), 0
    while elapsed < min_seconds:
        rows = (start_row + np.arange(chunk)) % B
        t0 = time.perf_counter()
        oracle.score_batch(m, ctx, pctx, wl.src_len, wl.s_prev[rows], wl.y_prev[rows], wl.sent_id[rows],
                           wl.req[rows], intermediates=False)
        dt = time.perf_counter() - t0
        elapsed += dt
        done += len(rows)
        start_row = (start_row + len(rows)) % B
        rate = len(rows) / dt
        chunk = int(max(threads, min(4 * B, rate * min(min_seconds - elapsed + 1.0, max_seconds - elapsed))))
    return {"value": done / elapsed, "unit": UNIT, "cores": threads, "kind": "oracle",
            "sample": f"{done} rows of the same workload (consecutive rows of the {B}-row batch, wrapping "
                      f"round it), one step each, fp64, {elapsed:.1f} s wall; source encoding excluded",
            "host": {"nproc": os.cpu_count(), "cpu_model": cpu_model(),
                     "OMP_NUM_THREADS": os.environ.get("OMP_NUM_THREADS")}}


def cpu_model() -> str:
    """The host CPU's model name (Linux /proc/cpuinfo), or "unknown"."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def copy_probe(nbytes: int, reps: int = 5):
    import torch
    n = nbytes // 4
    x = torch.ones(n, device="cuda")
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    for _ in range(reps):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": n * 4, "reps": reps}), flush=True)


def library_gemms(args, reps: int = 20):
    """The vendor GEMM library (torch.matmul: hipBLASLt) on the step's GEMM
    shapes at the workload's weight precision, plain products without the
    kernels' fused epilogues (no GRU cell, no tanh, no log-sum-exp; the vocab
    product writes its B x V logits), plus a large square product as the
    library's best case.  Context for the kernels' fractions of peak; none of
    this is on the scoring path."""
    import torch
    from paper_1605_04809_amd.workloads import CONFIGS
    cfg = CONFIGS[args.config]
    dt = torch.bfloat16 if cfg.wtype == "bf16" else torch.float32
    torch.backends.cuda.matmul.allow_tf32 = False
    B, E, H, A, V = cfg.B, cfg.E, cfg.H, cfg.A, cfg.V
    C = 2 * H
    shapes = {"query": (B, H, A), "gru1": (B, E + H, 3 * H), "gru2": (B, H + C, 3 * H),
              "readout": (B, H + E + C, E), "vocab": (B, E, V), "square_8192": (8192, 8192, 8192)}
    out = {}
    gen = torch.Generator(device="cuda").manual_seed(0)
    for name, (M, K, N) in shapes.items():
        a = torch.tanh(torch.randn(M, K, device="cuda", generator=gen)).to(dt)
        b = (torch.randn(K, N, device="cuda", generator=gen) * cfg.sigma_w).to(dt)
        c = torch.empty(M, N, device="cuda", dtype=dt)
        for _ in range(5):
            torch.matmul(a, b, out=c)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            torch.matmul(a, b, out=c)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        tf = 2.0 * M * K * N / (ms * 1e-3) / 1e12
        out[name] = {"M": M, "K": K, "N": N, "us": round(ms * 1e3, 2), "tflops": round(tf, 1),
                     "frac": round(tf / PEAK_TFLOPS[cfg.wtype], 4)}
        del a, b, c
    print(json.dumps({"metric": "library GEMM TFLOP/s on the step's shapes", "library": "torch.matmul (hipBLASLt)",
                      "dtype": cfg.wtype, "reps": reps, "config": {"workload": cfg.name}, "gemms": out}), flush=True)


def forest_bench(args):
    """ScoreBatch (Section 5.1, Figure 2) on a synthetic stack of the en->ru shape.

    Three ways to score the same (hypothesis, phrase) pairs:
      forest     one row per tree node with children, CSR requests, states
                 gathered on the device (nmt_score_forest);
      edge rows  the paper's batching: one row per tree edge at each depth
                 (H_{i-1} repeats a node's state once per outgoing edge);
      naive      one single-row query per word of every expansion (timed on a
                 sample of words and scaled to all of them).
    """
    import torch
    from paper_1605_04809_amd import binding as nb
    from paper_1605_04809_amd.workloads import CONFIGS, make_workload, make_forest

    cfg = CONFIGS[args.config]
    wl = make_workload(cfg, B=1)
    fw = make_forest(cfg, n_hyp=args.forest_hyps, seed=11, max_phrases=4, max_len=4, branch=3)
    model = nb.Model.from_workload(wl)
    cu = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    src = nb.nmt_encode(model, cu(wl.src_ids), wl.src_len)
    f = nb.Forest(fw.hyp_word, fw.hyp_sent, fw.pair_hyp, fw.phrases)
    sh = f.shape()
    hs = cu(fw.hyp_state)
    pair_logp = torch.empty(len(fw.phrases), device="cuda")
    ws = torch.empty(nb.nmt_forest_workspace_bytes(model, f), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()

    def timed(fn, reps):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    ms_forest = timed(lambda: nb.nmt_score_forest(model, src, f, hs, pair_logp, workspace=ws, stream=stream),
                      args.steps)
    # The paper's edge rows: each tree edge of a level is a row of its own,
    # repeating its source node's input (Section 5.1: H_0 = [h0; h0; h1; h1]).
    # An edge row's new state is the input state of its child edges, so a
    # deeper edge gathers its state from its parent edge's output row.
    levels = [f.level(d) for d in range(1, sh["depth"] + 1)]
    H = cfg.H
    paths = f.pair_paths()
    src_edge = np.full(sh["n_req"], -1, np.int64)
    for k in range(1, sh["depth"]):
        live = paths[:, k] >= 0
        src_edge[paths[live, k]] = paths[live, k - 1]
    edge_in, q0 = [], 0
    for d, lv in enumerate(levels):
        rows = np.repeat(np.arange(lv["y_prev"].size), np.diff(lv["req_off"]))
        state_row = lv["state_row"][rows] if d == 0 else src_edge[q0:q0 + rows.size]
        edge_in.append(dict(state_row=cu(state_row.astype(np.int32)), y=cu(lv["y_prev"][rows]),
                            sent=cu(lv["sent_id"][rows]), off=cu(np.arange(rows.size + 1, dtype=np.int32)),
                            req=cu(lv["req"]), n=rows.size, q0=q0))
        q0 += rows.size
    max_e = max(e["n"] for e in edge_in)
    edge_states = torch.empty((sh["n_req"], H), device="cuda")
    e_logp = torch.empty(sh["n_req"], device="cuda")
    ws_e = torch.empty(nb.nmt_score_workspace_bytes(model, max_e), dtype=torch.uint8, device="cuda")

    def edge_rows():
        for d, e in enumerate(edge_in):
            pool = hs if d == 0 else edge_states
            nb.nmt_score_forest_step(model, src, pool, e["state_row"], e["y"], e["sent"], e["off"], e["req"],
                                     e_logp[e["q0"]:e["q0"] + e["n"]], edge_states[e["q0"]:e["q0"] + e["n"]],
                                     workspace=ws_e, stream=stream)
    ms_edges = timed(edge_rows, max(2, args.steps // 2))
    # both batchings must give every edge the same log-probability
    req_logp = torch.empty(sh["n_req"], device="cuda")
    nb.nmt_score_forest(model, src, f, hs, pair_logp, req_logp=req_logp, workspace=ws, stream=stream)
    edge_rows()
    torch.cuda.synchronize()
    same = float((req_logp - e_logp).abs().max())
    # naive: one single-row query per word, on a sample
    n_words = sum(len(p) for p in fw.phrases)
    sample = min(64, n_words)
    s1 = hs[:1].contiguous()
    y1, sid1, r1 = cu(fw.hyp_word[:1]), cu(fw.hyp_sent[:1]), cu(np.array([fw.phrases[0][0]], np.int32))
    lp1, sn1 = torch.empty(1, device="cuda"), torch.empty((1, H), device="cuda")
    ws1 = torch.empty(nb.nmt_score_workspace_bytes(model, 1), dtype=torch.uint8, device="cuda")
    ms_one = timed(lambda: nb.nmt_score_batch(model, src, s1, y1, sid1, r1, lp1, sn1, workspace=ws1, stream=stream),
                   sample)
    out = {"metric": "ScoreBatch scored (hypothesis, phrase) pairs/s", "value": len(fw.phrases) / (ms_forest * 1e-3),
           "unit": "pairs/s", "higher_is_better": True, "dtype": cfg.wtype, "data": "synthetic",
           "config": {"workload": f"forest on {cfg.name}", "hypotheses": args.forest_hyps, "pairs": len(fw.phrases),
                      "words": n_words, "edges": sh["n_req"], "forest_rows": sh["n_rows"], "depth": sh["depth"],
                      "rows_per_level": [int(lv["y_prev"].size) for lv in levels],
                      "edges_per_level": [int(lv["req"].size) for lv in levels]},
           "ms_forest": ms_forest, "ms_edge_rows": ms_edges,
           "ms_naive_per_word_estimate": ms_one * n_words, "naive_queries": n_words,
           "forest_queries": sh["depth"],
           "speedup_vs_edge_rows": ms_edges / ms_forest, "speedup_vs_naive": ms_one * n_words / ms_forest,
           "max_abs_diff_forest_vs_edge_rows": same}
    f.close()
    src.close()
    model.close()
    print(json.dumps(out), flush=True)


def ensemble_bench(args):
    """Several models per step (Sections 5 and 6.2): K models of the workload's
    shape as separate features scoring the same rows in one
    nmt_score_ensemble call, and the element-wise parameter average of the
    same K models (Section 6.3, nmt_model_average)."""
    import torch
    from paper_1605_04809_amd import binding as nb
    from paper_1605_04809_amd.workloads import CONFIGS, make_workload

    cfg = CONFIGS[args.config]
    K = args.ensemble
    wl = make_workload(cfg)
    B = cfg.B
    cu = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    models = [nb.Model.from_workload(wl)]
    for k in range(1, K):
        other = make_workload(cfg.replace(seed=cfg.seed + 1000 * k), B=1)
        models.append(nb.Model(other.params, cfg.V_src, cfg.V, cfg.E, cfg.H, cfg.A, cfg.wtype))
    srcs = [nb.nmt_encode(m, cu(wl.src_ids), wl.src_len) for m in models]
    s_prev = [cu(wl.s_prev) for _ in range(K)]
    s_new = [torch.empty_like(x) for x in s_prev]
    y_prev, sent_id, req = cu(wl.y_prev), cu(wl.sent_id), cu(wl.req)
    logp = torch.empty((K, B), device="cuda")
    score = torch.empty(B, device="cuda")
    ws = torch.empty(nb.nmt_ensemble_workspace_bytes(models, B), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    weights = [1.0 / K] * K

    def step():
        nb.nmt_score_ensemble(models, srcs, s_prev, y_prev, sent_id, req, logp, s_new, weights=weights,
                              score=score, workspace=ws, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    if not bool(torch.isfinite(score).all()):
        raise SystemExit("non-finite ensemble scores")
    # parameter averaging: read K models, write one (host clock; the call waits for its stream)
    avg = nb.nmt_model_average(models, stream=stream)
    avg.close()
    reps = 3
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        nb.nmt_model_average(models, stream=stream).close()
    ms_avg = (time.perf_counter() - t0) / reps * 1e3
    wbytes = (2 if cfg.wtype == "bf16" else 4) * sum(
        int(np.prod(v.shape)) for v in wl.params.values())
    out = {"metric": f"ensemble of {K} models as separate features: scored hypothesis-words/s",
           "value": B / (ms * 1e-3), "unit": "hypothesis-words/s (each scored by every model)",
           "higher_is_better": True, "dtype": cfg.wtype, "data": "synthetic",
           "config": {"workload": f"{K} x {cfg.name}", "models": K, "B": B, "V": cfg.V, "H": cfg.H},
           "ms_per_step": ms, "model_words_per_s": K * B / (ms * 1e-3),
           "average": {"ms": ms_avg, "models": K, "param_bytes_per_model": wbytes,
                       "GBps_read_plus_write": (K + 1) * wbytes / (ms_avg * 1e-3) / 1e9,
                       "timing": "host clock around the call, which allocates the new model and waits"}}
    for x in srcs:
        x.close()
    for m in models:
        m.close()
    print(json.dumps(out), flush=True)


def rescore_bench(args):
    """Stack rescoring (Section 5.3, Figure 4) of one sentence's synthetic
    stacks (stack limit 1000, the paper's setting) with the workload's model:
    each stack's predecessors go through one nmt_rescore_stack call, which
    returns the scores to the host as the decoder needs them."""
    import torch
    from paper_1605_04809_amd import binding as nb
    from paper_1605_04809_amd.workloads import CONFIGS, make_workload, make_stacks

    cfg = CONFIGS[args.config]
    wl = make_workload(cfg, B=1)
    sent = 0
    J = int(wl.src_len[sent])
    sw = make_stacks(cfg, src_len=J, stack_size=args.stack_size, seed=13, sent=sent)
    cu = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    model = nb.Model.from_workload(wl)
    s0 = torch.empty((cfg.S, cfg.H), device="cuda")
    src = nb.nmt_encode(model, cu(wl.src_ids), wl.src_len, s0)
    n_total = sw.n_roots + sum(len(p) for p, _ in sw.stacks)
    # the decoder hands each stack over as flat arrays (parents, phrase offsets, words)
    flat = [(np.ascontiguousarray(p, dtype=np.int32),) + nb.phrases_csr(phr) for p, phr in sw.stacks]

    def run():
        r = nb.Rescorer([model], [src], [s0], n_total)
        per = []
        for parents, off, words in flat:
            t0 = time.perf_counter()
            lp, _ = r.rescore_csr(parents, off, words)
            per.append((time.perf_counter() - t0) * 1e3)
            if not np.all(np.isfinite(lp)):
                raise SystemExit("non-finite rescoring scores")
        shape = r.info()
        r.close()
        return per, shape

    run()  # warm-up (also grows the scratch buffers once)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    per, _ = run()
    ms = (time.perf_counter() - t0) * 1e3
    hyps = sum(len(p) for p, _ in sw.stacks)
    words = sum(len(ph) for _, phr in sw.stacks for ph in phr)
    pairs = sum(len({(int(a), tuple(b)) for a, b in zip(p, phr)}) for p, phr in sw.stacks)
    out = {"metric": "stack rescoring: rescored hypotheses/s", "value": hyps / (ms * 1e-3),
           "unit": "hypotheses/s", "higher_is_better": True, "dtype": cfg.wtype, "data": "synthetic",
           "config": {"workload": f"stack rescoring on {cfg.name}", "source_len": J, "stacks": len(sw.stacks),
                      "stack_limit": args.stack_size, "hypotheses": hyps, "distinct_predecessors": pairs,
                      "phrase_words": words},
           "ms_sentence": ms, "ms_per_stack_max": max(per), "ms_per_stack_mean": ms / len(sw.stacks),
           "phrase_words_per_s": words / (ms * 1e-3),
           "timing": "host clock around each nmt_rescore_stack call on the flattened stack (it returns the scores to the host)"}
    src.close()
    model.close()
    print(json.dumps(out), flush=True)


EXTRA_WORKLOADS = ("tiny", "ruen_b1000", "phrase_h500", "bf16_b4096")


def _events_pass(torch, stream, fn, k):
    """k calls of fn with an event before each and after the last, on the
    launch stream: per-call times (ms) and the whole pass (ms)."""
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(k + 1)]
    torch.cuda.synchronize()
    ev[0].record(stream)
    for i in range(k):
        fn()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(k)]
    return per, ev[0].elapsed_time(ev[k])


def _plain_pass(torch, stream, fn, k):
    """k calls of fn bracketed by synchronisation and two events (ms total)."""
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(stream)
    for _ in range(k):
        fn()
    t1.record(stream)
    torch.cuda.synchronize()
    return t0.elapsed_time(t1)


def phrase_forest(wl):
    """The phrase workload as ScoreBatch input (Section 5.1, Figure 2): each
    hypothesis (its last word, sentence and state) with its one target phrase;
    the forest's level d holds the hypotheses whose phrase has at least d
    tokens, so the batch shrinks as phrases end."""
    phrases = [list(map(int, wl.phrase_tok[b, :wl.phrase_len[b]])) for b in range(len(wl.y_prev))]
    return wl.y_prev, wl.sent_id, np.arange(len(phrases), dtype=np.int32), phrases


def bench_workload(name, args, cpu_seconds, headline=False):
    """Time one workload: W warm-up steps, a pass of K steps with an event
    around each of the library's kernels (the roofline's kernel duration), a
    plain pass of K steps between two events (throughput), and a pass with an
    event between steps (median step time).  A step of the phrase workload is
    its whole ScoreBatch: one batched step per tree depth, the batch shrinking
    as phrases end, and the per-phrase sums (nmt_score_forest)."""
    import torch
    from paper_1605_04809_amd import binding as nb
    from paper_1605_04809_amd.workloads import CONFIGS, make_workload

    cfg = CONFIGS[name]
    wl = make_workload(cfg)
    model = nb.Model.from_workload(wl)
    cu = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    src_ids = cu(wl.src_ids)
    src = nb.nmt_encode(model, src_ids, wl.src_len)
    stream = torch.cuda.current_stream()

    # Source initialisation (off the scoring loop), timed on its own: host
    # wall clock around encode + synchronise, the source's allocation included.
    torch.cuda.synchronize()
    enc_ms = []
    for _ in range(3):
        t_enc = time.perf_counter()
        extra = nb.nmt_encode(model, src_ids, wl.src_len, stream=stream)
        torch.cuda.synchronize()
        enc_ms.append((time.perf_counter() - t_enc) * 1e3)
        extra.close()

    if cfg.phrase_max:
        hyp_word, hyp_sent, pair_hyp, phrases = phrase_forest(wl)
        forest = nb.Forest(hyp_word, hyp_sent, pair_hyp, phrases)
        sh = forest.shape()
        levels = [forest.level(d) for d in range(1, sh["depth"] + 1)]
        rows_per_level = [int(lv["y_prev"].size) for lv in levels]
        hs = cu(wl.s_prev)
        out_logp = torch.empty(len(phrases), device="cuda")
        ws = torch.empty(nb.nmt_forest_workspace_bytes(model, forest), dtype=torch.uint8, device="cuda")
        calls_per_step = sh["depth"]
        scored = sh["n_req"]                      # requested tokens over all levels
        row_sent = np.concatenate([lv["sent_id"] for lv in levels])

        def step():
            nb.nmt_score_forest(model, src, forest, hs, out_logp, workspace=ws, stream=stream)
        check = out_logp
    else:
        B = cfg.B
        s_prev, y_prev, sent_id, req = cu(wl.s_prev), cu(wl.y_prev), cu(wl.sent_id), cu(wl.req)
        logp = torch.empty(B, device="cuda")
        logZ = torch.empty(B, device="cuda")
        s_new = torch.empty((B, cfg.H), device="cuda")
        ws = torch.empty(nb.nmt_score_workspace_bytes(model, B), dtype=torch.uint8, device="cuda")
        calls_per_step = 1
        scored = B
        row_sent = wl.sent_id
        rows_per_level = [B]

        def step():
            nb.nmt_score_batch(model, src, s_prev, y_prev, sent_id, req, logp, s_new, logZ, workspace=ws,
                               stream=stream)
        check = logp

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if nb.nmt_stream_status(model) != nb.NMT_OK:
        raise SystemExit(f"{name}: device reported an id error during warm-up")

    K = args.steps
    nb.nmt_profile_begin(model, K * calls_per_step)
    ms_total_prof = _plain_pass(torch, stream, step, K)
    phases = nb.nmt_profile_end(model, stream)
    assert phases["steps"] == K * calls_per_step
    ms_total = _plain_pass(torch, stream, step, K)
    per_step, _ = _events_pass(torch, stream, step, K)
    if not bool(torch.isfinite(check).all()):
        raise SystemExit(f"{name}: non-finite log-probabilities")

    ms_step = ms_total / K
    graph = None
    if not cfg.phrase_max and cfg.B <= 128:
        # Small batches are launch-bound: the same step captured once in a
        # HIP graph (torch.cuda.CUDAGraph over the library's launches on the
        # capture stream) and replayed, K replays between two events.
        cap = torch.cuda.Stream()
        cap.wait_stream(stream)
        with torch.cuda.stream(cap):
            for _ in range(3):
                nb.nmt_score_batch(model, src, s_prev, y_prev, sent_id, req, logp, s_new, logZ, workspace=ws)
        stream.wait_stream(cap)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            nb.nmt_score_batch(model, src, s_prev, y_prev, sent_id, req, logp, s_new, logZ, workspace=ws)
        for _ in range(args.warmup):
            g.replay()
        per_g, tot_g = _events_pass(torch, stream, g.replay, K)
        graph = {"ms_per_step": tot_g / K, "ms_per_step_median": float(np.median(per_g)),
                 "note": "the step captured once in a HIP graph and replayed (same kernels, same inputs)"}
    total_flops, vocab_flops = step_flops(cfg, wl.src_len, row_sent)
    peak = PEAK_TFLOPS[cfg.wtype]
    vocab_ms = phases["vocab"] / K
    achieved = vocab_flops / (vocab_ms * 1e-3) / 1e12
    res = {
        "value": scored / (ms_step * 1e-3),
        "unit": UNIT,
        "ms_per_step": ms_step,
        "ms_per_step_median": float(np.median(per_step)),
        "ms_per_step_p10_p90": [float(np.percentile(per_step, 10)), float(np.percentile(per_step, 90))],
        "dtype": cfg.wtype,
        "config": {"workload": cfg.name, "V": cfg.V, "E": cfg.E, "H": cfg.H, "A": cfg.A,
                   "S": cfg.S, "src_len": f"U{{{cfg.len_lo}..{cfg.len_hi}}}", "Tpad": cfg.Tpad,
                   "weights": cfg.wtype, "rows_per_step": rows_per_level},
        "roofline": {"bound": "mfma", "kernel": "k_vocab_lse", "achieved": achieved, "peak": peak,
                     "unit": "TFLOP/s", "frac": achieved / peak,
                     "traffic": read_traffic(cfg.name), "algorithmic_flops_per_step": vocab_flops,
                     "launches_per_step": calls_per_step, "avg_launch_ms": vocab_ms / calls_per_step},
        "step_tflops": total_flops / (ms_step * 1e-3) / 1e12,
        "mfma_util_step_pct": 100.0 * total_flops / (ms_step * 1e-3) / 1e12 / peak,
        "phase_ms": {k: v / K for k, v in phases.items() if k != "steps"},
        "ms_per_step_with_phase_events": ms_total_prof / K,
        "encode": {"ms": float(np.median(enc_ms)), "sentences": cfg.S,
                   "ms_per_sentence": float(np.median(enc_ms)) / cfg.S},
    }
    if cfg.wtype == "f32":
        res["precomputed"] = {
            "per_model": "per-word tables Emb.W_x [V x 3H] and Emb.W_y [V x E], built once at model creation",
            "per_source": "the annotations' projections ctx.[W_c(GRU2) | W_c(readout)] [S x Tpad x (3H+E)], built "
                          "with the keys when the source is encoded (inside encode.ms)",
            "step": "gathers the tables' rows by previous word and mixes the projections with the attention "
                    "weights; step_tflops counts only what the step computes"}
    if graph:
        res["graph"] = graph
    if cfg.phrase_max:
        res["config"].update(hypotheses=cfg.B, phrase_tokens="U{1..%d}" % cfg.phrase_max, scored_tokens=scored)
        res["timing"] = ("one step = nmt_score_forest over the 500 phrases: one batched step per depth, the "
                         "batch shrinking as phrases end, states kept on the device, per-phrase sums; the "
                         "forest's index arrays (%d bytes, built on the host) are uploaded inside each call"
                         % (4 * (4 * sh["n_rows"] + sh["depth"] + sh["n_req"] + sh["depth"] * len(phrases))))
    else:
        res["config"]["B"] = cfg.B
    if cpu_seconds > 0:
        res["cpu_baseline"] = cpu_baseline(wl, min_seconds=cpu_seconds, max_seconds=max(30.0, 3 * cpu_seconds))
    if cfg.phrase_max:
        forest.close()
    src.close()
    model.close()
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="enru_b2000")
    ap.add_argument("--only", action="store_true", help="time only --config (no other workloads in the line)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", type=int, default=0)
    ap.add_argument("--print-kernel-hash", action="store_true")
    ap.add_argument("--forest", action="store_true")
    ap.add_argument("--forest-hyps", type=int, default=1000)
    ap.add_argument("--ensemble", type=int, default=0, help="K models per step (separate line)")
    ap.add_argument("--rescore", action="store_true", help="stack rescoring of one sentence (separate line)")
    ap.add_argument("--stack-size", type=int, default=1000)
    ap.add_argument("--library-gemms", action="store_true", help="vendor GEMM library on the step's shapes")
    args = ap.parse_args()
    if args.print_kernel_hash:
        print(kernel_source_hash())
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              f"(asked for --gpus {args.gpus}, WORLD_SIZE={world}).", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.forest:
        forest_bench(args)
        return
    if args.ensemble:
        ensemble_bench(args)
        return
    if args.rescore:
        rescore_bench(args)
        return
    if args.library_gemms:
        library_gemms(args)
        return

    cpu = 0.0 if args.no_cpu_baseline else 10.0
    head = bench_workload(args.config, args, cpu, headline=True)
    out = {
        "metric": METRIC,
        "value": head["value"],
        "unit": UNIT,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": head["dtype"],
        "data": "synthetic: seeded N(0, 0.01) random-init weights of the paper's shape, no trained model",
        "config": head["config"],
        "roofline": head["roofline"],
    }
    out["roofline"]["algorithmic_flops_per_launch"] = out["roofline"].pop("algorithmic_flops_per_step") / \
        out["roofline"]["launches_per_step"]
    if "cpu_baseline" in head:
        out["cpu_baseline"] = head["cpu_baseline"]
    for k in ("ms_per_step_median", "ms_per_step_p10_p90", "step_tflops", "mfma_util_step_pct", "phase_ms",
              "ms_per_step_with_phase_events", "encode", "graph"):
        if k in head:
            out[k] = head[k]
    out["mfma_util_vocab_pct"] = 100.0 * out["roofline"]["frac"]
    if not args.only:
        # The other workloads, each timed the same way in this process (their
        # CPU baselines on shorter samples, so the run stays within minutes).
        out["workloads"] = {}
        for name in EXTRA_WORKLOADS:
            if name == args.config:
                continue
            r = bench_workload(name, args, 0.0 if args.no_cpu_baseline else 4.0)
            r["roofline"]["algorithmic_flops_per_launch"] = r["roofline"].pop("algorithmic_flops_per_step") / \
                r["roofline"]["launches_per_step"]
            out["workloads"][name] = r
            print(f"# {name}: {r['ms_per_step']:.4f} ms per step, {r['value']:.4g} {UNIT}", file=sys.stderr,
                  flush=True)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
