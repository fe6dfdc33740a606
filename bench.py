"""Benchmark of one GVA decode step on one MI355X.

A step is the whole decode path of Algorithm 1 for one batch: append the
step's new value rows and rotated positional key at position len-1, absorb
and rotate the query, attend over every cached row in splits, and merge the
splits.  The attention call takes the current token's rows (v_new, kr_new):
the workgroup that owns position len-1 stores them into the caches and
attends over them in the same launch, so the append costs no launch of its
own.  Inputs are seeded synthetic tensors already resident in HBM before
the timed region starts.

Prints ONE JSON line.  ``value`` is whole-step throughput in GB/s of
algorithmic bytes (every cached value / positional-key row read once, M and
q read once, new rows read+written once, fp32 output written once) divided
by the measured step time.

  python bench.py [--steps K] [--warmup W] [--workload b32_t8k] [--splits S]
                  [--absorb auto|fused|separate] [--no-cpu-baseline]
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import gva_inputs  # noqa: E402
from paper_2609_13285_amd import gva, traffic  # noqa: E402

METRIC = "decode attention GB/s (fraction of HBM peak) and tokens/s"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, AMD's published figure
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak, AMD's published figure
SIDE_WARM_S = 0.5          # minimum untimed warm-up of each side comparison, seconds
SETTLE_STEPS = 300         # steps after which a fresh process's step time has settled
# the decode kernel's sources (the traffic record is valid only for these)
KERNEL_SRCS = [os.path.join(ROOT, "paper_2609_13285_amd", "csrc", f)
               for f in ("gva_common.h", "gva_decode.hip")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_decode_b32_t8k.json")


def metric_label(w) -> str:
    """The metric named for the workload it is measured on: batch, cached
    rows (K = 1024) and storage dtype, e.g. "B=32 T=8K bf16"."""
    def rows(n):
        return f"{n // 1024}K" if n % 1024 == 0 else str(n)
    if w.lengths == "full":
        span = rows(w.t_max)
    elif w.lengths == "uniform_half":
        span = f"{rows(w.t_max // 2)}..{rows(w.t_max)}"
    else:
        span = f"{rows(w.len_min)}..{rows(w.t_max)}"
    return f"{METRIC}, B={w.batch} T={span} {w.dtype}"


def kernel_sha() -> str:
    h = hashlib.sha256()
    for path in KERNEL_SRCS:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str, splits: int):
    """HBM bytes per decode launch from committed rocprofv3 counters, if they
    were taken on the current kernel source with the same launch shape."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_sha") != kernel_sha() or rec.get("workload") != workload \
            or rec.get("num_splits") != splits:
        return None
    return rec.get("hbm_bytes_per_launch")


def copy_calibration(mb: int, reps: int = 5):
    """A plain device copy of known size, for scaling FETCH_SIZE/WRITE_SIZE."""
    n = mb * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n * 4, "reps": reps}))


def _pmc_means(csv_path: str, counter: str):
    """Mean of one counter per kernel name in a rocprofv3 counter CSV."""
    import csv
    acc = {}
    with open(csv_path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            acc.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
    return {k: sum(v) / len(v) for k, v in acc.items()}


def write_traffic(fetch_csv, write_csv, copy_fetch_csv, copy_write_csv, workload, splits, copy_mb):
    """HBM bytes per decode launch from FETCH_SIZE / WRITE_SIZE, each scaled
    by what the same counter reads for a plain device copy of known size."""
    def pick(means, key):
        hits = [v for k, v in means.items() if key in k]
        if len(hits) != 1:
            raise SystemExit(f"{len(hits)} kernels named like {key} in the counter file (need one)")
        return hits[0]
    copy_bytes = copy_mb * (1 << 20)
    f_copy = pick(_pmc_means(copy_fetch_csv, "FETCH_SIZE"), "copyBuffer")
    w_copy = pick(_pmc_means(copy_write_csv, "WRITE_SIZE"), "copyBuffer")
    f_dec = pick(_pmc_means(fetch_csv, "FETCH_SIZE"), "decode_bf16_kernel")
    w_dec = pick(_pmc_means(write_csv, "WRITE_SIZE"), "decode_bf16_kernel")
    rec = {"workload": workload, "num_splits": splits, "kernel_sha": kernel_sha(),
           "fetch_scale_bytes_per_unit": copy_bytes / f_copy,
           "write_scale_bytes_per_unit": copy_bytes / w_copy,
           "fetch_bytes_per_launch": f_dec * copy_bytes / f_copy,
           "write_bytes_per_launch": w_dec * copy_bytes / w_copy}
    rec["hbm_bytes_per_launch"] = round(rec["fetch_bytes_per_launch"] + rec["write_bytes_per_launch"])
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))


def cpu_baseline(w, inp, seq, pos, budget_s: float = 20.0, min_s: float = 10.0):
    """The fp64 oracle on the host cores, on a bounded sample of sequences.

    Sequences are taken one at a time until ``budget_s`` of oracle time is
    spent; when the whole batch takes less than ``min_s``, whole passes over
    it are repeated until ``min_s`` is reached, so the rate rests on about
    ten seconds of CPU work either way."""
    import oracle
    threads = oracle.max_threads()
    v = inp["v"].clone()
    kr = inp["kr"].clone()
    oracle.append(v, kr, inp["v_new"], inp["kr_new"], seq, pos, w.rope_base)
    esize = 2 if w.dtype == "bf16" else 4

    def one(b):
        sl = slice(b, b + 1)
        t0 = time.perf_counter()
        o, _ = oracle.decode(inp["q"][sl], inp["m"], v[sl], kr[sl], inp["lens"][sl],
                             rope_base=w.rope_base, n_threads=threads)
        dt = time.perf_counter() - t0
        nb = traffic.decode_bytes(inp["lens"][sl], 1, w.n_heads, w.n_groups, w.d_v,
                                  w.d_c, w.d_r, esize)
        return o[0], dt, nb

    order = list(range(w.batch))
    done, t_used, nbytes = [], 0.0, 0
    o_all = {}
    while order and t_used < budget_s:
        b = order.pop(0)
        o_all[b], dt, nb = one(b)
        done.append(b)
        t_used += dt
        nbytes += nb
    passes = 1
    if not order:
        while t_used < min_s:
            for b in range(w.batch):
                _, dt, nb = one(b)
                t_used += dt
                nbytes += nb
            passes += 1
    # the same oracle on one thread, one sequence (the longest), for scale
    b1 = int(inp["lens"].argmax())
    sl = slice(b1, b1 + 1)
    t0 = time.perf_counter()
    oracle.decode(inp["q"][sl], inp["m"], v[sl], kr[sl], inp["lens"][sl], rope_base=w.rope_base,
                  n_threads=1)
    t1 = time.perf_counter() - t0
    nb1 = traffic.decode_bytes(inp["lens"][sl], 1, w.n_heads, w.n_groups, w.d_v, w.d_c, w.d_r, esize)
    rec = {"value": nbytes / t_used / 1e9, "unit": "GB/s", "cores": threads, "kind": "oracle",
           "value_1_thread": nb1 / t1 / 1e9,
           "seconds": round(t_used, 3),
           "sample": f"fp64 oracle decode of {len(done)} of {w.batch} sequences "
                     f"(all {w.n_heads} heads, full length) after the step's append"
                     + (f", {passes} passes" if passes > 1 else "")}
    return rec, o_all


MALL_BYTES = 256 << 20


def warm(fns, calls: int, seconds: float) -> None:
    """Untimed calls of each of fns in turn: at least ``calls`` each, and
    until ``seconds`` of wall time have passed.  The side comparisons use it
    so that their kernels are timed past the device's power-management ramp
    in a fresh process (an MFMA-bound launch runs up to ~25% slower for its
    first tens of milliseconds), whatever --warmup the headline step uses."""
    t0 = time.perf_counter()
    i = 0
    while i < calls or time.perf_counter() - t0 < seconds:
        for f in fns:
            f(i)
        i += 1
        if i % 8 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()


def timed(step, steps: int, stream) -> float:
    """Mean ms per step over ``steps`` calls of step(i), bracketed by events
    on ``stream`` with no events inside."""
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(stream)
    for i in range(steps):
        step(i)
    t_end.record(stream)
    torch.cuda.synchronize()
    return t_start.elapsed_time(t_end) / steps


def layer_stack(args, w, inp, d, S, split_rows, fused, dec_b):
    """An N-layer decode step (the step of one token through N attention
    layers, each with its own caches, query, maps and workspace): one
    gva_decode_step call per layer, timed three ways -- through the Python
    binding on every call, with the calls marshalled once (gva.prepare), and
    as one captured HIP graph per step.  The library allocates, synchronises
    and clears nothing, so its launches are captured as they are.  Sets of
    layer caches rotate like the single-layer caches so no step finds its
    rows in the MALL."""
    n = args.layers
    n_sets = min(8, max(2, math.ceil(2 * MALL_BYTES / (n * dec_b))))
    v_t, kr_t = gva.tiled(inp["v"]), gva.tiled(inp["kr"])
    small = {k: inp[k].cuda() for k in ("q", "m", "lens", "v_new", "kr_new")}
    layers = []
    for _ in range(n):
        layer = {k: t.clone() for k, t in small.items()}
        layer["caches"] = [(v_t.cuda(), kr_t.cuda()) for _ in range(n_sets)]
        layer["bufs"] = gva.DecodeBuffers(d, S)
        layer["ws"] = gva.workspace_for(d, S, split_rows)
        layers.append(layer)
    del v_t, kr_t

    def run(i, st=None):
        st = st if st is not None else torch.cuda.current_stream()   # the capture stream while capturing
        for L in layers:
            vc, kc = L["caches"][i % n_sets]
            gva.gva_decode_step(d, L["q"], L["m"], vc, kc, L["lens"], S, L["bufs"].o, L["bufs"].lse,
                                workspace=L["ws"], v_new=L["v_new"],
                                kr_new=L["kr_new"] if w.d_r > 0 else None, split_rows=split_rows, stream=st)

    stream = torch.cuda.current_stream()
    for i in range(args.warmup):
        run(i)
    eager_ms = timed(run, args.steps, stream)
    prepared = [gva.prepare(run, c, stream) for c in range(n_sets)]
    for i in range(args.warmup):
        prepared[i % n_sets]()
    prepared_ms = timed(lambda i: prepared[i % n_sets](), args.steps, stream)
    graphs = []
    for c in range(n_sets):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            run(c)
        graphs.append(g)
    for i in range(args.warmup):
        graphs[i % n_sets].replay()
    graph_ms = timed(lambda i: graphs[i % n_sets].replay(), args.steps, stream)
    launches = n * ((0 if fused else 1) + 1 + (1 if S > 1 else 0))
    return {"n_layers": n, "launches_per_step": launches, "cache_sets": n_sets,
            "eager_ms_per_step": round(eager_ms, 5), "prepared_ms_per_step": round(prepared_ms, 5),
            "graph_ms_per_step": round(graph_ms, 5),
            "eager_us_per_layer": round(eager_ms * 1000 / n, 2),
            "prepared_us_per_layer": round(prepared_ms * 1000 / n, 2),
            "graph_us_per_layer": round(graph_ms * 1000 / n, 2),
            "graph_GBps": round(n * dec_b / (graph_ms * 1e-3) / 1e9, 1)}


def gqa_comparison(args, w, inp, d, S, split_rows, fused, dev, caches, stream):
    """Attention only (the caches as stored, no append), GVA against the
    matched GQA baseline on the same values, lengths and query content
    slice, each rotating through its own cache copies; both merge their
    splits with gva_combine."""
    n = len(caches)
    k_gqa = inp["k_gqa"] if "k_gqa" in inp else gva_inputs.gqa_keys(w, args.seed)
    k_tiled = gva.tiled(k_gqa)
    del k_gqa
    kcaches = [k_tiled.cuda() for _ in range(n)]
    del k_tiled
    bufs = gva.DecodeBuffers(d, S)
    q_abs = torch.empty(w.batch, w.n_heads, w.d_v, dtype=torch.float32, device="cuda")
    q_rot = torch.empty(w.batch, w.n_heads, w.d_r, dtype=torch.float32, device="cuda")

    def gva_calls(i):
        vc, kc = caches[i]
        if fused:
            gva.gva_decode_attention(d, vc, kc, dev["lens"], S, bufs.o_part, bufs.lse_part,
                                     q=dev["q"], m=dev["m"], split_rows=split_rows, stream=stream)
        else:
            gva.gva_absorb_query(d, dev["q"], dev["m"], dev["lens"], q_abs, q_rot, stream)
            gva.gva_decode_attention(d, vc, kc, dev["lens"], S, bufs.o_part, bufs.lse_part,
                                     q_abs=q_abs, q_rot=q_rot if w.d_r > 0 else None,
                                     split_rows=split_rows, stream=stream)
        if S > 1:
            gva.gva_combine(d, bufs.o_part, bufs.lse_part, S, bufs.o, bufs.lse, stream)

    def gqa_calls(i):
        gva.gva_gqa_decode_attention(d, dev["q"], kcaches[i], caches[i][0], dev["lens"], S,
                                     bufs.o_part, bufs.lse_part, split_rows=split_rows, stream=stream)
        if S > 1:
            gva.gva_combine(d, bufs.o_part, bufs.lse_part, S, bufs.o, bufs.lse, stream)

    gva_fns = [gva.prepare(gva_calls, c) for c in range(n)]
    gqa_fns = [gva.prepare(gqa_calls, c) for c in range(n)]

    def gva_attn(i):
        gva_fns[i % n]()

    def gqa_attn(i):
        gqa_fns[i % n]()

    warm([gva_attn, gqa_attn], args.warmup, SIDE_WARM_S)
    t_gva = timed(gva_attn, args.steps, stream)
    t_gqa = timed(gqa_attn, args.steps, stream)
    elem = 2
    out_b = w.batch * w.n_heads * w.d_v * 4
    b_gva = traffic.decode_bytes(inp["lens"], w.batch, w.n_heads, w.n_groups, w.d_v, w.d_c,
                                 w.d_r, elem) + out_b
    b_gqa = traffic.gqa_decode_bytes(inp["lens"], w.batch, w.n_heads, w.n_groups, w.d_v, elem) + out_b
    del kcaches
    return {"what": "attention only (caches as stored), GVA vs matched GQA, same split plan",
            "gva_ms": round(t_gva, 5), "gqa_ms": round(t_gqa, 5),
            "time_ratio_gva_over_gqa": round(t_gva / t_gqa, 4),
            "gva_bytes": b_gva, "gqa_bytes": b_gqa, "byte_ratio_gva_over_gqa": round(b_gva / b_gqa, 4),
            "gva_GBps": round(b_gva / (t_gva * 1e-3) / 1e9, 1),
            "gqa_GBps": round(b_gqa / (t_gqa * 1e-3) / 1e9, 1)}


def rope_comparison(args, w, inp, S, split_rows, dev, caches, stream):
    """GVA with ordinary RoPE (keys reconstructed and rotated per position,
    the variant that cannot absorb M_h) against absorbed GVA without a
    positional slice, on the same values, lengths, query content slice and
    maps: attention + combine, caches as stored, same split plan.  The
    contrast kernel is bound by the matrix cores, not by HBM: its roofline
    is priced in bf16 MFMA flops."""
    n = len(caches)
    d0 = gva.make_dims(w.batch, w.n_heads, w.n_groups, w.d_v, w.d_c, 0, w.t_max, w.dtype, w.rope_base)
    q0 = dev["q"][..., :w.d_c].contiguous()
    bufs = gva.DecodeBuffers(d0, S)
    fused0 = gva.gva_prefer_fused(d0, S, split_rows)
    q_abs = torch.empty(w.batch, w.n_heads, w.d_v, dtype=torch.float32, device="cuda")

    def combine():
        if S > 1:
            gva.gva_combine(d0, bufs.o_part, bufs.lse_part, S, bufs.o, bufs.lse, stream)

    def absorbed_calls(i):
        vc = caches[i][0]
        if fused0:
            gva.gva_decode_attention(d0, vc, None, dev["lens"], S, bufs.o_part, bufs.lse_part,
                                     q=q0, m=dev["m"], split_rows=split_rows, stream=stream)
        else:
            gva.gva_absorb_query(d0, q0, dev["m"], dev["lens"], q_abs, None, stream)
            gva.gva_decode_attention(d0, vc, None, dev["lens"], S, bufs.o_part, bufs.lse_part,
                                     q_abs=q_abs, split_rows=split_rows, stream=stream)
        combine()

    def rope_calls(i, with_combine=True):
        gva.gva_rope_decode_attention(d0, q0, dev["m"], caches[i][0], dev["lens"], S,
                                      bufs.o_part, bufs.lse_part, split_rows=split_rows, stream=stream)
        if with_combine:
            combine()

    abs_fns = [gva.prepare(absorbed_calls, c) for c in range(n)]
    rope_fns = [gva.prepare(rope_calls, c) for c in range(n)]
    rope_only_fns = [gva.prepare(rope_calls, c, False) for c in range(n)]

    def absorbed(i):
        abs_fns[i % n]()

    def rope(i, with_combine=True):
        (rope_fns if with_combine else rope_only_fns)[i % n]()

    try:                     # the group's W_h must fit one workgroup's LDS
        rope(0)
    except gva.GvaError as e:
        if e.status != gva.GVA_ERR_UNSUPPORTED:
            raise
        return {"skipped": f"gva_rope_decode_attention: {gva.status_string(e.status)} at H/G = "
                           f"{w.heads_per_group}, d_v = {w.d_v}, d_c = {w.d_c} (the W_h of a group's "
                           f"heads, {w.heads_per_group * w.d_v * w.d_c * 2} bytes, exceed one workgroup's LDS)"}
    warm([absorbed, rope], args.warmup, SIDE_WARM_S)
    t_abs = timed(absorbed, args.steps, stream)
    t_rope = timed(rope, args.steps, stream)
    # the contrast kernel alone, its launches back to back
    k_ms = t_rope if S == 1 else timed(lambda i: rope(i, with_combine=False), args.steps, stream)
    rows = int(inp["lens"].clamp(min=0).sum())
    flops = traffic.rope_decode_flops(rows, w.n_heads, w.d_v, w.d_c)
    bytes_ = traffic.decode_bytes(inp["lens"], w.batch, w.n_heads, w.n_groups, w.d_v, w.d_c, 0, 2)
    tflops = flops / (k_ms * 1e-3) / 1e12
    return {"what": "attention only (caches as stored): GVA with ordinary RoPE (per-position key "
                    "reconstruction) vs absorbed GVA with d_r = 0, same inputs and split plan",
            "absorbed_ms": round(t_abs, 5), "rope_ms": round(t_rope, 5),
            "time_ratio_rope_over_absorbed": round(t_rope / t_abs, 4),
            "absorbed_GBps": round(bytes_ / (t_abs * 1e-3) / 1e9, 1),
            "roofline": {"kernel": "rope_decode_kernel", "bound": "mfma", "achieved": round(tflops, 2),
                         "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                         "frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": None,
                         "algorithmic_flops_per_launch": flops, "avg_launch_ms": round(k_ms, 5),
                         "avg_launch_timing": "launches back to back between two events"}}


def prefill_kernel_name(w, N: int) -> str:
    """The prefill kernel gva_prefill_attention launches for one sequence
    of N prompt rows at w's head shapes (the library's rule, for the label):
    columns per wave at d_v = 128 and d_r <= 32 once its workgroups number
    2 per CU (4 at H/G = 8), else the tile-split kernel."""
    hpg = w.n_heads // w.n_groups
    items = w.n_groups * -(-N // (128 // hpg))
    per_wave = w.d_v == 128 and w.d_r <= 32 and items >= (4 if hpg >= 8 else 2) * gva.device_cu_count()
    return "prefill_vt_kernel" if per_wave else "prefill_bf16_kernel"


def prefill_comparison(args, w, caches, dev, stream):
    """A prompt of T tokens for one sequence at the workload's head shapes
    (its rows are the first sequence's cached rows): absorption + causal
    attention (gva_prefill_absorb + gva_prefill_attention), against the
    matched-GQA prefill (explicit key stream of width d_v, no positional
    term) on the same values.  Dense contractions: priced on the bf16 MFMA
    roofline."""
    N = w.t_max
    w1 = w.replace(batch=1)
    d1 = gva.make_dims(1, w.n_heads, w.n_groups, w.d_v, w.d_c, w.d_r, w.t_max, w.dtype, w.rope_base)
    v1, kr1 = caches[0][0][:1], caches[0][1][:1]
    lens1 = torch.full((1,), N, dtype=torch.int32, device="cuda")
    q = gva_inputs.prefill_queries(w1, args.seed, N).cuda()
    qg = gva_inputs.prefill_queries(w1, args.seed, N, gqa=True).cuda()
    g = torch.Generator().manual_seed(args.seed + 11)
    kg = gva.tiled(torch.randn(1, w.n_groups, w.t_max, w.d_v, generator=g).to(torch.bfloat16)).cuda()
    q_abs = torch.empty(1, N, w.n_heads, w.d_v, dtype=torch.float32, device="cuda")
    q_rot = torch.empty(1, N, w.n_heads, w.d_r, dtype=torch.float32, device="cuda")
    o = torch.empty(1, N, w.n_heads, w.d_v, dtype=torch.float32, device="cuda")
    lse = torch.empty(1, N, w.n_heads, dtype=torch.float32, device="cuda")
    qr = q_rot if w.d_r > 0 else None
    krc = kr1 if w.d_r > 0 else None

    def absorb(i):
        gva.gva_prefill_absorb(d1, N, q, dev["m"], lens1, q_abs, qr, stream)

    def attend(i):
        gva.gva_prefill_attention(d1, N, q_abs, qr, v1, krc, lens1, o, lse, stream)

    def gqa(i):
        gva.gva_gqa_prefill_attention(d1, N, qg, kg, v1, lens1, o, lse, stream)

    steps = max(5, args.steps // 10)
    warm([absorb, attend, gqa], 2, SIDE_WARM_S)
    t_abs = timed(absorb, steps, stream)
    t_att = timed(attend, steps, stream)
    t_gqa = timed(gqa, steps, stream)
    k_ms = t_att
    f_gva = traffic.prefill_flops(N, N, w.n_heads, w.d_v, w.d_r)
    f_gqa = traffic.prefill_flops(N, N, w.n_heads, w.d_v, 0)
    tf = f_gva / (k_ms * 1e-3) / 1e12
    return {"what": f"causal prefill of {N} tokens, batch 1, at the workload's head shapes: GVA "
                    "(absorb + attention) vs matched GQA attention on the same values",
            "n_tokens": N, "absorb_ms": round(t_abs, 5), "gva_attention_ms": round(t_att, 5),
            "gqa_attention_ms": round(t_gqa, 5),
            "time_ratio_gva_over_gqa": round(t_att / t_gqa, 4),
            "time_ratio_gva_with_absorb_over_gqa": round((t_att + t_abs) / t_gqa, 4),
            "flop_ratio_gva_over_gqa": round(f_gva / f_gqa, 4),
            "gqa_TFLOPs": round(f_gqa / (t_gqa * 1e-3) / 1e12, 2),
            "roofline": {"kernel": prefill_kernel_name(w, N), "bound": "mfma", "achieved": round(tf, 2),
                         "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                         "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": None,
                         "algorithmic_flops_per_launch": f_gva, "avg_launch_ms": round(k_ms, 5),
                         "avg_launch_timing": "launches back to back between two events"}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    # In a fresh process the step time settles only after a few hundred
    # steps (b32_t8k: ~86.5 us over steps 11-110, ~84 us from step 300 on).
    ap.add_argument("--warmup", type=int, default=300)
    ap.add_argument("--workload", default="b32_t8k", choices=sorted(gva_inputs.WORKLOADS))
    ap.add_argument("--splits", type=int, default=0,
                    help="splits per sequence (0: gva_pick_splits' plan)")
    ap.add_argument("--split-rows", type=int, default=0,
                    help="with --splits: fixed rows per split (0: even splits)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--absorb", choices=("auto", "fused", "separate"), default="auto",
                    help="absorb the query inside the attention kernel (fused) or in its own "
                         "gva_absorb_query launch (separate); auto picks by split count")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MB")
    ap.add_argument("--write-traffic", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV",
                    "COPY_WRITE_CSV"), help="summarise rocprofv3 --pmc CSVs into the traffic record")
    ap.add_argument("--copy-mb", type=int, default=1024)
    ap.add_argument("--cache-copies", type=int, default=0,
                    help="cache copies the steps rotate through (0: enough that the bytes one "
                         "rotation streams exceed twice the 256 MB last-level cache, at least 2)")
    ap.add_argument("--paged", type=int, default=0, metavar="PAGE_ROWS",
                    help="read the caches from page pools of PAGE_ROWS rows through a block table "
                         "(pages in random pool order)")
    ap.add_argument("--layers", type=int, default=0,
                    help="also time an N-layer decode step (each layer its own caches, query "
                         "and maps) eagerly and as one HIP graph replay")
    ap.add_argument("--no-prefill", action="store_true",
                    help="skip the causal-prefill timing (bf16 workloads)")
    ap.add_argument("--no-rope", action="store_true",
                    help="skip the ordinary-RoPE contrast timing (bf16 workloads)")
    ap.add_argument("--no-gqa", action="store_true",
                    help="skip the matched-GQA comparison (bf16 workloads; a key cache is drawn for workloads whose inputs carry none)")
    args = ap.parse_args()
    if args.write_traffic:
        write_traffic(*args.write_traffic, args.workload, args.splits or 1, args.copy_mb)
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "one GPU only: the decode path runs on a single GPU; sharding it "
                          "(by sequence, by group with the positional keys replicated, or by "
                          "context with gva_combine merging the shards) is not built",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    gva.lib()  # fail loudly if the HIP library is missing
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return

    w = gva_inputs.workload(args.workload)
    inp = gva_inputs.make_inputs(w, args.seed)
    d = gva.make_dims(w.batch, w.n_heads, w.n_groups, w.d_v, w.d_c, w.d_r, w.t_max, w.dtype,
                      w.rope_base)
    max_len = int(inp["lens"].max())
    if args.splits:
        S, split_rows = args.splits, args.split_rows
    else:
        S, split_rows = gva.plan_for(d, inp["lens"])
    elem = 2 if w.dtype == "bf16" else 4
    lens = inp["lens"]
    dec_b = traffic.decode_bytes(lens, w.batch, w.n_heads, w.n_groups, w.d_v, w.d_c, w.d_r, elem)
    # Rotate through enough cache copies that no step finds its rows left in
    # the 256 MB last-level cache (MALL) by the previous one.
    n_copies = args.cache_copies or min(64, max(2, math.ceil(2 * MALL_BYTES / dec_b)))
    dev = {k: inp[k].cuda() for k in ("q", "m", "lens", "v_new", "kr_new")}
    v_tiled, kr_tiled = gva.tiled(inp["v"]), gva.tiled(inp["kr"])   # the library's cache layout
    paging = None
    if args.paged:
        # every sequence's pages drawn in random order from one pool
        paging = gva.make_paging(d, args.paged, w.batch * (w.t_max // args.paged))
        gen = torch.Generator().manual_seed(args.seed + 7)
        block_table = torch.randperm(paging.n_pages, generator=gen).reshape(w.batch, paging.max_pages)
        block_table = block_table.to(torch.int32)
        v_tiled, kr_tiled = gva.to_pages(v_tiled, kr_tiled, block_table, paging)
        dev["block_table"] = block_table.cuda()
    caches = [(v_tiled.cuda(), kr_tiled.cuda()) for _ in range(n_copies)]
    del v_tiled, kr_tiled
    seq = torch.arange(w.batch, dtype=torch.int32)
    pos = (inp["lens"] - 1).clamp(min=0).to(torch.int32)
    bufs = gva.DecodeBuffers(d, S)
    fused = gva.gva_prefer_fused(d, S, split_rows) if args.absorb == "auto" else args.absorb == "fused"
    q_abs = torch.empty(w.batch, w.n_heads, w.d_v, dtype=torch.float32, device="cuda")
    q_rot = torch.empty(w.batch, w.n_heads, w.d_r, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    pend = dict(v_new=dev["v_new"], kr_new=dev["kr_new"] if w.d_r > 0 else None,
                split_rows=split_rows)

    ws = gva.workspace_for(d, S, split_rows) if paging is None else None
    one_call = paging is None and args.absorb == "auto"

    def step_calls(i, attention_only=False):
        # Algorithm 1: the attention launch appends the current token's rows
        # to the caches and attends over them.  With the library's own
        # absorption choice the step is one gva_decode_step call (the same
        # launches as below).
        vc, kc = caches[i]
        if one_call and not attention_only:
            gva.gva_decode_step(d, dev["q"], dev["m"], vc, kc, dev["lens"], S, bufs.o, bufs.lse, workspace=ws,
                                stream=stream, **pend)
            return
        if not fused and not attention_only:
            gva.gva_absorb_query(d, dev["q"], dev["m"], dev["lens"], q_abs, q_rot, stream)
        qkw = dict(q=dev["q"], m=dev["m"]) if fused else \
            dict(q_abs=q_abs, q_rot=q_rot if w.d_r > 0 else None)
        if paging is not None:
            gva.gva_paged_decode_attention(d, paging, vc, kc, dev["block_table"], dev["lens"], S,
                                           bufs.o_part, bufs.lse_part, stream=stream, **qkw, **pend)
        else:
            gva.gva_decode_attention(d, vc, kc, dev["lens"], S, bufs.o.unsqueeze(2) if S == 1 else bufs.o_part,
                                     bufs.lse.unsqueeze(2) if S == 1 else bufs.lse_part, stream=stream,
                                     **qkw, **pend)
        if S > 1 and not attention_only:   # one split: the attention writes the output
            gva.gva_combine(d, bufs.o_part, bufs.lse_part, S, bufs.o, bufs.lse, stream)

    # Each step's C calls are checked and marshalled once, per cache copy
    # (gva.prepare): the timed loop then issues the library calls alone, so
    # the Python binding's per-call checks (~10 us) do not pace the small
    # workloads' steps.
    step_fns = [gva.prepare(step_calls, c) for c in range(n_copies)]
    attn_fns = [gva.prepare(step_calls, c, True) for c in range(n_copies)]

    def step(i, attention_only=False):
        (attn_fns if attention_only else step_fns)[i % n_copies]()

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    ms_per_step = timed(step, args.steps, stream)

    # The roofline's launch time.  A step of one launch (one split, the
    # absorption fused) is that launch: its time is the timed steps' own, so
    # value and roofline come from one measurement.  Otherwise the attention
    # launches are timed alone, the same steps' launches back to back between
    # two events (the absorption and combine launches left out, their inputs
    # being in place).
    single_launch = fused and S == 1
    if single_launch:
        decode_ms = ms_per_step
        launch_timing = f"the {args.steps} timed steps (each step is this one launch)"
    else:
        if not fused:    # the attention launches' absorbed queries
            gva.gva_absorb_query(d, dev["q"], dev["m"], dev["lens"], q_abs, q_rot, stream)
        decode_ms = timed(lambda i: step(i, attention_only=True), args.steps, stream)
        launch_timing = f"{args.steps} attention launches back to back between two events on the launch stream"
    # The same steps again once the device has settled (a fresh process runs
    # its first few hundred steps slower): reported beside the figures above,
    # which keep exactly the --warmup steps they were given.
    settled_ms = None
    if args.warmup < SETTLE_STEPS:
        for i in range(SETTLE_STEPS - args.warmup):
            step(args.warmup + args.steps + i)
        settled_ms = timed(step, args.steps, stream)
    achievable, probe_wg = gva.probe_read_bandwidth(stream=stream)
    # a plain streaming read of the launch's algorithmic bytes, rotating over
    # as many buffers as the caches: the same start-up and tail, no compute
    same_ms, same_wg = gva.probe_read_time(dec_b, copies=n_copies, stream=stream)

    step_b = traffic.step_bytes(lens, w.batch, w.n_heads, w.n_groups, w.d_v, w.d_c, w.d_r, elem,
                                appended_rows=w.batch)
    # the attention launch appends the current rows; with one split it also
    # writes the output
    launch_b = traffic.launch_bytes(lens, w.batch, w.n_heads, w.n_groups, w.d_v, w.d_c, w.d_r, elem,
                                    appended_rows=w.batch, writes_output=S == 1)
    value = step_b / (ms_per_step * 1e-3) / 1e9
    achieved = launch_b / (decode_ms * 1e-3) / 1e9

    out = {
        "metric": metric_label(w),
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "t_max": w.t_max,
                   "n_heads": w.n_heads, "n_groups": w.n_groups, "d_v": w.d_v, "d_c": w.d_c,
                   "d_r": w.d_r, "num_splits": S, "split_rows": split_rows, "fused_absorb": fused,
                   "page_rows": args.paged or None,
                   "total_cached_rows": int(lens.clamp(min=0).sum()), "cache_copies": n_copies,
                   "parallelism": "none"},
        "frac_of_hbm_peak": round(value / HBM_PEAK_GBS, 4),
        "tokens_per_s": round(w.batch / (ms_per_step * 1e-3), 1),
        "tokens_heads_per_s": round(w.batch * w.n_heads / (ms_per_step * 1e-3), 1),
        "roofline": {
            "kernel": "decode_bf16_kernel" if w.dtype == "bf16" else "decode_f32_kernel",
            "bound": "hbm",
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic(w.name, S),
            "algorithmic_bytes_per_launch": launch_b,
            "avg_launch_ms": round(decode_ms, 5),
            "avg_launch_timing": launch_timing,
            "achievable_read_GBps": round(achievable, 1),
            "frac_of_achievable": round(achieved / achievable, 4),
            "achievable_probe": f"gva_probe_read, 2 GiB, {probe_wg} workgroups",
            "same_bytes_read_ms": round(same_ms, 5),
            "frac_of_same_bytes_read": round(same_ms * launch_b / dec_b / decode_ms, 4),
            "same_bytes_probe": f"gva_probe_read over the launch's algorithmic bytes, {n_copies} buffers "
                                f"in rotation, {same_wg} workgroups, 50 launches back to back",
        },
        "cpu_baseline": None,
    }
    if settled_ms is not None:
        out["settled"] = {"warmup_steps": SETTLE_STEPS, "ms_per_step": round(settled_ms, 5),
                          "value": round(step_b / (settled_ms * 1e-3) / 1e9, 2),
                          "frac_of_hbm_peak": round(step_b / (settled_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}

    o_gpu = (bufs.o_part[:, :, 0] if S == 1 and paging is not None else bufs.o).cpu()
    if paging is not None and args.layers > 0:
        raise SystemExit("--paged times the decode step only")
    if args.layers > 0:
        out["layer_stack"] = layer_stack(args, w, inp, d, S, split_rows, fused, dec_b)
    if w.dtype == "bf16" and not args.no_gqa and paging is None:
        out["gqa_comparison"] = gqa_comparison(args, w, inp, d, S, split_rows, fused, dev, caches,
                                               stream)
    if w.dtype == "bf16" and not args.no_rope and paging is None:
        out["rope_comparison"] = rope_comparison(args, w, inp, S, split_rows, dev, caches, stream)
    if w.dtype == "bf16" and not args.no_prefill and paging is None and w.t_max <= 16384:
        out["prefill_comparison"] = prefill_comparison(args, w, caches, dev, stream)
    if not args.no_cpu_baseline:
        rec, o_ref = cpu_baseline(w, inp, seq, pos)
        errs = [float((o_gpu[b].double() - o_ref[b]).abs().max()) for b in o_ref]
        rec["max_abs_err_vs_gpu"] = max(errs) if errs else None
        out["cpu_baseline"] = rec
    print(json.dumps(out))


if __name__ == "__main__":
    main()
