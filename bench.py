"""Benchmark of the MLA-Online step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 5] [--split-keys S]

A step is one pass of the whole path over the 256K-context workload, with every
input already resident in HBM and the plan for the segment table built once
beforehand (mla_online_plan): mla_online_attend_planned (device half of the plan
from the device-resident protected set, relocation, segment-wise attention with
the merge done by online rescaling, bf16 head outputs) and
mla_sliced_oproj_add_planned (sliced o-proj with the artifact add, f32 z).  Prints one
JSON line.  `value` is achieved TFLOP/s of attention + o-proj algorithmic work
over the whole step; `roofline` reports the attention kernel alone against the
dense bf16 MFMA peak; `cpu_baseline` times the fp64 oracle on a bounded row
sample on the host cores.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MLA-Online attn+o-proj TFLOP/s & % bf16 MFMA peak; merged rows/s at 256K"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0


def algorithmic_work(wl):
    """Exact algorithmic FLOPs and bytes of the instantiated workload.

    attention: every online head-row at position t scores t+1 keys over
    d_c + d_r dims and accumulates t+1 latent rows of d_c dims:
    (t+1) * (2*(d_c+d_r) + 2*d_c) flops.  Global heads run on every row, Local
    heads on protected rows.  o-proj: 2*d_c*d_model/n_pg flops per head-row.
    """
    g = wl.geom
    pos = np.empty(wl.n_rows, dtype=np.float64)
    for ks, ln, ro in wl.segs:
        pos[ks:ks + ln] = ro + np.arange(ln)
    per_key = 2.0 * g.d_qk + 2.0 * g.d_latent
    prot = np.asarray(wl.prot_rows, dtype=np.int64)
    vis_glob = float((pos + 1).sum()) * g.n_groups
    vis_loc = float((pos[prot] + 1).sum()) * g.n_local
    flop_attn = (vis_glob + vis_loc) * per_key
    head_rows = wl.n_rows * g.n_groups + len(prot) * g.n_local
    flop_oproj = head_rows * 2.0 * g.d_latent * g.d_model / g.n_proj_groups
    return flop_attn, flop_oproj, head_rows


def profiled_traffic():
    """HBM-side bytes per attention launch from the committed rocprofv3 counter
    summary, or None once the attention source differs from the profiled one."""
    import hashlib
    src = b"".join(open(os.path.join(ROOT, "paper_2609_07008_amd", "csrc", f), "rb").read()
                   for f in ("attend.hip", "common.h"))
    sha = hashlib.sha256(src).hexdigest()[:16]
    path = os.path.join(ROOT, "profiles", "mla_online_step_256k.md")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        parts = line.strip().split(":")
        if len(parts) == 2 and parts[0].startswith("attend_"):
            fields[parts[0]] = parts[1].strip()
    if fields.get("attend_source_sha256_16") != sha:
        return None
    return float(fields["attend_traffic_bytes_per_launch"])


def stratified_rows(wl, seed: int = 7):
    """Row sample for the oracle, interleaving the row kinds of the workload: the
    first and last row of every segment and the rows on both sides of each
    segment boundary (in request order), protected document rows, unprotected
    document rows and query rows (the query block is the last segment).  Seeded;
    the order alternates kinds so a time-bounded prefix still covers all of them."""
    rng = np.random.default_rng(seed)
    segs = np.asarray(wl.segs, dtype=np.int64)
    n = wl.n_rows
    prot = np.asarray(wl.prot_rows, dtype=np.int64)
    q0 = int(segs[np.argmax(segs[:, 2]), 0])          # first storage row of the query block
    is_prot = np.zeros(n, dtype=bool)
    is_prot[prot] = True
    edges = []
    for ks, ln, _ in segs[np.argsort(segs[:, 2])]:
        edges += [int(ks), int(ks + ln - 1)]
    doc = np.arange(q0)
    kinds = [rng.permutation(np.unique(edges)),
             rng.permutation(prot[prot < q0]),
             rng.permutation(doc[~is_prot[:q0]]),
             np.concatenate([[q0, n - 1], rng.permutation(np.arange(q0 + 1, n - 1))])]
    out, seen, i = [], set(), 0
    while any(i < len(k) for k in kinds):
        for k in kinds:
            if i < len(k) and int(k[i]) not in seen:
                seen.add(int(k[i]))
                out.append(int(k[i]))
        i += 1
        if len(out) >= 1024:
            break
    return out


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, budget_s: float = 20.0):
    """The fp64 oracle as it stands, timed on a bounded prefix of a stratified row
    sample of the same workload (all online heads of each row, unfactorized)."""
    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # noqa: BLE001
        cores = len(os.sched_getaffinity(0))
    g = wl.geom
    t0 = time.perf_counter()
    kv = wl.kv()
    keys = O.TrueKeys(kv, wl.segs, g.d_latent, g.rope_base)
    w_o = wl.w_o()
    setup = time.perf_counter() - t0
    prot = set(np.asarray(wl.prot_rows).tolist())
    pos = np.empty(wl.n_rows, dtype=np.int64)
    for ks, ln, ro in wl.segs:
        pos[ks:ks + ln] = ro + np.arange(ln)
    per_key = 2.0 * g.d_qk + 2.0 * g.d_latent
    done_rows, flops, elapsed = 0, 0.0, 0.0
    t_start = time.perf_counter()
    for r in stratified_rows(wl):
        zr = wl.z_off(rows=[r])
        O.reference_rows(wl, [r], z_off={r: zr[0]}, kv=kv, keys=keys, w_o=w_o)
        heads = g.n_groups + (g.n_local if r in prot else 0)
        flops += (pos[r] + 1) * per_key * heads + heads * 2.0 * g.d_latent * g.d_model / g.n_proj_groups
        done_rows += 1
        elapsed = time.perf_counter() - t_start
        if elapsed > budget_s:
            break
    return {"value": flops / elapsed / 1e12, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "rows_per_s": done_rows / elapsed, "cpu": cpu_model(),
            "sample": f"first {done_rows} rows of a stratified sample of the same workload (segment edges, "
                      f"protected / unprotected document rows, query rows; fp64, all online heads of each "
                      f"row, unfactorized), {elapsed:.1f} s after {setup:.1f} s of key setup"}


def merge_per_segment(wl, torch, stream, reps: int = 3):
    """Standalone mla_segment_merge on per-segment partials of the workload's query
    rows: every query-row slot (Global and Local heads) holds one partial per
    visible segment.  Partials are synthetic (the merge reads them, nothing else
    depends on their values); returns merged slot rows/s and achieved GB/s."""
    from paper_2609_07008_amd import mla
    g = wl.geom
    segs = np.asarray(wl.segs, dtype=np.int64)
    q0 = int(segs[np.argmax(segs[:, 2]), 0])
    n_q = wl.n_rows - q0
    n_slots = n_q * g.n_heads
    per_slot = int(segs.shape[0])                      # query rows see every segment
    n_parts = n_slots * per_slot
    dev = "cuda"
    part_o = torch.empty((n_parts, g.d_latent), dtype=torch.float32, device=dev).normal_()
    part_lse = torch.empty(n_parts, dtype=torch.float32, device=dev).normal_()
    part_ptr = torch.arange(0, n_parts + 1, per_slot, dtype=torch.int64, device=dev)
    out_o = torch.empty((n_slots, g.d_latent), dtype=torch.bfloat16, device=dev)
    out_lse = torch.empty(n_slots, dtype=torch.float32, device=dev)
    args = (n_slots, g.d_latent, part_o, part_lse, part_ptr, mla.MLA_BF16, out_o, out_lse)
    mla.segment_merge(*args, stream=stream)
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        mla.segment_merge(*args, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1) / 1e3)
    t = float(np.median(ts))
    nbytes = n_parts * (4 * g.d_latent + 4) + n_slots * (2 * g.d_latent + 4) + (n_slots + 1) * 8
    del part_o, part_lse, part_ptr, out_o, out_lse
    torch.cuda.empty_cache()
    return {"partials": n_parts, "slots": n_slots, "query_rows": n_q, "partials_per_slot": per_slot,
            "ms": round(t * 1e3, 3), "slot_rows_per_s": round(n_slots / t, 1),
            "query_rows_per_s": round(n_q / t, 1), "gb_s": round(nbytes / t / 1e9, 1),
            "pct_hbm_peak": round(100 * nbytes / t / 1e9 / PEAK_HBM_GBS, 1)}


def offline_producer(wl, torch, stream, reps: int = 2, seed: int = 70080):
    """mla_offline_produce (the MLA-Off native producer) on the workload's geometry
    and segment table: the Local-head artifact of every row.  Inputs are drawn on
    the device (torch.Generator seeded with `seed`; latent and queries ~ N(0, 1/dim),
    W_o std 0.02, as the workload's recipe) because the all-row Local-head queries
    are too large to draw on the host within the benchmark's time."""
    from paper_2609_07008_amd import mla
    g = wl.geom
    n = wl.n_rows
    hl = g.heads_per_group - 1
    if hl < 1:
        return None
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)

    def draw(shape, std):
        x = torch.empty(shape, dtype=torch.float32, device="cuda").normal_(0.0, 1.0, generator=gen)
        return (x * std).to(torch.bfloat16)

    kv = torch.cat([draw((n, g.d_latent), g.d_latent ** -0.5), draw((n, g.d_rope), g.d_rope ** -0.5)], 1)
    q = torch.empty((n, g.n_groups, hl, g.d_qk), dtype=torch.bfloat16, device="cuda")
    for c0 in range(0, n, 16384):   # chunked draw keeps the float32 staging small
        c1 = min(n, c0 + 16384)
        q[c0:c1, :, :, :g.d_latent] = draw((c1 - c0, g.n_groups, hl, g.d_latent), g.d_latent ** -0.5)
        q[c0:c1, :, :, g.d_latent:] = draw((c1 - c0, g.n_groups, hl, g.d_rope), g.d_rope ** -0.5)
    rows_w = (g.n_heads // g.n_proj_groups) * g.d_latent
    w_o = draw((g.n_proj_groups, rows_w, g.d_model // g.n_proj_groups), 0.02)
    z = torch.empty((n, g.d_model), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(mla.offline_produce_query(g, wl.segs), dtype=torch.uint8, device="cuda")
    args = (g, wl.segs, kv, q, wl.glob_head, w_o, mla.MLA_BF16, z, ws)
    mla.offline_produce(*args, stream=stream)
    torch.cuda.synchronize()
    # three calls back to back, as when documents are produced one after another:
    # each call's host plan (about 4 ms at this size) overlaps the previous call's
    # kernels, except the first call's, which is counted once in the three
    ts, one = [], []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(3):
            mla.offline_produce(*args, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1) / 3e3)
        e0.record(stream)
        mla.offline_produce(*args, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        one.append(e0.elapsed_time(e1) / 1e3)
    t = float(np.median(ts))
    # algorithmic work: each row's Local heads attend to u+1 keys of their own segment
    keys = float(sum(int(ln) * (int(ln) + 1) // 2 for _, ln, _ in np.asarray(wl.segs)))
    flop_attn = keys * g.n_groups * hl * (2.0 * g.d_qk + 2.0 * g.d_latent)
    flop_proj = n * g.n_groups * hl * 2.0 * g.d_latent * g.d_model / g.n_proj_groups
    del kv, q, w_o, z, ws
    torch.cuda.empty_cache()
    return {"ms": round(t * 1e3, 3), "ms_isolated_call": round(float(np.median(one)) * 1e3, 3),
            "rows_per_s": round(n / t, 1), "flop": flop_attn + flop_proj,
            "tflops": round((flop_attn + flop_proj) / t / 1e12, 3),
            "pct_bf16_peak": round(100 * (flop_attn + flop_proj) / t / 1e12 / PEAK_BF16_TFLOPS, 2),
            "local_head_rows": n * g.n_groups * hl, "out": "bf16 [rows, d_model]",
            "inputs": f"device-drawn, torch.Generator seed {seed}"}


def protected_set(wl, torch, stream, budgets=(0.10, 0.20, 0.25), reps: int = 5, seed: int = 70080):
    """mla_protected_rows (eq:protected) on the workload's segment table: query
    block, 1 % dirty rows, first/last 128 rows of relocated segments, the 32K
    tail, and the Indexer top-up to each budget level.  Indexer scores are
    seeded N(0, 1) draws; returns per budget the median time of one isolated call,
    the average of 20 back-to-back calls, and |A|."""
    from paper_2609_07008_amd import mla
    segs = np.asarray(wl.segs, dtype=np.int64)
    n = wl.n_rows
    q = int(np.argmax(segs[:, 2]))
    rng = np.random.default_rng(seed)
    flags = np.zeros(n, dtype=np.uint8)
    flags[rng.choice(n, size=n // 100, replace=False)] |= 2
    fl = torch.from_numpy(flags).cuda()
    sc = torch.from_numpy(rng.standard_normal(n).astype(np.float32)).cuda()
    ws = torch.empty(mla.protected_rows_query(segs), dtype=torch.uint8, device="cuda")
    out = torch.empty(n, dtype=torch.int32, device="cuda")
    cnt = torch.empty(1, dtype=torch.int32, device="cuda")
    res = {}
    for b in budgets:
        args = (segs, q, 128, 32768, b, fl, sc, out, cnt, ws)
        mla.protected_rows(*args, stream=stream)
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            mla.protected_rows(*args, stream=stream)
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(20):
            mla.protected_rows(*args, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        res[f"{b:.2f}"] = {"us": round(float(np.median(ts)) * 1e3, 1),
                           "us_back_to_back": round(e0.elapsed_time(e1) / 20 * 1e3, 1),
                           "protected": int(cnt.item())}
    return {"rows": n, "budgets": res, "edge_rows": 128, "tail_rows": 32768, "dirty_rows": n // 100}


def moe_fanout_bench(torch, stream, n_rows: int, n_experts: int = 256, tau: float = 0.9, reps: int = 10):
    """mla_moe_fanout (eq:moe) on seeded router weights for every row of the
    workload (256 experts, top-6, minimum fanout 3, tau 0.9): median time, the
    algorithmic HBM rate, and the mean fanout."""
    from paper_2609_07008_amd import mla
    from workloads import router_weights
    p = torch.from_numpy(router_weights(n_rows, n_experts, seed=70080)).cuda()
    idx = torch.empty((n_rows, 6), dtype=torch.int32, device="cuda")
    w = torch.empty((n_rows, 6), dtype=torch.float32, device="cuda")
    k = torch.empty((n_rows,), dtype=torch.int32, device="cuda")
    cnt = torch.empty((n_experts,), dtype=torch.int32, device="cuda")
    args = (p, tau, idx, w, k, cnt)
    mla.moe_fanout(*args, stream=stream)
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        mla.moe_fanout(*args, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    ms = float(np.median(ts))
    nbytes = n_rows * n_experts * 4 + n_rows * (6 * 8 + 4) + n_experts * 4
    return {"rows": n_rows, "experts": n_experts, "tau": tau, "ms": round(ms, 4),
            "GB_per_s": round(nbytes / (ms * 1e-3) / 1e9, 1), "bytes": nbytes,
            "mean_fanout": round(float(k.float().mean().item()), 4)}


def shared_wb_bench(torch, stream, z, reps: int = 5):
    """mla_shared_wb: y = W_b z over every row of the workload, z the step's own
    bf16 output (mla_sliced_oproj_add_planned with a bf16 z), W_b [4096, 4096]
    bf16 with std 0.02 drawn on the device, y fp32 (and, as a second figure, y
    bf16, the output type of a bf16 serving stack): median time and the MFMA
    rate against the dense bf16 peak."""
    from paper_2609_07008_amd import mla
    n_rows, d = int(z.shape[0]), int(z.shape[1])
    g = torch.Generator(device="cuda")
    g.manual_seed(70082)
    w = (torch.randn((d, d), generator=g, device="cuda") * 0.02).to(torch.bfloat16)
    flop = 2.0 * n_rows * d * d

    def timed(y):
        mla.shared_wb(z, w, y, stream=stream)
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            mla.shared_wb(z, w, y, stream=stream)
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return float(np.median(ts))

    y = torch.empty((n_rows, d), dtype=torch.float32, device="cuda")
    ms = timed(y)
    del y
    y = torch.empty((n_rows, d), dtype=torch.bfloat16, device="cuda")
    ms_bf16 = timed(y)
    del w, y
    return {"rows": n_rows, "d_in": d, "d_out": d, "ms": round(ms, 3), "flop": flop, "z": "the step's bf16 z",
            "TFLOP_per_s": round(flop / (ms * 1e-3) / 1e12, 1), "frac_of_bf16_peak": round(flop / (ms * 1e-3) / 2.5e15, 4),
            "y_bf16": {"ms": round(ms_bf16, 3), "TFLOP_per_s": round(flop / (ms_bf16 * 1e-3) / 1e12, 1),
                       "frac_of_bf16_peak": round(flop / (ms_bf16 * 1e-3) / 2.5e15, 4)}}


def dense_oproj(wl, out_o, dev, torch, stream, reps: int = 5):
    """The dense first projection (n_pg = 1: every head's 512 outputs into all
    d_model channels) on the step's merged head outputs and protected rows, with
    a device-drawn dense W_o [1, H*d_c, d_model] (bf16, std 0.02): the other W_a
    layout the step supports, timed on the same rows as the grouped one."""
    from dataclasses import replace
    from paper_2609_07008_amd import mla
    g = replace(wl.geom, n_proj_groups=1)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(70084)
    w_o = (torch.randn((1, g.n_heads * g.d_latent, g.d_model), generator=gen, device="cuda") * 0.02).to(torch.bfloat16)
    n_rows, n_prot = wl.n_rows, wl.n_prot
    n_glob = n_rows * g.n_groups
    o_glob = out_o[:n_glob]
    o_loc = out_o[n_glob:n_glob + n_prot * g.n_local] if n_prot * g.n_local else None
    z = torch.empty((n_rows, g.d_model), dtype=torch.float32, device="cuda")
    prot_d = torch.from_numpy(np.ascontiguousarray(wl.prot_rows, dtype=np.int32)).cuda()
    args = (g, n_rows, o_glob, o_loc, wl.glob_head, prot_d, n_prot, w_o, dev["z_off"], z)
    mla.sliced_oproj_add(*args, stream=stream)
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        mla.sliced_oproj_add(*args, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    ms = float(np.median(ts))
    head_rows = n_rows * g.n_groups + n_prot * g.n_local
    flop = head_rows * 2.0 * g.d_latent * g.d_model
    nbytes = ((n_rows - n_prot) * g.d_model * 2 + n_rows * g.d_model * 4 + head_rows * g.d_latent * 2
              + w_o.numel() * 2)
    del w_o, z
    return {"ms": round(ms, 3), "flop": flop, "TFLOP_per_s": round(flop / (ms * 1e-3) / 1e12, 1),
            "pct_bf16_peak": round(100 * flop / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 2),
            "GB_per_s": round(nbytes / (ms * 1e-3) / 1e9, 1), "bytes": nbytes,
            "w_o": f"dense [1, {g.n_heads * g.d_latent}, {g.d_model}] bf16"}


def device_peaks(torch, stream, att_tflops: float, oproj_gbs: float, reps: int = 3):
    """The rates measured on this device that the step's kernels are set against,
    beside the data-sheet figures: the dense bf16 matrix-core rate from
    mla_probe_mfma_bf16 (waves doing nothing but MFMA 32x32x16 bf16), and a device
    copy's HBM rate (torch's copy of 2 GiB of float32: half reads, half writes)."""
    from paper_2609_07008_amd import mla
    sink = torch.zeros(4, dtype=torch.float32, device="cuda")
    mla.probe_mfma_bf16(200, sink, stream=stream)
    torch.cuda.synchronize()
    ts = []
    flop = 0.0
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        flop = mla.probe_mfma_bf16(4000, sink, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1) / 1e3)
    mfma = flop / float(np.median(ts)) / 1e12
    n = 1 << 29
    x = torch.ones(n, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    y.copy_(x)
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps + 2):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        y.copy_(x)
        e1.record(stream)
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1) / 1e3)
    copy = 2 * n * 4 / float(np.median(ts)) / 1e12
    del x, y, sink
    return {"mfma_bf16_TFLOP_per_s": round(mfma, 1), "mfma_probe": "mla_probe_mfma_bf16, 4000 products per chain",
            "attention_frac_of_measured_mfma": round(att_tflops / mfma, 4),
            "copy_TB_per_s": round(copy, 3), "copy": "torch copy_ of 2 GiB float32",
            "oproj_add_frac_of_copy": round(oproj_gbs / 1e3 / copy, 4)}


def host_plan_step(wl, dev, torch, stream, split: int, reps: int = 3):
    """The same step through the host-plan entry points (mla_online_attend, which
    builds and uploads its plan from the host on every call, writes f32 partials,
    then mla_segment_merge and mla_sliced_oproj_add), for comparison with the
    plan-once path that the headline times."""
    from paper_2609_07008_amd import step
    st = step.OnlineStep(wl.geom, wl.segs, wl.prot_rows, wl.glob_head, split, with_part_seg=False)
    st.run(dev["kv"], dev["q_glob"], dev["q_loc"], dev["w_o"], dev["z_off"])
    torch.cuda.synchronize()
    t = []
    for _ in range(reps):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        e[0].record(stream)
        st.attend(dev["kv"], dev["q_glob"], dev["q_loc"])
        e[1].record(stream)
        st.merge()
        e[2].record(stream)
        st.oproj(dev["w_o"], dev["z_off"])
        e[3].record(stream)
        torch.cuda.synchronize()
        t.append([e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2]), e[2].elapsed_time(e[3]), e[0].elapsed_time(e[3])])
    t = np.median(np.asarray(t), axis=0)
    out = {"ms": {"attend": round(float(t[0]), 3), "merge": round(float(t[1]), 3), "oproj": round(float(t[2]), 3),
                  "step": round(float(t[3]), 3)}, "partials": st.n_parts}
    del st
    torch.cuda.empty_cache()
    return out


class ClockSampler:
    """Shader clock of the GPU sampled from the amdgpu driver's current DPM level
    (/sys/class/drm/card*/device/pp_dpm_sclk, the line marked '*', which is what
    rocm-smi --showgpuclocks reports) in a background thread while the timed steps
    run: the clock under this load decides the dense peak the chip can reach
    (2.5 PFLOP/s is quoted at 2.4 GHz).  A file read, no child process."""

    def __init__(self):
        import glob
        import threading
        self.samples, self.error = [], None
        paths = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
        self.path = paths[0] if paths else None
        self._stop = threading.Event()
        self._thr = threading.Thread(target=self._loop, daemon=True)

    def _read(self):
        import re
        with open(self.path) as f:
            for line in f:
                if line.rstrip().endswith("*"):
                    m = re.search(r"([0-9.]+)\s*Mhz", line, re.I)
                    if m:
                        return float(m.group(1))
        raise ValueError("no current level in " + self.path)

    def _loop(self):
        if self.path is None:
            self.error = "no pp_dpm_sclk file"
            return
        while not self._stop.is_set():
            try:
                self.samples.append(self._read())
            except Exception as e:  # noqa: BLE001
                self.error = f"{type(e).__name__}: {e}"[:200]
                return
            self._stop.wait(0.25)

    def __enter__(self):
        self._thr.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        self._thr.join(timeout=5)

    def report(self):
        out = {"source": f"{self.path} (current DPM level) during the timed steps", "sclk_mhz": self.samples}
        if self.samples:
            out["median_mhz"] = float(np.median(self.samples))
            out["peak_bf16_tflops_at_clock"] = round(PEAK_BF16_TFLOPS * out["median_mhz"] / 2400.0, 1)
        if self.error:
            out["error"] = self.error
        return out


def rotary_value_step(wl, dev, torch, stream, split: int, reps: int = 2):
    """The step with a rotary value (the value is the whole latent row; each
    segment's RoPE output dims restored and rotated back by R(-(t - p_s))) on the
    same resident inputs, with a W_o of d_c + d_r rows per head (bf16, std 0.02,
    drawn on the device).  Work counted as the method's: 2*576 + 2*576 flop per
    visible key and head-row, plus the o-proj over 576-wide head outputs."""
    from dataclasses import replace
    from paper_2609_07008_amd import mla, step
    g = replace(wl.geom, value_rope=True)
    dv = g.d_latent + g.d_rope
    gen = torch.Generator(device="cuda")
    gen.manual_seed(70083)
    hp = g.n_heads // g.n_proj_groups
    w_o = (torch.randn((g.n_proj_groups, hp * dv, g.d_model // g.n_proj_groups), generator=gen, device="cuda")
           * 0.02).to(torch.bfloat16)
    st = step.PlannedStep(g, wl.segs, wl.glob_head, split, wl.n_rows, bookkeeping=False)
    prot_d, n_d = dev["prot_d"], dev["n_prot_d"]
    st.run(prot_d, n_d, dev["kv"], dev["q_glob"], dev["q_loc"], w_o, dev["z_off"])
    torch.cuda.synchronize()
    t = []
    for _ in range(reps):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        e[0].record(stream)
        st.attend(prot_d, n_d, dev["kv"], dev["q_glob"], dev["q_loc"])
        e[1].record(stream)
        st.oproj(prot_d, n_d, w_o, dev["z_off"])
        e[2].record(stream)
        torch.cuda.synchronize()
        t.append([e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2]), e[0].elapsed_time(e[2])])
    t = np.median(np.asarray(t), axis=0)
    pos = wl.row_position()
    prot = np.asarray(wl.prot_rows, dtype=np.int64)
    vis = float((pos + 1).sum()) * g.n_groups + float((pos[prot] + 1).sum()) * g.n_local
    flop_attn = vis * (2.0 * (g.d_latent + g.d_rope) + 2.0 * dv)
    head_rows = wl.n_rows * g.n_groups + len(prot) * g.n_local
    flop_oproj = head_rows * 2.0 * dv * g.d_model / g.n_proj_groups
    ms = float(t[2])
    out = {"ms": {"attend": round(float(t[0]), 3), "oproj": round(float(t[1]), 3), "step": round(ms, 3)},
           "flop": flop_attn + flop_oproj,
           "TFLOP_per_s": round((flop_attn + flop_oproj) / (ms * 1e-3) / 1e12, 1),
           "pct_bf16_peak": round(100 * (flop_attn + flop_oproj) / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 2),
           "head_output_width": dv}
    del st, w_o
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", type=int, default=5)
    ap.add_argument("--split-keys", type=int, default=-1,
                    help="chunking of each row's visible segments; -1 = one chunk per slot")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-merge-per-segment", action="store_true",
                    help="skip the standalone merge of per-segment partials of the query rows")
    ap.add_argument("--no-rotary-value", action="store_true",
                    help="skip the rotary-value step measurement")
    ap.add_argument("--no-offline-producer", action="store_true",
                    help="skip the MLA-Off producer measurement on the same geometry")
    ap.add_argument("--step-only", action="store_true",
                    help="time the step only: skip every other measurement (for profiler runs)")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--prot-cap", type=int, default=-1,
                    help="capacity of the plan for the protected set; -1 = every row")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (reference for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only: the step is measured on the "
                                   "full set of heads of one layer on one device"}))
        sys.exit(2)

    import torch
    from workloads import make_workload
    from paper_2609_07008_amd import device_inputs, step

    torch.cuda.set_device(0)
    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n, "copies": 3}), flush=True)
        return
    wl = make_workload(args.workload)
    g = wl.geom
    split = wl.n_rows if args.split_keys < 0 else args.split_keys
    t0 = time.perf_counter()
    dev = device_inputs.upload(wl)
    torch.cuda.synchronize()
    t_upload = time.perf_counter() - t0
    # plan once for the segment table, capacity = every row; the protected set
    # lives on the device and each step only enqueues kernels
    dev["prot_d"] = torch.from_numpy(np.ascontiguousarray(wl.prot_rows, dtype=np.int32)).cuda()
    dev["n_prot_d"] = torch.tensor([wl.n_prot], dtype=torch.int32, device="cuda")
    prot_cap = wl.n_rows if args.prot_cap < 0 else args.prot_cap
    st = step.PlannedStep(g, wl.segs, wl.glob_head, split, prot_cap, bookkeeping=False)
    flop_attn, flop_oproj, head_rows = algorithmic_work(wl)
    prot_d, n_d = dev["prot_d"], dev["n_prot_d"]

    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        st.run(prot_d, n_d, dev["kv"], dev["q_glob"], dev["q_loc"], dev["w_o"], dev["z_off"])
    torch.cuda.synchronize()

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    with ClockSampler() as clock:
        t_wall = time.perf_counter()
        for k in range(args.steps):
            e = ev[k]
            e[0].record(stream)
            st.attend(prot_d, n_d, dev["kv"], dev["q_glob"], dev["q_loc"])
            e[1].record(stream)
            st.oproj(prot_d, n_d, dev["w_o"], dev["z_off"])
            e[2].record(stream)
        torch.cuda.synchronize()
        t_wall = time.perf_counter() - t_wall
    if int(st.status.item()) != 0:
        raise RuntimeError(f"the device plan rejected the protected set (status {int(st.status.item())})")
    t_att = np.median([e[0].elapsed_time(e[1]) for e in ev]) / 1e3
    t_opj = np.median([e[1].elapsed_time(e[2]) for e in ev]) / 1e3
    t_step = np.median([e[0].elapsed_time(e[2]) for e in ev]) / 1e3

    value = (flop_attn + flop_oproj) / t_step / 1e12
    att_tflops = flop_attn / t_att / 1e12
    oproj_bytes = (wl.n_rows - wl.n_prot) * g.d_model * 2 + wl.n_rows * g.d_model * 4 + head_rows * g.d_latent * 2
    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(t_step * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"workload {args.workload}: {wl.name}", "rows": wl.n_rows,
                   "segments": int(wl.segs.shape[0]), "heads": g.n_heads, "groups": g.n_groups,
                   "protected_rows": wl.n_prot, "d_latent": g.d_latent, "d_rope": g.d_rope,
                   "d_model": g.d_model, "proj_groups": g.n_proj_groups, "split_keys": split,
                   "prot_cap": prot_cap, "max_items": int(st.info.max_items),
                   "path": "mla_online_plan once; per step mla_online_attend_planned (merge in the attention "
                           "kernel, bf16 head outputs) + mla_sliced_oproj_add_planned (f32 z)"},
        "pct_bf16_peak": round(100 * value / PEAK_BF16_TFLOPS, 2),
        "merged_rows_per_s": round(wl.n_rows / t_step, 1),
        "flop_attn": flop_attn,
        "flop_oproj": flop_oproj,
        "ms": {"attend": round(t_att * 1e3, 3), "oproj": round(t_opj * 1e3, 3),
               "wall_per_step": round(t_wall / args.steps * 1e3, 3), "upload_s": round(t_upload, 2)},
        "hbm_gbs": {"oproj_add": round(oproj_bytes / t_opj / 1e9, 1)},
        "roofline": {"bound": "mfma", "achieved": round(att_tflops, 3), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(att_tflops / PEAK_BF16_TFLOPS, 4), "traffic": profiled_traffic(),
                     "kernel": "attend_kernel<512,64> (timed with the device plan kernels of "
                               "mla_online_attend_planned)"},
    }
    out["clock"] = clock.report()
    if args.step_only:
        print(json.dumps(out), flush=True)
        return
    # the step's z in bf16 (the hand-off to W_b), then W_b on it
    from paper_2609_07008_amd import mla
    z16 = torch.empty((wl.n_rows, g.d_model), dtype=torch.bfloat16, device="cuda")
    n_glob = wl.n_rows * g.n_groups
    ts = []
    for _ in range(4):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        mla.sliced_oproj_add_planned(g, st.info, st.out_o[:n_glob], st.out_o[n_glob:], wl.glob_head, prot_d, n_d,
                                     dev["w_o"], dev["z_off"], z16, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    ms16 = float(np.median(ts[1:]))
    b16 = (wl.n_rows - wl.n_prot) * g.d_model * 2 + wl.n_rows * g.d_model * 2 + head_rows * g.d_latent * 2
    out["oproj_bf16_z"] = {"ms": round(ms16, 3), "GB_per_s": round(b16 / (ms16 * 1e-3) / 1e9, 1)}
    out["shared_wb"] = shared_wb_bench(torch, stream, z16)
    del z16
    out["dense_oproj"] = dense_oproj(wl, st.out_o, dev, torch, stream)
    del st
    torch.cuda.empty_cache()
    out["host_plan_step"] = host_plan_step(wl, dev, torch, stream, split)
    if not args.no_rotary_value:
        out["rotary_value"] = rotary_value_step(wl, dev, torch, stream, split)
    del dev
    torch.cuda.empty_cache()
    if not args.no_merge_per_segment:
        out["merge_per_segment"] = merge_per_segment(wl, torch, stream)
    if not args.no_offline_producer:
        out["offline_producer"] = offline_producer(wl, torch, stream)
    out["protected_set"] = protected_set(wl, torch, stream)
    out["moe_fanout"] = moe_fanout_bench(torch, stream, wl.n_rows)
    out["device_peaks"] = device_peaks(torch, stream, att_tflops, out["hbm_gbs"]["oproj_add"])
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
