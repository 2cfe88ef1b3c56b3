#!/usr/bin/env python3
"""Throughput of the batched centroid + residual LoRA apply on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload prefill|qproj|decode8b|zipf|zipf-baseline|...]

Prints ONE JSON line.  A step is one pass of the hot path over one batch: the
device plan build (grouping by centroid) followed by the apply of every table of
the workload, a decoder layer's seven tables per salt_apply_batch (one shrink and
one expand launch per layer).  Inputs (x, y, maps, pinned centroids, resident
residuals) are in HBM before the timed region starts.

Default workload (the metric's configuration): Llama-3.2-3B, all seven
projections of its 28 layers (196 tables), bf16 prefill of 8192 tokens in 256
user segments, 8 centroids of rank 64, residuals of rank 1.  The default run also
reports, as sub-records, the q_proj decode batch (T = 64), the Llama-3.1-8B
decode layer (T = 256, with 32 residual swaps per step overlapped with the
apply) and the Zipf multi-tenant layer (T = 512) against its rank-16 LoRA
baseline.

Timing: HIP events on the stream the kernels run on, around the K timed steps.
For the roofline, salt_apply_batch_timed's events record each shrink and expand
kernel's own start and end; the dominant kernel is the one with the larger mean
duration, its achieved bandwidth = its algorithmic bytes / that duration.
``cpu_baseline`` times the fp64 oracle on a bounded sample of the same workload
on this host, BLAS on one thread and on all cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

HBM_PEAK_GBPS = 8000.0   # MI355X HBM3E
METRIC = "Centroid+residual LoRA apply: tokens/s and achieved HBM GB/s, Llama-3.2-3B"

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# sources that fix the apply kernels' machine code and launch shapes: counter
# summaries under profiles/ hold for these contents only
KERNEL_SOURCES = ("salt_apply.hip", "salt_device.h", "salt_layout.h", "salt_launch.h", "salt_internal.h")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for n in KERNEL_SOURCES:
        h.update(open(os.path.join(ROOT, "paper_2608_03579_amd", "csrc", n), "rb").read())
    return h.hexdigest()[:16]


# ---------------------------------------------------------------------------
# algorithmic bytes
# ---------------------------------------------------------------------------
def _adapter_rows(w, maps):
    """Rank rows of adapters one table's apply reads: each referenced centroid
    at r_c, each referenced residual slot at its own rank."""
    tok_c, tok_u = maps
    cents = np.unique(tok_c[tok_c >= 0])
    slots = np.unique(tok_u[tok_u >= 0])
    return len(cents) * w.r_c + int(sum(int(w.slot_rank[s]) for s in slots))


def kernel_bytes(w, maps, table):
    """(shrink, expand) algorithmic bytes of one table: the shrink reads x once
    and the A factors of the referenced adapters once; the expand reads and
    writes y once and reads their B factors once; each reads the 16-byte token
    records."""
    _, n_in, n_out = w.tables[table]
    es = w.esize
    T = len(maps[0])
    rows = _adapter_rows(w, maps)
    return es * (T * n_in + rows * n_in) + 16 * T, es * (2 * T * n_out + rows * n_out) + 16 * T


def apply_bytes(w, maps, table):
    """Algorithmic HBM bytes of one table's apply: x once, y read + write once,
    each referenced centroid's A and B once, each referenced residual at its own
    rank once, and the per-token plan records (16 B each)."""
    _, n_in, n_out = w.tables[table]
    T = len(maps[0])
    return w.esize * (T * n_in + 2 * T * n_out + _adapter_rows(w, maps) * (n_in + n_out)) + 16 * T


def apply_flops(w, maps, table):
    tok_c, tok_u = maps
    _, n_in, n_out = w.tables[table]
    r = np.where(tok_c >= 0, w.r_c, 0) + np.where(tok_u >= 0, w.slot_rank[np.maximum(tok_u, 0)], 0)
    return int(2 * (n_in + n_out) * r.sum())


# ---------------------------------------------------------------------------
# CPU baseline: the oracle as it stands, bounded sample, on this host
# ---------------------------------------------------------------------------
def host_info():
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    blas = "unknown"
    try:
        cfg = np.show_config(mode="dicts")
        b = cfg.get("Build Dependencies", {}).get("blas", {})
        blas = f"{b.get('name', '?')} {b.get('version', '')}".strip()
    except Exception:   # pragma: no cover
        pass
    return {"cpu_model": model, "logical_cpus": os.cpu_count(), "blas": blas}


def _oracle_pass(data, w, chunk, budget_s):
    """Plan once per batch, then the apply of every table on chunks of `chunk`
    tokens, until budget_s has passed at the end of a chunk."""
    import oracle
    n_tab = len(data)
    pairs = 0
    t0 = time.perf_counter()
    start = 0
    while True:
        if start == 0:
            oracle.plan(w.tok_c, w.tok_u)
        rows = list(range(start, min(w.T, start + chunk)))
        for t in range(n_tab):
            x, y0, cat, cb, res = data[t]
            oracle.apply(x, y0, cat, cb, res, w.tok_c, w.tok_u, w.gamma, rows=rows)
        pairs += len(rows) * n_tab
        start = (start + chunk) % w.T
        if time.perf_counter() - t0 >= budget_s:
            break
    return pairs / n_tab / (time.perf_counter() - t0), pairs // n_tab


def cpu_baseline(w, dw, budget_s=3.0, repeats=3):
    """Tokens/s of the oracle through every table of workload w (the 28-layer
    prefill repeats the seven tables of dw, as the GPU run does), BLAS on one
    thread and on all cores; median of `repeats` runs each, after one warm-up."""
    import oracle
    from threadpoolctl import threadpool_info, threadpool_limits
    d = dw.dtype
    data = []
    for t in range(len(dw.tables)):
        x = oracle.decode(dw.x(t), d)
        y0 = oracle.decode(dw.y0(t), d)
        cat, cb = (oracle.decode(a, d) for a in dw.centroids(t)) if dw.n_centroids else (None, None)
        res = {int(s): tuple(oracle.decode(a, d) for a in dw.residual(int(s), t)) for s in dw.referenced_slots()}
        data.append((x, y0, cat, cb, res))
    reps = len(w.tables) // len(dw.tables)
    data = data * reps
    chunk = min(w.T, 64)
    out = {}
    for name, limit in (("single_thread", 1), ("all_cores", None)):
        with threadpool_limits(limits=limit):
            threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
            _oracle_pass(data, w, chunk, 0.3)
            runs = [_oracle_pass(data, w, chunk, budget_s) for _ in range(repeats)]
        vals = sorted(r[0] for r in runs)
        out[name] = {"value": vals[len(vals) // 2], "cores": threads if limit is None else 1,
                     "tokens_per_run": runs[0][1], "runs": [round(v, 1) for v in vals]}
        log(f"cpu baseline {name}: {out[name]['value']:.1f} tokens/s ({threads if limit is None else 1} threads)")
    best = max(out.values(), key=lambda r: r["value"])
    hi = host_info()
    return {"value": best["value"], "unit": "tokens/s", "cores": best["cores"], "kind": "oracle",
            "sample": (f"the first {best['tokens_per_run']} tokens through all {len(w.tables)} tables per run (plan + "
                       f"apply, chunks of {chunk} tokens), median of {repeats} runs of ~{budget_s:.0f} s after a "
                       f"warm-up; fp64 numpy; single thread {out['single_thread']['value']:.1f} tokens/s, all "
                       f"cores ({out['all_cores']['cores']} BLAS threads) {out['all_cores']['value']:.1f} tokens/s; "
                       f"{hi['cpu_model']}, {hi['logical_cpus']} logical cpus, BLAS {hi['blas']}"),
            "single_thread": out["single_thread"], "all_cores": out["all_cores"], "host": hi}


# ---------------------------------------------------------------------------
# GPU
# ---------------------------------------------------------------------------
WORKLOADS = {
    "prefill": dict(cfg=3, rot=1, steps=10, warmup=2),
    "qproj": dict(cfg=2, rot=128, steps=2000, warmup=200),
    "decode8b": dict(cfg=4, rot=4, steps=500, warmup=50, swaps=True),
    "zipf": dict(cfg=5, rot=4, steps=500, warmup=50),
    "zipf-baseline": dict(cfg=5, rot=4, baseline=True, steps=200, warmup=20),
    # Sec. 3.3's long tail: the Zipf batch with the users of slots >= 100 served by
    # concatenated rank-65/66 adapters (no centroid), the head by centroid + residual
    "longtail": dict(cfg=5, rot=4, tail=100, steps=200, warmup=20),
    # Sec. 3.3: a centroid fused into the base weights of one Llama-3.2-3B layer
    "fuse": dict(cfg=5, rot=2, steps=20, warmup=3, fuse=True),
    # Sec. 3.1 Eq. 2 / Sec. 4.5: layer-wise cosine of two rank-16 adapters over the
    # 196 tables of the 28-layer Llama-3.2-3B
    "gram": dict(cfg=3, rot=1, steps=10, warmup=2, gram=True),
}
# sub-records of the default run: shorter than a workload's own defaults
SUB_RECORDS = (("qproj", 1000, 100), ("decode8b", 200, 20), ("zipf", 200, 20), ("zipf-baseline", 100, 10))


def make_workload(spec):
    from paper_2608_03579_amd import synth
    w = synth.make(spec["cfg"], 0, baseline=spec.get("baseline", False))
    if spec.get("tail"):
        w = synth.long_tail(w, spec["tail"])
    # the 28-layer prefill draws adapter and activation values for one layer and
    # repeats them over the layers (each table still has its own memory)
    dw = synth.make(3, 0, layers=1) if spec["cfg"] == 3 else w
    return w, dw


def layer_groups(w):
    """Tables applied together: a decoder layer's seven projections."""
    names = [n for n, _, _ in w.tables]
    groups, cur, layer = [], [], None
    for t, n in enumerate(names):
        l = n.split(".")[0] if "." in n else ""
        if cur and l != layer:
            groups.append(cur)
            cur = []
        cur.append(t)
        layer = l
    groups.append(cur)
    return groups


def build_context(w, dw, rot, salt):
    """A context whose tables are `rot` copies of the workload's tables, with
    every centroid pinned and every referenced residual loaded; adapter values
    come from dw, whose tables repeat to give w's."""
    shapes = [(i, o) for _, i, o in w.tables] * rot
    ctx = salt.Context(w.dtype, shapes, w.n_centroids, w.r_c, w.n_slots, w.r_u_max, max(1, w.T))
    n_tab, n_dat = len(w.tables), len(dw.tables)
    reps = (n_tab // n_dat) * rot
    if w.n_centroids:
        for t in range(n_dat):
            at, b = dw.centroids(t)
            for k in range(reps):
                ctx.pin_centroids(k * n_dat + t, at, b)
    for s in w.referenced_slots():
        s = int(s)
        r = int(w.slot_rank[s])
        blob = dw.residual_blob(s)
        ctx.load_residual(s, r, np.tile(blob, reps) if r else None)
    ctx.wait_loads()
    return ctx


def run_gpu(name, w, dw, spec, steps, warmup, hip, salt, meas=None):
    rot = spec["rot"]
    n_tab, n_dat = len(w.tables), len(dw.tables)
    log(f"{name}: {w.name}; T={w.T}, tables={n_tab}, rotation={rot}")
    t_setup = time.perf_counter()
    ctx = build_context(w, dw, rot, salt)
    stream = hip.Stream()
    # x and y per table copy: the rotation keeps consecutive steps on disjoint
    # memory (the working set stays above the 256 MB Infinity Cache)
    xs, ys = [None] * (n_tab * rot), [None] * (n_tab * rot)
    for t in range(n_dat):
        x0 = hip.DeviceArray.from_host(dw.x(t))
        y0 = hip.DeviceArray.from_host(dw.y0(t))
        for k in range(rot * (n_tab // n_dat)):
            i = k * n_dat + t
            xs[i] = hip.DeviceArray(x0.shape, x0.dtype)
            ys[i] = hip.DeviceArray(y0.shape, y0.dtype)
            xs[i].copy_from(x0)
            ys[i].copy_from(y0)
        hip.synchronize()
        x0.free()
        y0.free()
    plans = []
    for k in range(rot):
        p = ctx.plan()
        p.set_maps(w.tok_c, w.tok_u, w.gamma, stream.h)
        plans.append(p)
    stream.synchronize()
    tile_m, n_tiles, launches = plans[0].tiling()
    groups = layer_groups(w)
    log(f"{name}: setup {time.perf_counter() - t_setup:.1f} s; tiles of {tile_m} tokens: {n_tiles}; "
        f"{len(groups)} apply_batch calls per step, {launches} launches each")

    def tabs(slot, g):
        return [slot * n_tab + t for t in g]

    def step(k):
        slot = k % rot
        p = plans[slot]
        p.build(stream.h)
        for g in groups:
            tt = tabs(slot, g)
            ctx.apply_batch(tt, p, [xs[i].ptr for i in tt], [ys[i].ptr for i in tt], stream.h)

    for k in range(warmup):
        step(k)
    stream.synchronize()
    e0, e1 = hip.Event(), hip.Event()
    hip.synchronize()
    e0.record(stream)
    t0 = time.perf_counter()
    for k in range(steps):
        step(k)
    enqueue = time.perf_counter() - t0
    e1.record(stream)
    e1.synchronize()
    wall = time.perf_counter() - t0
    ms_total = e0.elapsed_ms(e1)
    ms_step = ms_total / steps
    log(f"{name}: timed {steps} steps: {ms_total:.3f} ms GPU ({wall * 1e3:.1f} ms wall, host enqueue "
        f"{enqueue * 1e3:.1f} ms), {ms_step * 1e3:.2f} us/step")

    # roofline: each launch's shrink and expand kernels timed by their own events
    maps = (w.tok_c, w.tok_u)
    kb = [kernel_bytes(w, maps, t) for t in range(n_tab)]
    bytes_tab = np.array([apply_bytes(w, maps, t) for t in range(n_tab)], dtype=np.float64)
    n_meas = meas or max(2, min(200, 2000 // max(1, len(groups))))
    ev = [hip.Event() for _ in range(4 * n_meas * len(groups))]
    for p in plans[:n_meas]:
        p.build(stream.h)  # a short timed run may not have built every rotated plan
    i = 0
    for k in range(n_meas):
        slot = k % rot
        for g in groups:
            tt = tabs(slot, g)
            ctx.apply_batch_timed(tt, plans[slot], [xs[j].ptr for j in tt], [ys[j].ptr for j in tt], stream.h,
                                  [e.h for e in ev[4 * i:4 * i + 4]])
            i += 1
    stream.synchronize()
    sh = np.array([ev[4 * j].elapsed_ms(ev[4 * j + 1]) for j in range(i)]).reshape(n_meas, len(groups))
    ex = np.array([ev[4 * j + 2].elapsed_ms(ev[4 * j + 3]) for j in range(i)]).reshape(n_meas, len(groups))
    for e in ev + [e0, e1]:
        e.destroy()
    sh_us, ex_us = sh.mean() * 1e3, ex.mean() * 1e3
    # all groups of a workload have the same shapes (28 identical layers)
    g0 = groups[0]
    sh_bytes = float(sum(kb[t][0] for t in g0))
    ex_bytes = float(sum(kb[t][1] for t in g0))
    dominant = "k_expand" if ex_us >= sh_us else "k_shrink"
    dom_us, dom_bytes = (ex_us, ex_bytes) if dominant == "k_expand" else (sh_us, sh_bytes)
    achieved = dom_bytes / (dom_us * 1e-6) / 1e9
    log(f"{name}: per launch of {len(g0)} tables: k_shrink {sh_us:.2f} us ({sh_bytes / sh_us / 1e3:.0f} GB/s), "
        f"k_expand {ex_us:.2f} us ({ex_bytes / ex_us / 1e3:.0f} GB/s)")

    swap = run_swaps(w, dw, ctx, plans, groups, tabs, xs, ys, stream, hip, salt) if spec.get("swaps") else None
    for p in plans:
        p.close()
    for d in xs + ys:
        d.free()
    ctx.close()
    stream.destroy()
    step_bytes = float(bytes_tab.sum())
    return {
        "workload": w.name, "T": w.T, "tables": len(w.tables),
        "ms_per_step": ms_step, "tokens_per_s": w.T / (ms_step * 1e-3),
        "step_bytes": step_bytes, "step_GBps": step_bytes / (ms_step * 1e-3) / 1e9,
        "step_frac": step_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        "step_flops": float(sum(apply_flops(w, maps, t) for t in range(n_tab))),
        "tiling": {"tile_tokens": tile_m, "tiles": n_tiles, "launches_per_apply": launches,
                   "tables_per_launch": len(g0), "launches_per_step": 2 * len(groups) + 1},
        "kernels": {"k_shrink": {"avg_us": sh_us, "bytes_per_launch": int(sh_bytes),
                                 "GBps": sh_bytes / (sh_us * 1e-6) / 1e9},
                    "k_expand": {"avg_us": ex_us, "bytes_per_launch": int(ex_bytes),
                                 "GBps": ex_bytes / (ex_us * 1e-6) / 1e9}},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": None,
                     "kernel": f"{dominant} (salt_apply_batch of {len(g0)} tables)",
                     "bytes_per_launch": int(dom_bytes), "avg_us": dom_us,
                     "timing": f"avg_us: mean duration over {sh.size} launches, from the HIP events "
                               "salt_apply_batch_timed records at the kernel's own start and end on its stream"},
        "swap": swap,
    }


def run_swaps(w, dw, ctx, plans, groups, tabs, xs, ys, stream, hip, salt, n=32, reps=20):
    """Config-4 residual swaps: 32 new users' residuals per step, pinned host
    blobs of the layer's seven tables (327,680 B at rank 2), H2D on a context's
    side stream.  The swaps go to a context of exactly those seven tables, so a
    blob is one user's real per-layer residual; the apply they overlap with runs
    on the bench's rotated tables (slots no in-flight batch reads, as the next
    step's users would be).  Reported: swap-only, apply-only and overlapped
    step times, rank 2 against rank 16, one salt_load_residuals call against one
    salt_load_residual per blob."""
    shapes = [(i, o) for _, i, o in dw.tables]
    ctx2 = salt.Context(w.dtype, shapes, 0, 0, n, 2, 1)
    ctx16 = salt.Context(w.dtype, shapes, 0, 0, n, 16, 1)
    nb2, nb16 = ctx2.residual_bytes(2), ctx16.residual_bytes(16)
    src = dw.residual_blob(int(w.referenced_slots()[0]))
    bufs2 = [salt.HostBuffer(nb2) for _ in range(n)]
    bufs16 = [salt.HostBuffer(nb16) for _ in range(n)]
    for b in bufs2:
        b.view(np.uint16)[:] = src
    for b in bufs16:
        b.view(np.uint16)[:] = np.tile(src, 8)

    def swap2(r=0):
        assert ctx2.load_residuals_ptr(list(range(n)), [2] * n, [b.ptr for b in bufs2], [nb2] * n) == 0

    def swap2_each(r=0):
        for i, b in enumerate(bufs2):
            assert ctx2.load_residual_ptr(i, 2, b.ptr, nb2) == 0

    def swap16(r=0):
        assert ctx16.load_residuals_ptr(list(range(n)), [16] * n, [b.ptr for b in bufs16], [nb16] * n) == 0

    def apply_step(k):
        slot = k % len(plans)
        plans[slot].build(stream.h)
        for g in groups:
            tt = tabs(slot, g)
            ctx.apply_batch(tt, plans[slot], [xs[i].ptr for i in tt], [ys[i].ptr for i in tt], stream.h)

    def timed(fn):
        out = []
        for r in range(reps + 2):
            hip.synchronize()
            t0 = time.perf_counter()
            fn(r)
            stream.synchronize()
            ctx2.wait_loads()
            ctx16.wait_loads()
            if r >= 2:
                out.append(time.perf_counter() - t0)
        return float(np.median(out)) * 1e6

    apply_us = timed(apply_step)
    swap_us = timed(swap2)
    swap_each_us = timed(swap2_each)
    swap16_us = timed(swap16)
    both_us = timed(lambda r: (swap2(), apply_step(r)))
    for b in bufs2 + bufs16:
        b.free()
    ctx2.close()
    ctx16.close()
    r = {"blobs_per_step": n, "bytes_per_blob_r2": int(nb2), "bytes_per_blob_r16": int(nb16),
         "swap_only_us": swap_us, "swap_only_GBps": n * nb2 / (swap_us * 1e-6) / 1e9,
         "swap_one_call_per_blob_us": swap_each_us,
         "swap_r16_us": swap16_us, "swap_r16_GBps": n * nb16 / (swap16_us * 1e-6) / 1e9,
         "r16_over_r2_time": swap16_us / swap_us, "r16_over_r2_bytes": nb16 / nb2,
         "apply_only_step_us": apply_us, "overlapped_step_us": both_us,
         "timing": f"host wall time from the first enqueue until every stream involved has drained, median of "
                   f"{reps}"}
    log(f"swaps: {n} x {nb2} B rank 2 in {swap_us:.1f} us ({r['swap_only_GBps']:.1f} GB/s; one call per blob "
        f"{swap_each_us:.1f} us), rank 16 {swap16_us:.1f} us ({r['swap_r16_GBps']:.1f} GB/s); apply-only step "
        f"{apply_us:.1f} us, overlapped {both_us:.1f} us")
    return r


# committed rocprofv3 counter summaries: HBM traffic per launch of the dominant
# kernel, valid only for the kernel source they were taken on
TRAFFIC_PROFILES = {
    "prefill": "profiles/k_expand_llama32-3b_28layer_prefill_T8192_hbm_traffic.md",
    "qproj": "profiles/k_shrink_k_expand_llama32-3b_qproj_decode_T64_hbm_traffic.md",
    "decode8b": "profiles/k_shrink_k_expand_llama31-8b_decode_T256_trace_traffic.md",
    "zipf": "profiles/k_shrink_k_expand_llama32-3b_zipf_T512_trace_traffic.md",
}


def read_fields(path):
    fields = {}
    for line in open(path):
        if ":" in line:
            k, v = line.split(":", 1)
            fields[k.strip().lstrip("- ").strip()] = v.strip()
    return fields


def measured_traffic(workload, kernel):
    """Bytes per launch of `kernel` from the committed counter summary of this
    workload, or None when there is none or the kernel sources changed since."""
    rel = TRAFFIC_PROFILES.get(workload)
    if rel is None or not os.path.exists(os.path.join(ROOT, rel)):
        return None
    f = read_fields(os.path.join(ROOT, rel))
    if f.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    key = f"traffic_bytes_per_launch_{kernel}"
    return int(f[key]) if key in f else None


def gram_workload(rank=16):
    """Two rank-`rank` adapters over the 196 tables of the 28-layer Llama-3.2-3B, in
    residual-blob layout (slots 0 and 1 of a seeded workload)."""
    from paper_2608_03579_amd import synth
    tables = synth.make(3, 0).tables
    z = np.zeros(1, np.int32)
    return synth.Workload(cfg=7, seed=1, name="gram", dtype="bf16", tables=tables, n_centroids=0, r_c=0,
                          n_slots=2, r_u_max=rank, slot_rank=np.array([rank, rank], np.int32), tok_c=z - 1,
                          tok_u=z - 1, gamma=None)


def run_gram(args, hip, salt, rank=16):
    w = gram_workload(rank)
    tables = [(i, o) for _, i, o in w.tables]
    ctx = salt.Context("bf16", tables, 0, 0, 1, 0, 1)
    d1 = hip.DeviceArray.from_host(w.residual_blob(0))
    d2 = hip.DeviceArray.from_host(w.residual_blob(1))
    stream = hip.Stream()
    nbytes = 2 * rank * sum(i + o for i, o in tables) * 2
    for _ in range(args.warmup):
        ctx.adapter_gram(d1.ptr, rank, d2.ptr, rank, stream.h)
    e0, e1 = hip.Event(), hip.Event()
    times, walls = [], []
    for _ in range(args.steps):
        t0 = time.perf_counter()
        e0.record(stream)
        terms = ctx.adapter_gram(d1.ptr, rank, d2.ptr, rank, stream.h)
        e1.record(stream)
        stream.synchronize()
        walls.append(time.perf_counter() - t0)
        times.append(e0.elapsed_ms(e1))
    cos = terms[:, 0] / (np.sqrt(terms[:, 1] * terms[:, 2]) + 1e-8)
    ms = float(np.median(times))
    log(f"gram: {len(tables)} tables, {nbytes / 1e6:.1f} MB of factors; stream time {ms * 1e3:.1f} us "
        f"(median of {args.steps}), call wall {np.median(walls) * 1e6:.1f} us; |cos| max {np.abs(cos).max():.4f}")
    e0.destroy(); e1.destroy()
    d1.free(); d2.free()
    ctx.close()
    return w, {"ms": ms, "wall_ms": float(np.median(walls)) * 1e3, "bytes": nbytes}


def cpu_gram_baseline(w, rank=16, budget_s=12.0):
    """GB/s of the oracle (dense updates formed in float64, one BLAS thread) on the
    same tables, counted with the same bytes of factors."""
    import oracle
    from threadpoolctl import threadpool_limits
    done, nbytes = 0, 0.0
    with threadpool_limits(limits=1):
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < budget_s and done < len(w.tables):
            at1, b1 = (oracle.decode(a, "bf16") for a in w.residual(0, done))
            at2, b2 = (oracle.decode(a, "bf16") for a in w.residual(1, done))
            oracle.update_terms(at1, b1, at2, b2)
            nbytes += 2 * rank * (at1.shape[1] + b1.shape[1]) * 2
            done += 1
        dt = time.perf_counter() - t0
    return {"value": nbytes / dt / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"{done} of {len(w.tables)} tables (dense updates in fp64) in {dt:.1f} s; BLAS limited to "
                      f"1 thread; host has {os.cpu_count()} logical cpus"}


def fuse_bytes(n_in, n_out, r_c, esize=2):
    """Algorithmic bytes of one salt_fuse_centroid: W read and written once, the
    centroid's A and B read once."""
    return esize * (2 * n_in * n_out + r_c * (n_in + n_out))


def run_fuse(w, args, hip, salt):
    """One step = centroid 0 of every table folded into that table's base weight
    (gamma alternating +0.8 / -0.8 between steps so the weights stay put); the
    weights rotate over `rot` copies."""
    tables = [(i, o) for _, i, o in w.tables]
    n_tab = len(tables)
    ctx = salt.Context(w.dtype, tables, w.n_centroids, w.r_c, 1, 0, 1)
    for t in range(n_tab):
        at, b = w.centroids(t)
        ctx.pin_centroids(t, at, b)
    stream = hip.Stream()
    rot = WORKLOADS["fuse"]["rot"]
    ws = []
    for k in range(rot):
        for t in range(n_tab):
            ws.append(hip.DeviceArray.from_host(w.base_weight(t)))
    hip.synchronize()
    bytes_tab = np.array([fuse_bytes(i, o, w.r_c) for i, o in tables], dtype=np.float64)

    def step(k):
        g = 0.8 if k % 2 == 0 else -0.8
        base = (k % rot) * n_tab
        for t in range(n_tab):
            ctx.fuse_centroid(t, 0, g, ws[base + t].ptr, tables[t][1], stream.h)

    for k in range(args.warmup):
        step(k)
    stream.synchronize()
    e0, e1 = hip.Event(), hip.Event()
    e0.record(stream)
    for k in range(args.steps):
        step(k)
    e1.record(stream)
    stream.synchronize()
    ms_step = e0.elapsed_ms(e1) / args.steps
    n_meas = 20
    ev = [hip.Event() for _ in range(2 * n_meas)]
    per_tab = np.zeros(n_tab)
    for t in range(n_tab):
        for k in range(n_meas):
            ctx.fuse_centroid_timed(t, 0, 0.8 if k % 2 == 0 else -0.8, ws[(k % rot) * n_tab + t].ptr,
                                    tables[t][1], stream.h, ev[2 * k].h, ev[2 * k + 1].h)
        stream.synchronize()
        per_tab[t] = float(np.mean([ev[2 * k].elapsed_ms(ev[2 * k + 1]) for k in range(n_meas)]))
    for e in ev + [e0, e1]:
        e.destroy()
    for d in ws:
        d.free()
    ctx.close()
    dom = int(np.argmax(per_tab))
    achieved = bytes_tab[dom] / (per_tab[dom] * 1e-3) / 1e9
    log(f"fuse durations (us): " + ", ".join(f"{w.tables[t][0]} {per_tab[t] * 1e3:.2f}" for t in range(n_tab)))
    return {"ms_per_step": ms_step, "step_GBps": bytes_tab.sum() / (ms_step * 1e-3) / 1e9,
            "fuse_us": {w.tables[t][0]: round(per_tab[t] * 1e3, 3) for t in range(n_tab)},
            "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                         "frac": achieved / HBM_PEAK_GBPS, "traffic": None,
                         "kernel": f"k_fuse (salt_fuse_centroid) on {w.tables[dom][0]}",
                         "bytes_per_launch": int(bytes_tab[dom]), "avg_us": per_tab[dom] * 1e3,
                         "timing": f"avg_us: mean kernel duration over {n_meas} calls from HIP events that record "
                                   "the kernel's own start and end (salt_fuse_centroid_timed)"}}


def tables_summary(w):
    groups = layer_groups(w)
    names = [n.split(".", 1)[-1] for n, _, _ in (w.tables[t] for t in groups[0])]
    shapes = [f"{n} {w.tables[t][1]}->{w.tables[t][2]}" for n, t in zip(names, groups[0])]
    return f"{len(groups)} layers x [{', '.join(shapes)}]" if len(groups) > 1 else ", ".join(shapes)


def sub_record(name, res):
    keep = ("workload", "T", "tables", "ms_per_step", "tokens_per_s", "step_bytes", "step_GBps", "step_frac",
            "tiling", "kernels")
    r = {k: res[k] for k in keep}
    r["roofline"] = {k: res["roofline"][k] for k in ("kernel", "achieved", "frac", "avg_us", "bytes_per_launch")}
    r["roofline"]["traffic"] = measured_traffic(name, res["roofline"]["kernel"].split()[0])
    if res.get("swap"):
        r["swap"] = res["swap"]
    return r


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--workload", default="prefill", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-sub", action="store_true", help="skip the decode / Zipf sub-records")
    ap.add_argument("--meas", type=int, default=None, help="timed launches per table group for the roofline")
    ap.add_argument("--copy-mb", type=int, default=0,
                    help="also run a device-to-device copy of this many MiB (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: libsalt has no cross-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)
    spec = WORKLOADS[args.workload]
    steps = args.steps if args.steps is not None else spec["steps"]
    warmup = args.warmup if args.warmup is not None else spec["warmup"]
    args.steps, args.warmup = steps, warmup

    from paper_2608_03579_amd import hip, salt
    if hip.device_count() < 1:
        print("no HIP device visible", file=sys.stderr)
        sys.exit(1)
    hip.set_device(0)
    if spec.get("gram"):
        w, res = run_gram(args, hip, salt)
        cpu = None if args.no_cpu else cpu_gram_baseline(w)
        achieved = res["bytes"] / (res["ms"] * 1e-3) / 1e9
        print(json.dumps({
            "metric": "Adapter cosine in factor space (Sec. 3.1 Eq. 2, Sec. 4.5): achieved HBM GB/s, Llama-3.2-3B",
            "value": achieved, "unit": "GB/s", "n_gpus": 1, "steps": steps, "warmup": warmup,
            "ms_per_step": res["ms"], "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": "bf16", "data": "synthetic",
            "config": {"workload": "two rank-16 adapters, 196 tables of the 28-layer Llama-3.2-3B"},
            "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                         "frac": achieved / HBM_PEAK_GBPS, "traffic": None,
                         "kernel": "k_gram + k_gram_finish (salt_adapter_gram)",
                         "bytes_per_launch": res["bytes"], "avg_us": res["ms"] * 1e3,
                         "timing": "avg_us: median stream time of the whole call between HIP events"},
            "cpu_baseline": cpu}), flush=True)
        return
    if spec.get("fuse"):
        w, _ = make_workload(spec)
        res = run_fuse(w, args, hip, salt)
        print(json.dumps({
            "metric": "Centroid fused into the base weights (Sec. 3.3 node start-up): achieved HBM GB/s, "
                      "Llama-3.2-3B",
            "value": res["step_GBps"], "unit": "GB/s", "n_gpus": 1, "steps": steps, "warmup": warmup,
            "ms_per_step": res["ms_per_step"], "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": "bf16", "data": "synthetic",
            "config": {"workload": "llama3.2-3b one layer, centroid fused into the base weights"},
            "fuse_us": res["fuse_us"], "roofline": res["roofline"], "cpu_baseline": None}), flush=True)
        return

    w, dw = make_workload(spec)
    res = run_gpu(args.workload, w, dw, spec, steps, warmup, hip, salt, args.meas)
    dom = res["roofline"]["kernel"].split()[0]
    res["roofline"]["traffic"] = measured_traffic(args.workload, dom)
    subs = {}
    if args.workload == "prefill" and not args.no_sub:
        for name, s_steps, s_warm in SUB_RECORDS:
            sw, sdw = make_workload(WORKLOADS[name])
            subs[name] = sub_record(name, run_gpu(name, sw, sdw, WORKLOADS[name], s_steps, s_warm, hip, salt))
        z, zb = subs["zipf"], subs["zipf-baseline"]
        subs["zipf_salt_vs_rank16_baseline"] = {
            "bytes_ratio_baseline_over_salt": zb["step_bytes"] / z["step_bytes"],
            "tokens_per_s_ratio_salt_over_baseline": z["tokens_per_s"] / zb["tokens_per_s"]}
    cpu = None
    if not args.no_cpu:
        log("cpu baseline (oracle) ...")
        cpu = cpu_baseline(w, dw)
    if args.copy_mb:
        log(f"copy calibration: {args.copy_mb} MiB device-to-device")
        a_ = hip.DeviceArray((args.copy_mb << 20,), np.uint8)
        b_ = hip.DeviceArray((args.copy_mb << 20,), np.uint8)
        s_ = hip.Stream()
        for _ in range(3):
            b_.copy_from(a_, s_)
        s_.synchronize()
        a_.free()
        b_.free()
    out = {
        "metric": METRIC,
        "value": res["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "T": w.T, "tables": tables_summary(w),
                   "centroids": f"{w.n_centroids} x r{w.r_c}", "residual_slots": f"{w.n_slots} x r<={w.r_u_max}",
                   "accumulation": "fp32", "rotation": spec["rot"],
                   "step": "salt_plan_build + one salt_apply_batch per decoder layer (its 7 tables); maps staged "
                           "in HBM beforehand"},
        "achieved_GBps_step": res["step_GBps"],
        "step_bytes": res["step_bytes"],
        "tiling": res["tiling"],
        "kernels": res["kernels"],
        "roofline": res["roofline"],
        "cpu_baseline": cpu,
        "swap": res["swap"],
        "sub_records": subs or None,
        "kernel_source_sha256_16": kernel_source_hash(),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
