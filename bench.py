"""Benchmark: mixed-depth loop-step throughput of continuous depth batching.

One step = one cdb_loop_step over a mixed-depth decode batch of the
Ouro-1.4B-shaped looped LM (d 2048, 16 heads x 128, SwiGLU 5632, 24 core
layers, r_max 4, 16-token pages, depth-indexed KV per (sequence, loop, layer)).
The batch is 64 rows, one per sequence, as it stands mid-decode in refill mode:
positions drawn from the decode range of a 512-token prompt + 256 decode
tokens, exit depths from the categorical {1: .3, 2: .3, 3: .2, 4: .2}
size-biased by work items, loop indices below the depth.  Weights are seeded
random N(0, 0.02) in bf16; KV contents and states are random; everything is
resident in HBM before timing starts.

Prints one JSON line: loop-step rows (tokens) per second, ms per step, the
roofline of the dominant kernel (paged attention, HBM-bound) and the CPU
oracle's rate on a bounded sample of the same workload.  The "e2e" object
times whole decodes of the same workload through the host driver -- 64
requests, 256 decode tokens each after a 512-token prompt whose KV is
synthesized -- under CDB with refill, CDB without refill, and fixed-depth
continuous batching, next to the FLOP bound on the speed-up (Section 5, Eq. 2).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_attn_ouro_bs64_hbm_traffic.json")
# the decode attention kernel's source: its file and the device helpers it includes
ATTN_SRC = [os.path.join(ROOT, "paper_2608_09444_amd", "csrc", f) for f in ("attention.hip", "cdb_internal.h")]


def attention_source_sha256():
    import hashlib
    h = hashlib.sha256()
    for f in ATTN_SRC:
        h.update(open(f, "rb").read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per attention launch from the committed FETCH_SIZE / WRITE_SIZE
    passes, if they were taken on the attention source as it stands."""
    try:
        rec = json.load(open(TRAFFIC_FILE))
        if rec["attention_source_sha256"] != attention_source_sha256():
            return None
        return int(rec["hbm_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def setup(shape, w, n_rows, pos_lo, pos_hi, seed_stream=7):
    import numpy as np
    import torch

    import cdbgen
    import paper_2608_09444_amd as cdb
    dm = cdb.DeviceModel(shape, w)
    rows_np = cdbgen.decode_snapshot(n_rows, cdbgen.OURO_DEPTHS, shape.r_max, pos_lo, pos_hi, stream=seed_stream)
    max_pages = cdbgen.pages_for(pos_hi + 1)
    n_pages = n_rows * max_pages * shape.r_max
    kv = cdb.PagedKV(shape, n_rows, max_pages, 0, n_pages, 0, fill="random")
    g = torch.Generator(device="cuda")
    g.manual_seed(1234)
    kv.core.normal_(0.0, 1.0, generator=g)
    pt = np.arange(n_pages, dtype=np.int32).reshape(n_rows, max_pages, shape.r_max).transpose(0, 2, 1)
    full = np.full((n_rows, shape.r_max + 2, max_pages), -1, np.int32)
    full[:, 1:shape.r_max + 1, :] = pt
    kv.page_table.copy_(torch.from_numpy(full))
    state = cdb.State(shape, n_rows)
    state.h.normal_(0.0, 1.0, generator=g)
    rows = cdb.Rows(rows_np["slot"], rows_np["seq"], rows_np["pos"], rows_np["c"], rows_np["depth"])
    out = cdb.StepOut(n_rows)
    ws = cdb.Workspace(dm.desc, n_rows)
    torch.cuda.synchronize()
    return dm, kv, state, rows, rows_np, out, ws


def attention_bytes(shape, pos):
    """Algorithmic bytes of one paged-attention launch (one layer): K and V of
    every visible position of each row, q in (fp32) and the output (bf16)."""
    import numpy as np
    ctx = np.asarray(pos, dtype=np.int64) + 1
    return int(ctx.sum()) * 2 * shape.d * 2 + len(ctx) * shape.d * (4 + 2)


def step_bytes(shape, rows_np):
    """Algorithmic bytes of one loop step: core weights once, every layer's K/V
    over the visible context, the new K/V entries, copy-on-exit traffic, and the
    row states in and out."""
    import numpy as np
    import cdbgen
    pc = cdbgen.param_counts(shape)
    w = pc["core"] * 2 + shape.d * 2
    kv_tok = shape.n_core * 2 * shape.d * 2
    ctx = rows_np["pos"].astype(np.int64) + 1
    ex = rows_np["c"] + 1 == rows_np["depth"]
    copies = int(((shape.r_max - rows_np["depth"]) * ex).sum())
    n = len(ctx)
    return w + int(ctx.sum()) * kv_tok + n * kv_tok + copies * 2 * kv_tok + n * shape.d * 4 * 2


def step_flops(shape, rows_np):
    import numpy as np
    import cdbgen
    n = len(rows_np["pos"])
    ctx = rows_np["pos"].astype(np.int64) + 1
    return 2 * n * cdbgen.param_counts(shape)["core"] + 4 * shape.n_core * shape.d * int(ctx.sum())


def time_attention(shape, kv, rows, n_rows, launches):
    """Average duration of the paged-attention kernel on the loop-step batch,
    timed with events on the stream it is launched on (the row order is computed
    once and passed, so only the attention kernel runs per launch)."""
    import torch
    import paper_2608_09444_amd as cdb
    q = torch.randn((n_rows, shape.d), dtype=torch.float32, device="cuda")
    o = torch.empty((n_rows, shape.d), dtype=torch.bfloat16, device="cuda")
    ws = torch.zeros(256 + 4 * 256, dtype=torch.uint8, device="cuda")
    desc = cdb.make_desc(shape)
    st = torch.cuda.current_stream()
    cdb.cdb_paged_attention(desc, kv.c, rows.c, 1, 0, q, o, ws)  # computes the row order into ws[256:]
    order = ws.data_ptr() + 256
    for i in range(5):
        cdb.cdb_paged_attention(desc, kv.c, rows.c, 1, i % shape.n_core, q, o, ws, order=order)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(st)
    for i in range(launches):
        cdb.cdb_paged_attention(desc, kv.c, rows.c, 1, i % shape.n_core, q, o, ws, order=order)
    e1.record(st)
    e1.synchronize()
    return e0.elapsed_time(e1) / launches


def runner_ws(dm, rows, two):
    """The driver runner's workspace: one stage workspace, or two halves when
    the boundary stages run on their own stream (error words start at zero).
    Returns (buffer, half)."""
    import torch

    import paper_2608_09444_amd as cdb
    n = (cdb.cdb_workspace_bytes(dm.desc, rows) + 255) & ~255
    return torch.zeros(2 * n if two else n, dtype=torch.uint8, device="cuda"), n


def check_runner_ws(ws, half, what):
    import paper_2608_09444_amd as cdb
    codes = [cdb.cdb_read_device_error(ws)] + ([cdb.cdb_read_device_error(ws[half:])] if ws.numel() > half else [])
    if any(codes):
        raise RuntimeError(f"device error {codes} in {what}")


def host_threads():
    """The host cores this process may use: its CPU affinity, capped by
    OMP_NUM_THREADS when set (the job's CPU share on a shared host)."""
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    omp = os.environ.get("OMP_NUM_THREADS")
    if omp and omp.isdigit() and int(omp) > 0:
        n = min(n, int(omp))
    return max(1, n)


def host_info():
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    aff = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else None
    return {"nproc": os.cpu_count(), "affinity_cpus": aff, "omp_num_threads": os.environ.get("OMP_NUM_THREADS"),
            "cpu_model": model}


def reduced_legs(args):
    """Which legs run below their workload's full size in this invocation."""
    red = {}
    if 0 < args.serving_requests < 2000:
        red["serving"] = f"{args.serving_requests} of the trace's 2000 requests (--serving-requests 2000 for all)"
    if 0 < args.huginn_decode < 512:
        red["huginn_e2e"] = f"{args.huginn_decode} of 512 decode tokens per request"
    if args.no_long_context:
        red["long_context"] = "not run (--no-long-context)"
    if args.huginn_decode == 0:
        red["huginn"] = "not run"
    return red


def cpu_baseline(shape, w, rows_np, n_sample, threads, min_s=10.0):
    """The CPU oracle's loop step on `n_sample` rows of the same batch (same
    positions, depths, loop indices; seeded random KV and state)."""
    import numpy as np
    os.environ["OMP_NUM_THREADS"] = str(threads)
    import cdbgen
    import oracle
    threads = oracle.set_threads(threads)
    m = oracle.Model(shape, w, bf16_storage=True)
    idx = np.arange(n_sample)
    pos = rows_np["pos"][idx]
    pages = [cdbgen.pages_for(int(p) + 1) for p in pos]
    maxp = max(pages)
    # the row's plane over its whole context, plus the page at pos of every
    # deeper plane (copy-on-exit destinations)
    need = sum(pages) + sum(shape.r_max - int(rows_np["c"][i]) - 1 for i in idx)
    paged = oracle.Paged(shape, n_sample, maxp, 0, need, 0)
    nxt = 0
    for i in range(n_sample):
        plane = int(rows_np["c"][i]) + 1
        for pg in range(pages[i]):
            paged.page_table[i, plane, pg] = nxt
            nxt += 1
        for pl in range(plane + 1, shape.r_max + 1):
            paged.page_table[i, pl, pages[i] - 1] = nxt
            nxt += 1
    kvbits = cdbgen.random_kv_bf16(paged.core.shape, seed=5)
    paged.core[...] = cdbgen.bf16_to_f32(kvbits)
    del kvbits
    h = cdbgen.random_state(n_sample, shape.d, seed=6).astype(np.float64)
    slot = idx.astype(np.int32)
    # repeat the step on the same rows until at least min_s of CPU time
    steps, t0 = 0, time.perf_counter()
    while True:
        oracle.loop_step(m, paged, h, None, slot, slot, pos, rows_np["c"][idx], rows_np["depth"][idx])
        steps += 1
        dt = time.perf_counter() - t0
        if dt >= min_s or steps >= 50:
            break
    return {"value": n_sample * steps / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{n_sample} of the {len(rows_np['pos'])} rows of the timed batch (same positions, loop "
                      f"indices and depths; seeded random KV/state), {steps} loop steps in {dt:.1f}s"}


def e2e_decode(shape, dm, kv, n_seqs, prompt, n_decode, seed=3):
    """Whole decodes through the host driver in three modes; the KV pool's
    random contents stand in for the prompts' prefilled KV."""
    import numpy as np
    import torch

    import cdbgen
    import paper_2608_09444_amd as cdb
    from paper_2608_09444_amd import cost
    from paper_2608_09444_amd import driver as drv
    R = shape.r_max
    depths = [cdbgen.draw_depths(cdbgen.OURO_DEPTHS, n_decode, R, seed=seed, stream=q) for q in range(n_seqs)]
    mean_depth = float(np.mean(np.concatenate(depths)))
    first = cdbgen.prompt_ids(shape.vocab, 1, n_seqs, seed=seed + 1)[0]
    max_pages = kv.c.max_pages
    state = cdb.State(shape, n_seqs)
    ws = cdb.Workspace(dm.desc, 256)
    out_ids = torch.empty((n_seqs, n_decode), dtype=torch.int32, device="cuda")

    def run(n, nd, dep=None, **mode):
        d = drv.Driver(max_batch=64, max_active=n, r_max=R, max_seqs=n_seqs, max_pages=max_pages,
                       core_pages=kv.c.core_pages, **mode)
        for q in range(n):
            d.add_sequence(prompt, (depths if dep is None else dep)[q][:nd])
        scratch = torch.empty(d.scratch_bytes(shape.vocab), dtype=torch.uint8, device="cuda")
        rws, half = runner_ws(dm, 256, mode.get("boundary_stream", False))
        secs = d.run(dm.model, kv.c, state.c, scratch, first, rws, tokens_out=out_ids)
        check_runner_ws(rws, half, "the driver run")
        return secs, d.stats()

    run(4, 8)  # first use of the boundary kernels
    res = {"workload": f"{n_seqs} requests, prompt {prompt} (KV synthesized), {n_decode} decode tokens each, "
                       f"depths categorical {{1:.3,2:.3,3:.2,4:.2}}, max batch 64, full depth-indexed KV",
           "mean_depth": round(mean_depth, 4), "flop_bound": round(cost.flop_bound(shape, mean_depth), 4)}
    run(4, 8, boundary_stream=1)
    run(4, 8, graph_loop=True)
    for name, mode in (("cdb_refill", {}), ("cdb_no_refill", {"refill": False}), ("cb_fixed_depth",
                                                                               {"fixed_depth": True}),
                       ("cdb_refill_boundary_stream_fill", {"boundary_stream": 1}),
                       ("cdb_refill_boundary_stream_hold", {"boundary_stream": 2}),
                       ("cdb_refill_graph", {"graph_loop": True})):
        secs, st = run(n_seqs, n_decode, **mode)
        res[name] = {"tokens_per_s": round(st["tokens"] / secs, 1), "seconds": round(secs, 4),
                     "loop_steps": st["loop_steps"], "idle_rows": st["idle_rows"],
                     "coda_calls": st["coda_calls"],
                     "host_wait_us_per_loop_step": round(st["host_wait_us"] / max(1, st["loop_steps"]), 2)}
        log(f"e2e {name}: {st['tokens']} tokens in {secs:.3f}s, {st['loop_steps']} loop steps")
    cb = res["cb_fixed_depth"]["tokens_per_s"]
    res["speedup_refill_vs_cb"] = round(res["cdb_refill"]["tokens_per_s"] / cb, 4)
    res["graph_gain"] = round(res["cdb_refill_graph"]["tokens_per_s"] / res["cdb_refill"]["tokens_per_s"], 4)
    res["speedup_no_refill_vs_cb"] = round(res["cdb_no_refill"]["tokens_per_s"] / cb, 4)
    # no early exits (every token at r_max): CDB can gain nothing, so its ratio
    # to fixed depth is the scheduler's own overhead (Section 6.2)
    secs_nx, st_nx = run(n_seqs, n_decode, dep=[np.full(n_decode, R, np.int32)] * n_seqs)
    res["no_exit"] = {"cdb_refill_tokens_per_s": round(st_nx["tokens"] / secs_nx, 1), "seconds": round(secs_nx, 4),
                      "loop_steps": st_nx["loop_steps"],
                      "ratio_vs_cb": round(st_nx["tokens"] / secs_nx / cb, 4)}
    log(f"e2e no exits: {st_nx['tokens']} tokens in {secs_nx:.3f}s, {st_nx['loop_steps']} loop steps")

    # device-decided exits (gate score >= 0.5): with the lookahead the host
    # plans each loop step from decisions one step old; without it every loop
    # step waits for its own decisions (the GPU idles for the round trip)
    def run_gated(lookahead):
        d = drv.Driver(max_batch=64, max_active=n_seqs, r_max=R, max_seqs=n_seqs, max_pages=max_pages,
                       core_pages=kv.c.core_pages, gated=True, lookahead=lookahead, threshold=0.5)
        for q in range(n_seqs):
            d.add_sequence(prompt, None, n_decode=n_decode)
        scratch = torch.empty(d.scratch_bytes(shape.vocab), dtype=torch.uint8, device="cuda")
        secs = d.run(dm.model, kv.c, state.c, scratch, first, ws.buf, tokens_out=out_ids)
        if cdb.cdb_read_device_error(ws.buf) != 0:
            raise RuntimeError("device error in the gated driver run")
        st = d.stats()
        return {"tokens_per_s": round(st["tokens"] / secs, 1), "seconds": round(secs, 4),
                "loop_steps": st["loop_steps"], "mean_depth": round(st["loop_rows"] / st["tokens"], 4),
                "ms_per_loop_step": round(secs * 1e3 / st["loop_steps"], 4)}

    ga, gs = run_gated(True), run_gated(False)
    res["gated"] = {"threshold": 0.5, "lookahead": ga, "synchronous": gs}
    log(f"e2e gated: lookahead {ga['tokens_per_s']} tokens/s (depth {ga['mean_depth']}), synchronous "
        f"{gs['tokens_per_s']} tokens/s (depth {gs['mean_depth']})")
    # the same replayed refill run with the runner waiting after every loop
    # step: the device idles for each round trip and planning (what planning
    # one step ahead removes)
    secs_sync, st_sync = run(n_seqs, n_decode, sync_steps=True)
    a = res["cdb_refill"]["seconds"]
    res["sync_ablation"] = {"async_seconds": a, "sync_seconds": round(secs_sync, 4),
                            "idle_us_per_loop_step": round((secs_sync - a) / st_sync["loop_steps"] * 1e6, 2),
                            "slowdown": round(secs_sync / a, 4)}
    log(f"e2e sync ablation: {secs_sync:.3f}s vs {a:.3f}s asynchronous")
    return res


def own_pages(shape, rows_np, max_pages):
    """Page table [rows][r_max + 2][max_pages] of a loop-step snapshot in which
    every row maps its own pages: its loop plane over the whole context plus the
    page at pos of every deeper plane (copy-on-exit destinations).  Returns the
    table and the number of core pages it uses."""
    import numpy as np
    import cdbgen
    R = shape.r_max
    n = len(rows_np["pos"])
    pt = np.full((n, R + 2, max_pages), -1, np.int32)
    nxt = 0
    for i in range(n):
        plane = int(rows_np["c"][i]) + 1
        pg = cdbgen.pages_for(int(rows_np["pos"][i]) + 1)
        pt[i, plane, :pg] = np.arange(nxt, nxt + pg)
        nxt += pg
        for pl in range(plane + 1, R + 1):
            pt[i, pl, pg - 1] = nxt
            nxt += 1
    return pt, nxt


def time_loop_step(dm, kv, state, rows, so, ws, steps, warmup):
    """Milliseconds per cdb_loop_step on one batch, timed with events."""
    import torch
    import paper_2608_09444_amd as cdb
    st = torch.cuda.current_stream()
    for _ in range(warmup):
        cdb.cdb_loop_step(dm.model, kv.c, state.c, rows.c, so.c, ws.buf)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(st)
    for _ in range(steps):
        cdb.cdb_loop_step(dm.model, kv.c, state.c, rows.c, so.c, ws.buf)
    e1.record(st)
    e1.synchronize()
    if cdb.cdb_read_device_error(ws.buf) != 0:
        raise RuntimeError("device error in a timed loop step")
    return e0.elapsed_time(e1) / steps


def batch_sweep(shape, dm, sizes=(16, 32, 64, 128, 256), pos_lo=512, pos_hi=767, steps=10, warmup=3):
    """cdb_loop_step at several batch sizes on mid-decode refill batches of the
    same position and depth distributions.  Each row maps its own pages: its
    loop plane over the whole context plus the page at pos of every deeper
    plane (copy-on-exit destinations)."""
    import numpy as np
    import torch

    import cdbgen
    import paper_2608_09444_amd as cdb
    R = shape.r_max
    out = []
    for n in sizes:
        rows_np = cdbgen.decode_snapshot(n, cdbgen.OURO_DEPTHS, R, pos_lo, pos_hi, stream=20 + n)
        max_pages = cdbgen.pages_for(pos_hi + 1)
        pt, nxt = own_pages(shape, rows_np, max_pages)
        kv = cdb.PagedKV(shape, n, max_pages, 0, nxt, 0, fill="random")
        kv.core.normal_(0.0, 1.0)
        kv.page_table.copy_(torch.from_numpy(pt))
        state = cdb.State(shape, n)
        state.h.normal_(0.0, 1.0)
        rows = cdb.Rows(np.arange(n, dtype=np.int32), np.arange(n, dtype=np.int32), rows_np["pos"], rows_np["c"],
                        rows_np["depth"])
        so = cdb.StepOut(n)
        ws = cdb.Workspace(dm.desc, n)
        ms = time_loop_step(dm, kv, state, rows, so, ws, steps, warmup)
        sb = step_bytes(shape, rows_np)
        out.append({"rows": n, "ms_per_step": round(ms, 4), "rows_per_s": round(n / (ms * 1e-3), 1),
                    "hbm_frac": round(sb / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)})
        log(f"sweep {n} rows: {ms:.3f} ms/step, {n / (ms * 1e-3):.0f} rows/s")
        del kv, state, rows, so, ws
        torch.cuda.empty_cache()
    return out


def batch_e2e(shape, dm, sizes=(16, 32, 64, 128), n_seqs=384, prompt=512, n_decode=32, seed=5):
    """Whole decodes of the same 384 requests (prompt 512 with synthesized KV,
    32 decode tokens each, config 2's categorical depths) at several maximum
    batch sizes, with as many sequences in flight as the batch holds (so at
    least 3 batches' worth of requests wait at every size): CDB refill and
    no-refill against fixed-depth continuous batching (the paper's batch-size
    sweep, Section 6.2).  The pool holds the pages of the sequences in flight."""
    import numpy as np
    import torch

    import cdbgen
    import paper_2608_09444_amd as cdb
    from paper_2608_09444_amd import driver as drv
    R = shape.r_max
    depths = [cdbgen.draw_depths(cdbgen.OURO_DEPTHS, n_decode, R, seed=seed, stream=q) for q in range(n_seqs)]
    first = cdbgen.prompt_ids(shape.vocab, 1, n_seqs, seed=seed + 1)[0]
    max_pages = cdbgen.pages_for(prompt + n_decode)
    core_pages = max(sizes) * max_pages * R
    kv = cdb.PagedKV(shape, n_seqs, max_pages, 0, core_pages, 0, fill="random")
    kv.core.normal_(0.0, 1.0)
    state = cdb.State(shape, n_seqs)
    ws = cdb.Workspace(dm.desc, 256)
    out_ids = torch.empty((n_seqs, n_decode), dtype=torch.int32, device="cuda")
    res = {"workload": f"{n_seqs} requests, prompt {prompt} (KV synthesized), {n_decode} decode tokens each, depths "
                       f"categorical {{1:.3,2:.3,3:.2,4:.2}}, sequences in flight = max batch, full depth-indexed KV",
           "points": []}
    for B in sizes:
        e = {"max_batch": B}
        for name, mode in (("cdb_refill", {}), ("cdb_no_refill", {"refill": False}),
                           ("cb_fixed_depth", {"fixed_depth": True})):
            d = drv.Driver(max_batch=B, max_active=B, r_max=R, max_seqs=n_seqs, max_pages=max_pages,
                           core_pages=core_pages, **mode)
            for q in range(n_seqs):
                d.add_sequence(prompt, depths[q])
            scratch = torch.empty(d.scratch_bytes(shape.vocab), dtype=torch.uint8, device="cuda")
            secs = d.run(dm.model, kv.c, state.c, scratch, first, ws.buf, tokens_out=out_ids)
            if cdb.cdb_read_device_error(ws.buf) != 0:
                raise RuntimeError("device error in the batch-size sweep")
            st = d.stats()
            e[name] = {"tokens_per_s": round(st["tokens"] / secs, 1), "seconds": round(secs, 4),
                       "loop_steps": st["loop_steps"]}
        cb = e["cb_fixed_depth"]["tokens_per_s"]
        e["speedup_refill_vs_cb"] = round(e["cdb_refill"]["tokens_per_s"] / cb, 4)
        e["speedup_no_refill_vs_cb"] = round(e["cdb_no_refill"]["tokens_per_s"] / cb, 4)
        res["points"].append(e)
        log(f"batch e2e, max batch {B}: refill {e['speedup_refill_vs_cb']}x, no-refill "
            f"{e['speedup_no_refill_vs_cb']}x ({cb:.0f} tokens/s fixed depth)")
    del kv, state, ws, out_ids
    torch.cuda.empty_cache()
    return res


def latency_model(shape, dm, sizes=(16, 32, 64, 128, 256), contexts=(128, 512, 2048), steps=10, warmup=3):
    """The recurrent-step latency model of the paper's Appendix A on this
    kernel set: cdb_loop_step over B equal-length rows (every row at context L,
    loop index 0, no exit), timed on a grid of B and L and fitted by least
    squares to t = delta + gamma * N_b + alpha * N_c, with N_b = B rows and N_c
    = B * L context tokens.  Each row maps its own pages."""
    import numpy as np
    import torch

    import cdbgen
    import paper_2608_09444_amd as cdb
    R = shape.r_max
    pts = []
    for L in contexts:
        for n in sizes:
            rows_np = {"pos": np.full(n, L - 1, np.int32), "c": np.zeros(n, np.int32),
                       "depth": np.full(n, R, np.int32)}
            max_pages = cdbgen.pages_for(L)
            pt, nxt = own_pages(shape, rows_np, max_pages)
            kv = cdb.PagedKV(shape, n, max_pages, 0, nxt, 0, fill="random")
            kv.core.normal_(0.0, 1.0)
            kv.page_table.copy_(torch.from_numpy(pt))
            state = cdb.State(shape, n)
            state.h.normal_(0.0, 1.0)
            rows = cdb.Rows(np.arange(n, dtype=np.int32), np.arange(n, dtype=np.int32), rows_np["pos"],
                            rows_np["c"], rows_np["depth"])
            so = cdb.StepOut(n)
            ws = cdb.Workspace(dm.desc, n)
            ms = time_loop_step(dm, kv, state, rows, so, ws, steps, warmup)
            pts.append({"rows": n, "context": L, "ms_per_step": round(ms, 4)})
            del kv, state, rows, so, ws
            torch.cuda.empty_cache()
        log(f"latency model, context {L}: " + ", ".join(f"{p['rows']} rows {p['ms_per_step']:.3f} ms"
                                                         for p in pts if p["context"] == L))
    A = np.array([[1.0, p["rows"], p["rows"] * p["context"]] for p in pts])
    t = np.array([p["ms_per_step"] for p in pts])
    coef, *_ = np.linalg.lstsq(A, t, rcond=None)
    fit = A @ coef
    r2 = 1.0 - float(np.sum((t - fit) ** 2) / np.sum((t - t.mean()) ** 2))
    delta, gamma, alpha = (float(x) for x in coef)
    res = {"points": pts, "delta_ms": round(delta, 4), "gamma_us_per_row": round(gamma * 1e3, 3),
           "alpha_ns_per_context_token": round(alpha * 1e6, 3), "r2": round(r2, 5),
           "saturation_batch": {str(L): round(delta / (gamma + alpha * L), 1) for L in (128, 8192)}}
    log(f"latency model: delta {delta:.3f} ms, gamma {gamma * 1e3:.2f} us/row, alpha {alpha * 1e6:.2f} ns/token, "
        f"R2 {r2:.4f}")
    return res


def huginn_leg(n_decode, steps=20, warmup=3):
    """The Huginn-shaped model (prelude 2, recurrent block of 4 layers with the
    input-injection adapter looped up to 32 times, coda 2; d 5280, 55 x 96
    heads): the loop step at its mid-decode refill batch (128 rows at positions
    U[256, 767], lognormal depths, median 12, clipped to [4, 32]), and whole
    decodes through the host driver, CDB refill against fixed-depth continuous
    batching.  The decodes use the shared KV layout (one core plane per
    position, as in the paper's own runs): the depth-indexed layout of 128
    requests of 768 positions would take 274 GB.  The boundary stages wait for
    32 rows (or for the loop work to run out), the minimum boundary batch the
    paper sets for this model (Section 6.1): each prelude + coda pass streams
    more weight bytes (4 layers and a 65536-row LM head) than the core."""
    import numpy as np
    import torch

    import cdbgen
    import paper_2608_09444_amd as cdb
    from paper_2608_09444_amd import cost
    from paper_2608_09444_amd import driver as drv
    shape = cdbgen.HUGINN
    wl = cdbgen.WORKLOADS[3]
    R = shape.r_max
    t0 = time.time()
    w = cdbgen.model_weights(shape)
    dm = cdb.DeviceModel(shape, w)
    del w
    log(f"huginn: weights in {time.time() - t0:.1f}s")
    n_rows, pos_lo, pos_hi = wl.n_seqs, wl.prompt, wl.prompt + wl.decode - 1
    rows_np = cdbgen.decode_snapshot(n_rows, wl.depth, R, pos_lo, pos_hi, stream=30)
    max_pages = cdbgen.pages_for(pos_hi + 1)
    pt, n_pages = own_pages(shape, rows_np, max_pages)
    kv = cdb.PagedKV(shape, n_rows, max_pages, 0, n_pages, 0, fill="random")
    kv.core.normal_(0.0, 1.0)
    kv.page_table.copy_(torch.from_numpy(pt))
    state = cdb.State(shape, n_rows)
    state.h.normal_(0.0, 1.0)
    state.e.normal_(0.0, 1.0)
    rows = cdb.Rows(np.arange(n_rows, dtype=np.int32), np.arange(n_rows, dtype=np.int32), rows_np["pos"],
                    rows_np["c"], rows_np["depth"])
    so = cdb.StepOut(n_rows)
    ws = cdb.Workspace(dm.desc, n_rows)
    ms = time_loop_step(dm, kv, state, rows, so, ws, steps, warmup)
    sb = step_bytes(shape, rows_np)
    attn_ms = time_attention(shape, kv, rows, n_rows, steps * shape.n_core)
    ab = attention_bytes(shape, rows_np["pos"])
    log(f"huginn loop step: {ms:.3f} ms, {n_rows / (ms * 1e-3):.0f} rows/s; attention {attn_ms * 1e3:.1f} us")
    res = {"loop_step": {
        "workload": f"huginn-3.5b-shaped looped LM, mixed-depth decode loop step: {n_rows} rows at positions "
                    f"U[{pos_lo},{pos_hi}] (prompt {wl.prompt} + decode {wl.decode}), depths lognormal median 12, "
                    f"sigma 0.5, clipped to [4, 32]",
        "rows": n_rows, "ms_per_step": round(ms, 4), "tokens_per_s": round(n_rows / (ms * 1e-3), 1),
        "mean_context": float(np.mean(rows_np["pos"] + 1)),
        "exits_per_step": int((rows_np["c"] + 1 == rows_np["depth"]).sum()),
        "step_roofline": {"bound": "hbm", "algorithmic_bytes": sb, "achieved": round(sb / (ms * 1e-3) / 1e9, 1),
                          "peak": HBM_PEAK_GBS, "unit": "GB/s",
                          "frac": round(sb / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                          "flops": step_flops(shape, rows_np)},
        "attention_roofline": {"bound": "hbm", "kernel": "k_attn<96> (paged decode attention, one layer)",
                               "achieved": round(ab / (attn_ms * 1e-3) / 1e9, 1), "peak": HBM_PEAK_GBS,
                               "unit": "GB/s", "frac": round(ab / (attn_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                               "algorithmic_bytes": ab, "us_per_launch": round(attn_ms * 1e3, 2)}}}
    del kv, state, rows, so, ws
    torch.cuda.empty_cache()

    # whole decodes, shared layout: one core page per 16 positions and stage
    n_seqs, prompt = wl.n_seqs, wl.prompt
    depths = [cdbgen.draw_depths(wl.depth, n_decode, R, seed=3, stream=q) for q in range(n_seqs)]
    mean_depth = float(np.mean(np.concatenate(depths)))
    first = cdbgen.prompt_ids(shape.vocab, 1, n_seqs, seed=4)[0]
    max_pages = cdbgen.pages_for(prompt + n_decode)
    pages = n_seqs * max_pages
    kv = cdb.PagedKV(shape, n_seqs, max_pages, pages, pages, pages, fill="random")
    kv.core.normal_(0.0, 1.0)
    kv.pre.normal_(0.0, 1.0)
    kv.coda.normal_(0.0, 1.0)
    state = cdb.State(shape, n_seqs)
    ws = cdb.Workspace(dm.desc, 256)
    out_ids = torch.empty((n_seqs, n_decode), dtype=torch.int32, device="cuda")

    def run(n, nd, **mode):
        d = drv.Driver(max_batch=wl.max_batch, max_active=n, r_max=R, max_seqs=n_seqs, max_pages=max_pages,
                       core_pages=pages, pre_pages=pages, coda_pages=pages, has_prelude=True, has_coda=True,
                       kv_layout=drv.KV_SHARED, min_coda_batch=32, **mode)
        for q in range(n):
            d.add_sequence(prompt, depths[q][:nd])
        scratch = torch.empty(d.scratch_bytes(shape.vocab), dtype=torch.uint8, device="cuda")
        rws, half = runner_ws(dm, 256, mode.get("boundary_stream", False))
        secs = d.run(dm.model, kv.c, state.c, scratch, first, rws, tokens_out=out_ids)
        check_runner_ws(rws, half, "the huginn driver run")
        return secs, d.stats()

    run(4, 4)  # first use of the boundary kernels at this shape
    run(4, 4, boundary_stream=1)
    run(4, 4, graph_loop=True)
    e2e = {"workload": f"{n_seqs} requests, prompt {prompt} (KV synthesized), {n_decode} decode tokens each, depths "
                       f"lognormal median 12, sigma 0.5, clipped to [4, 32], max batch {wl.max_batch}, shared KV, "
                       f"minimum boundary batch 32",
           "mean_depth": round(mean_depth, 4), "flop_bound": round(cost.flop_bound(shape, mean_depth), 4)}
    for name, mode in (("cdb_refill", {}), ("cb_fixed_depth", {"fixed_depth": True}),
                       ("cdb_refill_boundary_stream_fill", {"boundary_stream": 1}),
                       ("cdb_refill_boundary_stream_hold", {"boundary_stream": 2}),
                       ("cdb_refill_graph", {"graph_loop": True})):
        secs, st = run(n_seqs, n_decode, **mode)
        e2e[name] = {"tokens_per_s": round(st["tokens"] / secs, 1), "seconds": round(secs, 4),
                     "loop_steps": st["loop_steps"], "loop_rows": st["loop_rows"], "idle_rows": st["idle_rows"],
                     "coda_calls": st["coda_calls"], "prelude_calls": st["prelude_calls"]}
        log(f"huginn e2e {name}: {st['tokens']} tokens in {secs:.3f}s, {st['loop_steps']} loop steps")
    e2e["speedup_refill_vs_cb"] = round(e2e["cdb_refill"]["tokens_per_s"] / e2e["cb_fixed_depth"]["tokens_per_s"], 4)
    e2e["boundary_stream_gain"] = {k: round(e2e["cdb_refill_boundary_stream_" + k]["tokens_per_s"] /
                                            e2e["cdb_refill"]["tokens_per_s"], 4) for k in ("fill", "hold")}
    e2e["graph_gain"] = round(e2e["cdb_refill_graph"]["tokens_per_s"] / e2e["cdb_refill"]["tokens_per_s"], 4)
    res["e2e"] = e2e
    del kv, state, ws, dm
    torch.cuda.empty_cache()
    return res


def long_context_step(shape, dm, steps=5, warmup=2):
    """The loop step at config 4's full batch: 256 rows at positions
    U[2048, 4223] (prompt U[2048, 4096] + decode 128), half of the tokens
    exiting at loop 1 and half at loop 4, drawn size-biased over the loop work.
    Each row maps its own pages (its loop plane over its context, plus the
    copy-on-exit destination page of every deeper plane): ≈ 160 GB of K/V, which
    one GPU holds although the whole depth-indexed cache of the config does not."""
    import numpy as np
    import torch

    import cdbgen
    import paper_2608_09444_amd as cdb
    wl = cdbgen.WORKLOADS[4]
    R = shape.r_max
    n_rows = wl.max_batch
    pos_lo, pos_hi = wl.prompt[0], wl.prompt[1] + wl.decode - 1
    rows_np = cdbgen.decode_snapshot(n_rows, wl.depth, R, pos_lo, pos_hi, stream=40)
    max_pages = cdbgen.pages_for(pos_hi + 1)
    pt, n_pages = own_pages(shape, rows_np, max_pages)
    kv = cdb.PagedKV(shape, n_rows, max_pages, 0, n_pages, 0, fill="random")
    g = torch.Generator(device="cuda")
    g.manual_seed(1234)
    kv.core.normal_(0.0, 1.0, generator=g)
    kv.page_table.copy_(torch.from_numpy(pt))
    state = cdb.State(shape, n_rows)
    state.h.normal_(0.0, 1.0, generator=g)
    rows = cdb.Rows(np.arange(n_rows, dtype=np.int32), np.arange(n_rows, dtype=np.int32), rows_np["pos"],
                    rows_np["c"], rows_np["depth"])
    so = cdb.StepOut(n_rows)
    ws = cdb.Workspace(dm.desc, n_rows)
    log(f"long context loop step: {n_rows} rows, {n_pages} core pages "
        f"({kv.core.numel() * 2 / 1e9:.0f} GB)")
    ms = time_loop_step(dm, kv, state, rows, so, ws, steps, warmup)
    if cdb.cdb_read_device_error(ws.buf) != 0:
        raise RuntimeError("device error in the long-context loop step")
    sb = step_bytes(shape, rows_np)
    attn_ms = time_attention(shape, kv, rows, n_rows, steps * shape.n_core)
    ab = attention_bytes(shape, rows_np["pos"])
    log(f"long context loop step: {ms:.3f} ms, {n_rows / (ms * 1e-3):.0f} rows/s; attention {attn_ms * 1e3:.1f} us")
    res = {"workload": f"ouro-shaped mixed-depth decode loop step: {n_rows} rows at positions U[{pos_lo},{pos_hi}] "
                       f"(prompt U[{wl.prompt[0]},{wl.prompt[1]}] + decode {wl.decode}), depths 50% 1 / 50% 4 per token",
           "rows": n_rows, "ms_per_step": round(ms, 4), "tokens_per_s": round(n_rows / (ms * 1e-3), 1),
           "mean_context": float(np.mean(rows_np["pos"] + 1)),
           "exits_per_step": int((rows_np["c"] + 1 == rows_np["depth"]).sum()),
           "step_roofline": {"bound": "hbm", "algorithmic_bytes": sb, "achieved": round(sb / (ms * 1e-3) / 1e9, 1),
                             "peak": HBM_PEAK_GBS, "unit": "GB/s",
                             "frac": round(sb / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                             "flops": step_flops(shape, rows_np)},
           "attention_roofline": {"bound": "hbm", "kernel": "k_attn<128> (paged decode attention, one layer)",
                                  "achieved": round(ab / (attn_ms * 1e-3) / 1e9, 1), "peak": HBM_PEAK_GBS,
                                  "unit": "GB/s", "frac": round(ab / (attn_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                                  "algorithmic_bytes": ab, "us_per_launch": round(attn_ms * 1e3, 2)}}
    del kv, state, rows, so, ws
    torch.cuda.empty_cache()
    return res


def long_context_leg(shape, dm, headroom_gib=16):
    """Config 4: 256 requests with prompts uniform in [2048, 4096] (KV
    synthesized as zeros), 128 decode tokens each, half of the tokens exiting at
    loop 1 and half at loop 4.  The depth-indexed cache of all 256 would take
    ≈ 630 GB, so under the full layout the driver admits requests while core
    pages last (KV-capacity admission) and the resident batch is what fits; the
    shared layout (one plane per position) holds all of them.  Each layout runs
    CDB refill against fixed-depth continuous batching on the same pool."""
    import numpy as np
    import torch

    import cdbgen
    import paper_2608_09444_amd as cdb
    from paper_2608_09444_amd import cost
    from paper_2608_09444_amd import driver as drv
    wl = cdbgen.WORKLOADS[4]
    R = shape.r_max
    n_seqs, n_decode = wl.n_seqs, wl.decode
    plen = cdbgen.lengths(wl.prompt, n_seqs, seed=cdbgen.PROMPT_SEED, stream=400)
    depths = [cdbgen.draw_depths(wl.depth, n_decode, R, stream=400 + q) for q in range(n_seqs)]
    mean_depth = float(np.mean(np.concatenate(depths)))
    first = cdbgen.prompt_ids(shape.vocab, 1, n_seqs, seed=5)[0]
    max_pages = cdbgen.pages_for(int(plen.max()) + n_decode)
    page_bytes = shape.n_core * 2 * shape.n_heads * cdbgen.PAGE_TOKENS * shape.head_dim * 2
    torch.cuda.empty_cache()
    free, _ = torch.cuda.mem_get_info()
    budget_pages = int((free - (headroom_gib << 30)) // page_bytes)
    state = cdb.State(shape, n_seqs)
    ws = cdb.Workspace(dm.desc, 256)
    out_ids = torch.empty((n_seqs, n_decode), dtype=torch.int32, device="cuda")
    res = {"workload": f"{n_seqs} requests, prompts uniform in [2048, 4096] (KV synthesized), {n_decode} decode tokens "
                       f"each, depths 50% 1 / 50% 4 per token, max batch {wl.max_batch}",
           "mean_depth": round(mean_depth, 4), "flop_bound": round(cost.flop_bound(shape, mean_depth), 4),
           "prompt_tokens": int(plen.sum())}
    res["loop_step"] = long_context_step(shape, dm)
    for lname, layout, planes in (("full", drv.KV_FULL, R), ("shared", drv.KV_SHARED, 1)):
        need = int(sum(cdbgen.pages_for(int(p) + n_decode) for p in plen)) * planes
        core_pages = min(need, budget_pages)
        kv = cdb.PagedKV(shape, n_seqs, max_pages, 0, core_pages, 0)
        torch.cuda.synchronize()
        log(f"long context, {lname} layout: {core_pages} core pages ({core_pages * page_bytes / 1e9:.0f} GB of "
            f"{need * page_bytes / 1e9:.0f} GB for all requests)")
        entry = {"core_pages": core_pages, "pool_gb": round(core_pages * page_bytes / 1e9, 1),
                 "all_requests_gb": round(need * page_bytes / 1e9, 1)}
        for name, mode in (("cdb_refill", {}), ("cb_fixed_depth", {"fixed_depth": True})):
            d = drv.Driver(max_batch=wl.max_batch, max_active=n_seqs, r_max=R, max_seqs=n_seqs, max_pages=max_pages,
                           core_pages=core_pages, kv_layout=layout, **mode)
            for q in range(n_seqs):
                d.add_sequence(int(plen[q]), depths[q])
            scratch = torch.empty(d.scratch_bytes(shape.vocab), dtype=torch.uint8, device="cuda")
            secs = d.run(dm.model, kv.c, state.c, scratch, first, ws.buf, tokens_out=out_ids)
            if cdb.cdb_read_device_error(ws.buf) != 0:
                raise RuntimeError("device error in the long-context driver run")
            st = d.stats()
            entry[name] = {"tokens_per_s": round(st["tokens"] / secs, 1), "seconds": round(secs, 3),
                           "loop_steps": st["loop_steps"], "loop_rows": st["loop_rows"],
                           "mean_rows_per_loop_step": round(st["loop_rows"] / max(st["loop_steps"], 1), 1),
                           "idle_rows": st["idle_rows"], "coda_calls": st["coda_calls"]}
            log(f"long context, {lname} layout, {name}: {st['tokens']} tokens in {secs:.2f}s, {st['loop_steps']} loop "
                f"steps, {st['loop_rows'] / max(st['loop_steps'], 1):.1f} rows per step")
        entry["speedup_refill_vs_cb"] = round(entry["cdb_refill"]["tokens_per_s"] /
                                              entry["cb_fixed_depth"]["tokens_per_s"], 4)
        res[lname] = entry
        del kv
        torch.cuda.empty_cache()
    del state, ws, out_ids
    torch.cuda.empty_cache()
    return res


def graph_leg(dm, kv, state, rows_np, steps, counts=(64, 40, 17)):
    """cdb_loop_step captured once in a HIP graph at the batch's row capacity,
    with the row count in device memory (cdb_rows.d_n_rows), and replayed at
    several counts: each count's replay is checked bit for bit against an eager
    call of exactly that many rows from the same saved state and cache (eager
    work and synchronisation between the replays); the full-count replay is
    timed."""
    import numpy as np
    import torch

    import paper_2608_09444_amd as cdb
    st = torch.cuda.current_stream()
    cap = len(rows_np["pos"])
    h0 = state.h.clone()
    ar = np.arange(cap, dtype=np.int32)
    d_n = torch.full((1,), cap, dtype=torch.int32, device="cuda")
    rows_g = cdb.Rows(ar, ar, rows_np["pos"], rows_np["c"], rows_np["depth"], d_n_rows=d_n)
    out_g = cdb.StepOut(cap)
    ws_g = cdb.Workspace(dm.desc, cap)
    ws_e = cdb.Workspace(dm.desc, cap)
    cdb.cdb_loop_step(dm.model, kv.c, state.c, rows_g.c, out_g.c, ws_g.buf)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(st)
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            cdb.cdb_loop_step(dm.model, kv.c, state.c, rows_g.c, out_g.c, ws_g.buf, stream=side)
    st.wait_stream(side)
    torch.cuda.synchronize()
    checked = {}
    for n in counts:
        # K/V written by a step at its own positions is rewritten identically by
        # the next call from the same state, so only the state is restored
        state.h.copy_(h0)
        sl = slice(0, n)
        rows_e = cdb.Rows(ar[sl], ar[sl], rows_np["pos"][sl], rows_np["c"][sl], rows_np["depth"][sl])
        out_e = cdb.StepOut(n)
        cdb.cdb_loop_step(dm.model, kv.c, state.c, rows_e.c, out_e.c, ws_e.buf)
        torch.cuda.synchronize()
        ref = (state.h.clone(), out_e.score[:n].clone(), out_e.mask[:n].clone(), out_e.counts.clone())
        state.h.copy_(h0)
        d_n.fill_(n)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = (state.h.clone(), out_g.score[:n].clone(), out_g.mask[:n].clone(), out_g.counts.clone())
        checked[str(n)] = all(torch.equal(a, b) for a, b in zip(ref, got))
    d_n.fill_(cap)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(st)
    for _ in range(steps):
        g.replay()
    e1.record(st)
    e1.synchronize()
    if cdb.cdb_read_device_error(ws_g.buf) != 0 or cdb.cdb_read_device_error(ws_e.buf) != 0:
        raise RuntimeError("device error in the graph replays")
    state.h.copy_(h0)
    ms = e0.elapsed_time(e1) / steps
    log(f"graph replay at {cap} rows: {ms:.3f} ms/step; replays at counts {list(checked)} identical to eager "
        f"calls: {checked}")
    return {"ms_per_step": round(ms, 4), "capacity": cap, "replays_match_eager": checked}


def idle_ablation(shape_name, n_decode=48, pause_s=1.0):
    """Whole decodes under the scheduler variants of Section 4.3, one after the
    other with `pause_s` of device silence between them, for a kernel trace to
    split into one segment per variant (GPU idle = the share of each segment
    with no kernel running): the synchronous scheduler (the host waits for every
    loop step), the asynchronous one, asynchronous with device-decided exits and
    the lookahead gate, asynchronous with the boundary stages on a second
    stream, and asynchronous with loop steps replayed from a graph.
    Ouro-shaped: 64 requests, prompt 512 (KV synthesized), full
    depth-indexed KV, max batch 64; Huginn-shaped (no gate variant: its
    convergence criterion has no threshold these random-init states straddle
    usefully): 128 requests, prompt 256, shared KV, max batch 128, minimum
    boundary batch 32."""
    import numpy as np
    import torch

    import cdbgen
    import paper_2608_09444_amd as cdb
    from paper_2608_09444_amd import driver as drv
    if shape_name == "ouro":
        shape, n_seqs, prompt, batch, layout, depth_spec = cdbgen.OURO, 64, 512, 64, drv.KV_FULL, cdbgen.OURO_DEPTHS
        extra = {}
    else:
        wl = cdbgen.WORKLOADS[3]
        shape, n_seqs, prompt, batch, layout, depth_spec = cdbgen.HUGINN, wl.n_seqs, wl.prompt, wl.max_batch, \
            drv.KV_SHARED, wl.depth
        extra = {"min_coda_batch": 32}
    R = shape.r_max
    dm = cdb.DeviceModel(shape, cdbgen.model_weights(shape))
    max_pages = cdbgen.pages_for(prompt + n_decode)
    per = R if layout == drv.KV_FULL else 1
    pages = n_seqs * max_pages
    kv = cdb.PagedKV(shape, n_seqs, max_pages, pages if shape.n_prelude else 0, pages * per,
                     pages if shape.n_coda else 0, fill="random")
    for pool in (kv.pre, kv.core, kv.coda):
        pool.normal_(0.0, 1.0)
    state = cdb.State(shape, n_seqs)
    depths = [cdbgen.draw_depths(depth_spec, n_decode, R, seed=3, stream=q) for q in range(n_seqs)]
    first = cdbgen.prompt_ids(shape.vocab, 1, n_seqs, seed=4)[0]
    order = [("synchronous", {"sync_steps": True}), ("asynchronous", {})]
    if shape.exit_kind == 0:  # the learned-gate form: a threshold of 0.5 on the random-init gate
        order.append(("asynchronous_lookahead_gate", {"gated": True, "lookahead": True, "threshold": 0.5}))
    order.append(("asynchronous_boundary_stream_fill", {"boundary_stream": 1}))
    order.append(("asynchronous_boundary_stream_hold", {"boundary_stream": 2}))
    order.append(("asynchronous_graph_replay", {"graph_loop": True}))
    res = {"order": [n for n, _ in order]}
    for k, (name, mode) in enumerate([("warmup", {})] + order):
        d = drv.Driver(max_batch=batch, max_active=n_seqs, r_max=R, max_seqs=n_seqs, max_pages=max_pages,
                       core_pages=pages * per, pre_pages=pages, coda_pages=pages, has_prelude=shape.n_prelude > 0,
                       has_coda=shape.n_coda > 0, kv_layout=layout, **extra, **mode)
        nd = 4 if name == "warmup" else n_decode
        for q in range(n_seqs):
            d.add_sequence(prompt, None if mode.get("gated") else depths[q][:nd], n_decode=nd)
        scratch = torch.empty(d.scratch_bytes(shape.vocab), dtype=torch.uint8, device="cuda")
        ws, half = runner_ws(dm, 256, mode.get("boundary_stream", False))
        torch.cuda.synchronize()
        time.sleep(pause_s)
        secs = d.run(dm.model, kv.c, state.c, scratch, first, ws)
        torch.cuda.synchronize()
        check_runner_ws(ws, half, f"the {name} run")
        st = d.stats()
        if name != "warmup":
            res[name] = {"seconds": round(secs, 4), "tokens_per_s": round(st["tokens"] / secs, 1),
                         "loop_steps": st["loop_steps"], "ms_per_loop_step": round(secs * 1e3 / st["loop_steps"], 4),
                         "host_wait_us_per_loop_step": round(st["host_wait_us"] / st["loop_steps"], 2)}
            log(f"idle ablation {shape_name} {name}: {res[name]}")
    time.sleep(pause_s)
    del kv, state, dm
    torch.cuda.empty_cache()
    return res


def idle_segments(csv_path, silence_ns=300_000_000):
    """Reads a rocprofv3 kernel trace (CSV) of an `--idle-ablation` run and
    splits it into one segment per decode at gaps longer than `silence_ns`.
    Per segment: span (first kernel start to last kernel end), busy (the union
    of the kernel intervals), idle = 1 - busy / span, and the largest gaps
    between kernels.  Host-side only; no device is touched."""
    import csv
    with open(csv_path, newline="") as f:
        iv = sorted((int(r["Start_Timestamp"]), int(r["End_Timestamp"])) for r in csv.DictReader(f))
    if not iv:
        raise SystemExit(f"{csv_path}: no kernels in the trace")
    segs, cur, cur_end = [], [iv[0]], iv[0][1]
    for a in iv[1:]:
        if a[0] - cur_end > silence_ns:
            segs.append(cur)
            cur, cur_end = [a], a[1]
        else:
            cur.append(a)
            cur_end = max(cur_end, a[1])
    segs.append(cur)
    out = []
    for seg in segs:
        t0, t1 = seg[0][0], max(e for _, e in seg)
        busy, end, gaps = 0, t0, []
        for s0, e0 in seg:
            if s0 > end and end > t0:
                gaps.append(s0 - end)
            if e0 > end:
                busy += e0 - max(s0, end)
                end = e0
        span = max(t1 - t0, 1)
        out.append({"kernels": len(seg), "span_ms": round(span / 1e6, 2), "busy_ms": round(busy / 1e6, 2),
                    "idle_pct": round((1 - busy / span) * 100, 2),
                    "largest_gaps_us": [round(g / 1e3, 1) for g in sorted(gaps)[-3:]]})
    return out


def copy_peak(gib=4, reps=5):
    """A plain device-to-device copy of `gib` GiB: the HBM rate a simple stream
    reaches on this part (read + write bytes per second)."""
    import torch
    n = gib << 28
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    e1.synchronize()
    gbs = 2.0 * n * 4 * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    log(f"copy of {gib} GiB: {gbs:.0f} GB/s")
    return round(gbs, 1)


def serving_leg(shape, dm, n_req, rate=20.0, max_batch=64, chunk=512, core_pages=24576, fixed_depth=False,
                boundary_stream=0, graph_loop=False):
    """A serving trace of the ouro-shaped model: Poisson arrivals at `rate`
    requests/s, prompt lengths lognormal (median 300, sigma 1, [16, 4096]),
    output lengths lognormal (median 400, sigma 1, [16, 2048]), categorical
    depths; the driver prefills every prompt through cdb_prefill in chunks of
    512 between loop steps and admits requests at every step while the KV pool
    (core_pages pages of the depth-indexed cache) has room.  Tokens/s over the
    whole run and the normalised latency ((finish - arrival) / output tokens)."""
    import numpy as np
    import torch

    import cdbgen
    import paper_2608_09444_amd as cdb
    from paper_2608_09444_amd import driver as drv
    wl = cdbgen.WORKLOADS[5]
    R = shape.r_max
    plen = cdbgen.lengths(wl.prompt, n_req, seed=cdbgen.PROMPT_SEED, stream=100)
    olen = cdbgen.lengths(wl.decode, n_req, seed=cdbgen.PROMPT_SEED, stream=101)
    arrivals = cdbgen.poisson_arrivals(n_req, rate)
    max_pages = cdbgen.pages_for(int(plen.max() + olen.max()))
    d = drv.Driver(max_batch=max_batch, max_active=max_batch, r_max=R, max_seqs=n_req, max_pages=max_pages,
                   core_pages=core_pages, prefill_chunk=chunk, fixed_depth=fixed_depth,
                   boundary_stream=boundary_stream, graph_loop=graph_loop)
    for q in range(n_req):
        d.add_request(cdbgen.prompt_ids(shape.vocab, 1, int(plen[q]), stream=q)[0],
                      cdbgen.draw_depths(wl.depth, int(olen[q]), R, stream=1000 + q), arrival=float(arrivals[q]))
    kv = cdb.PagedKV(shape, n_req, max_pages, 0, core_pages, 0)
    state = cdb.State(shape, n_req)
    ws, half = runner_ws(dm, chunk, boundary_stream)
    scratch = torch.empty(d.scratch_bytes(shape.vocab), dtype=torch.uint8, device="cuda")
    log(f"serving{' (fixed depth)' if fixed_depth else ''}{' (boundary stream)' if boundary_stream else ''}"
        f"{' (graph replay)' if graph_loop else ''}: "
        f"{n_req} requests at {rate}/s, {int(plen.sum())} prompt + {int(olen.sum())} output tokens")
    secs = d.run(dm.model, kv.c, state.c, scratch, None, ws)
    check_runner_ws(ws, half, "the serving run")
    st = d.stats()
    lat = d.latencies(n_req)
    lat = lat[lat >= 0]
    res = {"workload": f"{n_req} requests, Poisson {rate}/s, prompt lognormal(300, 1) in [16, 4096], output "
                       f"lognormal(400, 1) in [16, 2048], depths categorical {{1:.3,2:.3,3:.2,4:.2}}, max batch "
                       f"{max_batch}, prefill chunks of {chunk}, depth-indexed KV of {core_pages} core pages",
           "seconds": round(secs, 3), "tokens_per_s": round(st["tokens"] / secs, 1),
           "prompt_tokens_per_s": round(st["prefill_tokens"] / secs, 1),
           "normalized_latency_s": {"p50": round(float(np.percentile(lat, 50)), 5),
                                    "p99": round(float(np.percentile(lat, 99)), 5)},
           "finished": int(len(lat)), "loop_steps": st["loop_steps"], "idle_rows": st["idle_rows"],
           "prefill_calls": st["prefill_calls"], "coda_calls": st["coda_calls"],
           "host_wait_us_per_loop_step": round(st["host_wait_us"] / max(1, st["loop_steps"]), 2),
           "page_table_uploads": st["pt_uploads"], "page_table_upload_bytes": st["pt_upload_bytes"]}
    log(f"serving: {st['tokens']} tokens in {secs:.2f}s, p50/p99 normalized latency "
        f"{res['normalized_latency_s']['p50'] * 1e3:.1f}/{res['normalized_latency_s']['p99'] * 1e3:.1f} ms")
    del kv, state, ws, scratch
    torch.cuda.empty_cache()
    return res


def prefill_leg(shape, dm, kv, chunk=512, reps=5):
    """Chunked prefill at full width: one chunk of `chunk` prompt tokens of one
    sequence (positions 0..chunk-1) through cdb_prefill, timed with events on
    the stream it runs on.  FLOPs: every projection (2 per weight and row) of
    r_max core loops plus the LM head, and causal attention (4 * d per
    query-key pair per core layer and loop)."""
    import numpy as np
    import torch

    import cdbgen
    import paper_2608_09444_amd as cdb
    R = shape.r_max
    max_pages = kv.c.max_pages
    pages = cdbgen.pages_for(chunk)
    pt = np.full((kv.c.max_seqs, R + 2, max_pages), -1, np.int32)
    pt[0, 1:R + 1, :pages] = np.arange(pages * R, dtype=np.int32).reshape(R, pages)
    kv.page_table.copy_(torch.from_numpy(pt))
    ws = cdb.Workspace(dm.desc, chunk)
    tok = torch.as_tensor(cdbgen.prompt_ids(shape.vocab, 1, chunk, seed=9)[0], dtype=torch.int32, device="cuda")
    logits = torch.empty((chunk, shape.vocab), dtype=torch.float32, device="cuda")
    ids = torch.empty(chunk, dtype=torch.int32, device="cuda")
    st = torch.cuda.current_stream()
    cdb.cdb_prefill(dm.model, kv.c, 0, 0, tok, logits, ids, ws.buf)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(st)
    for _ in range(reps):
        cdb.cdb_prefill(dm.model, kv.c, 0, 0, tok, logits, ids, ws.buf)
    e1.record(st)
    e1.synchronize()
    if cdb.cdb_read_device_error(ws.buf) != 0:
        raise RuntimeError("device error in prefill")
    ms = e0.elapsed_time(e1) / reps
    pc = cdbgen.param_counts(shape)
    proj = 2.0 * chunk * (R * pc["core"] + pc["boundary_layers"] + shape.d * shape.vocab)
    attn = 4.0 * shape.d * shape.n_core * R * chunk * (chunk + 1) / 2
    tflops = (proj + attn) / (ms * 1e-3) / 1e12
    log(f"prefill: {chunk} tokens in {ms:.2f} ms, {tflops:.0f} TFLOP/s")
    return {"workload": f"one {chunk}-token prompt chunk (positions 0..{chunk - 1}), all r_max loops, coda, LM head",
            "tokens_per_s": round(chunk / (ms * 1e-3), 1), "ms_per_chunk": round(ms, 3),
            "flops": proj + attn, "achieved_tflops": round(tflops, 1), "peak_tflops": BF16_PEAK_TFLOPS,
            "mfma_frac": round(tflops / BF16_PEAK_TFLOPS, 4)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--cpu-sample", type=int, default=16, help="rows in the CPU-oracle sample (0 = skip)")
    ap.add_argument("--no-e2e", action="store_true", help="skip the whole-decode driver runs")
    ap.add_argument("--no-prefill", action="store_true", help="skip the chunked-prefill timing")
    ap.add_argument("--no-sweep", action="store_true", help="skip the loop-step batch-size sweep and the latency-model grid")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the graph-replay leg (its replays at fewer live rows would mix into per-kernel profiles)")
    ap.add_argument("--serving-requests", type=int, default=200,
                    help="requests in the serving-trace run (0 = skip; 2000 is the full trace)")
    ap.add_argument("--huginn-decode", type=int, default=512,
                    help="decode tokens per request in the Huginn-shaped whole-decode runs (0 = skip the Huginn leg; "
                         "512 is the full workload)")
    ap.add_argument("--no-long-context", action="store_true",
                    help="skip config 4's long-context loop step and decodes (about 250 GB of KV pools, ≈ 2 minutes)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="run one plain device copy of this many MiB first (a known-size reference for HBM counters)")
    ap.add_argument("--idle-ablation", action="store_true",
                    help="only the scheduler-variant decodes for a kernel trace (GPU idle per variant)")
    ap.add_argument("--idle-trace", metavar="CSV",
                    help="only analyse a kernel trace of an --idle-ablation run: GPU idle per decode segment "
                         "(host-side, no device)")
    args = ap.parse_args()
    if args.idle_trace:
        for k, seg in enumerate(idle_segments(args.idle_trace)):
            print(json.dumps({"segment": k, **seg}), flush=True)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU only: the loop step shards by sequence with no exchange between GPUs, "
              "and this benchmark runs and reports the single-GPU path (use --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import cdbgen
    import paper_2608_09444_amd as cdb
    if args.idle_ablation:
        print(json.dumps({"idle_ablation": {"ouro": idle_ablation("ouro"), "huginn": idle_ablation("huginn")}}),
              flush=True)
        return
    shape = cdbgen.OURO
    n_rows, pos_lo, pos_hi = 64, 512, 767
    log("setup")
    t0 = time.time()
    w = cdbgen.model_weights(shape)
    log(f"weights drawn in {time.time() - t0:.1f}s")
    dm, kv, state, rows, rows_np, out, ws = setup(shape, w, n_rows, pos_lo, pos_hi)
    st = torch.cuda.current_stream()
    if args.copy_calibration > 0:
        src = torch.ones(args.copy_calibration << 18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    def step():
        cdb.cdb_loop_step(dm.model, kv.c, state.c, rows.c, out.c, ws.buf)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    code = cdb.cdb_read_device_error(ws.buf)
    if code != 0:
        raise RuntimeError(f"device error {code} during warmup")
    log(f"timing {args.steps} steps")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(st)
    for _ in range(args.steps):
        step()
    e1.record(st)
    e1.synchronize()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    value = n_rows / (ms * 1e-3)
    sb = step_bytes(shape, rows_np)
    log(f"{ms:.3f} ms/step, {value:.0f} rows/s, step bytes {sb / 1e9:.2f} GB -> {sb / (ms * 1e-3) / 1e9:.0f} GB/s")

    graph = None
    if not args.no_graph:
        try:
            graph = graph_leg(dm, kv, state, rows_np, args.steps)
        except RuntimeError as e:  # a capture the runtime refuses is reported, not fatal
            graph = {"error": str(e)}
    copy_gbs = copy_peak()

    attn_ms = time_attention(shape, kv, rows, n_rows, args.steps * shape.n_core)
    ab = attention_bytes(shape, rows_np["pos"])
    attn_gbs = ab / (attn_ms * 1e-3) / 1e9
    log(f"attention {attn_ms * 1e3:.1f} us/launch, {ab / 1e6:.1f} MB -> {attn_gbs:.0f} GB/s")

    sweep = lat = None
    if not args.no_sweep:
        sweep = batch_sweep(shape, dm)
        lat = latency_model(shape, dm)

    e2e = None
    if not args.no_e2e:
        e2e = e2e_decode(shape, dm, kv, n_rows, pos_lo, pos_hi + 1 - pos_lo)
        e2e["batch_sweep"] = batch_e2e(shape, dm)

    prefill = None
    if not args.no_prefill:
        prefill = prefill_leg(shape, dm, kv)

    serving = None
    if args.serving_requests > 0:
        serving = {"cdb_refill": serving_leg(shape, dm, args.serving_requests),
                   "cb_fixed_depth": serving_leg(shape, dm, args.serving_requests, fixed_depth=True),
                   "cdb_refill_boundary_stream_fill": serving_leg(shape, dm, args.serving_requests,
                                                                  boundary_stream=1)}
        a, b = serving["cdb_refill"], serving["cb_fixed_depth"]
        serving["throughput_ratio"] = round(a["tokens_per_s"] / b["tokens_per_s"], 4)
        serving["p50_latency_reduction"] = round(1 - a["normalized_latency_s"]["p50"] /
                                                 b["normalized_latency_s"]["p50"], 4)
        serving["p99_latency_reduction"] = round(1 - a["normalized_latency_s"]["p99"] /
                                                 b["normalized_latency_s"]["p99"], 4)

    huginn = None
    long_ctx = None
    if args.huginn_decode > 0 or not args.no_long_context:
        del kv, state, rows, out, ws
        torch.cuda.empty_cache()
    if not args.no_long_context:
        try:
            long_ctx = long_context_leg(shape, dm)
        except (RuntimeError, torch.OutOfMemoryError) as e:  # reported in the record, not fatal to the line
            log(f"long context leg failed: {e}")
            long_ctx = {"error": str(e)}
            torch.cuda.empty_cache()
    if args.huginn_decode > 0:
        huginn = huginn_leg(args.huginn_decode)

    cpu = None
    if args.cpu_sample > 0:
        info = host_info()
        threads = host_threads()
        log(f"cpu baseline on {args.cpu_sample} rows, {threads} threads")
        cpu = cpu_baseline(shape, w, rows_np, args.cpu_sample, threads)
        log("cpu baseline on 1 row, 1 thread")
        one = cpu_baseline(shape, w, rows_np, 1, 1, min_s=8.0)
        cpu["single_core"] = {"value": one["value"], "cores": 1, "sample": one["sample"]}
        cpu.update(info)

    res = {
        "metric": "mixed-depth loop-step tokens/s (Ouro-1.4B-shaped, bs=64); % HBM/MFMA roofline",
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"mixed-depth decode loop step of an ouro-1.4b-shaped looped LM (d {shape.d}, "
                               f"{shape.n_heads} heads x {shape.head_dim}, SwiGLU {shape.d_ff}, {shape.n_core} core "
                               f"layers looped up to {shape.r_max} times): {n_rows} rows at positions U[512,767] "
                               f"(prompt 512 + decode 256), depths categorical {{1:.3,2:.3,3:.2,4:.2}}",
                   "rows": n_rows, "mean_context": float(np.mean(rows_np["pos"] + 1)),
                   "exits_per_step": int((rows_np["c"] + 1 == rows_np["depth"]).sum())},
        "roofline": {"bound": "hbm", "kernel": "k_attn<128> (paged decode attention, one layer)",
                     "achieved": round(attn_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(attn_gbs / HBM_PEAK_GBS, 4), "traffic": measured_traffic(),
                     "algorithmic_bytes": ab},
        "graph_replay": graph,
        "hbm_copy_gbs": copy_gbs,
        "step_roofline": {"bound": "hbm", "algorithmic_bytes": sb, "achieved": round(sb / (ms * 1e-3) / 1e9, 1),
                          "peak": HBM_PEAK_GBS, "unit": "GB/s",
                          "frac": round(sb / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                          "flops": step_flops(shape, rows_np)},
        "cpu_baseline": cpu,
        "batch_sweep": sweep, "latency_model": lat,
        "e2e": e2e,
        "prefill": prefill,
        "serving": serving,
        "huginn": huginn,
        "long_context": long_ctx,
        "reduced_legs": reduced_legs(args),
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
