"""GPU: the host driver running whole decodes through the HIP stage calls, and
the shared core KV layouts call by call against the oracle.

* Every row of a stage call is computed independently of the others, so the
  same requests decoded under different schedules (refill, no-refill, a
  minimum coda batch, other batch sizes) must give bit-identical tokens.
* The greedy tokens must follow the oracle's wherever the history agrees and
  the oracle's top-2 logit gap is clear of the tolerance.
"""
import dataclasses
import sys

import numpy as np
import pytest
import torch

import cdbgen
import oracle
import paper_2608_09444_amd as cdb
from paper_2608_09444_amd import driver as drv

pytestmark = pytest.mark.gpu

# logits agree within 2e-2 per element, so a top-2 gap above 4e-2 fixes the argmax
GAP = 4e-2


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _requests(shape, seed=40):
    plens = [17, 8, 33, 5, 20, 12]
    ndec = [10, 14, 6, 12, 9, 11]
    prompts = [cdbgen.prompt_ids(shape.vocab, 1, p, seed=seed, stream=q)[0] for q, p in enumerate(plens)]
    depths = [cdbgen.draw_depths(("uniform", 1, shape.r_max), n, shape.r_max, seed=seed + 1, stream=q)
              for q, n in enumerate(ndec)]
    return prompts, ndec, depths


def _driver_ws(gm, rows, cfg):
    """The runner's workspace: one stage workspace, or two (halves) when the
    boundary stages have their own stream; error words start at zero."""
    n = cdb.cdb_workspace_bytes(gm.desc, rows)
    n = (n + 255) & ~255
    return torch.zeros(2 * n if cfg.get("boundary_stream") else n, dtype=torch.uint8, device="cuda"), n


def _ws_errors(ws, half):
    return [cdb.cdb_read_device_error(ws), cdb.cdb_read_device_error(ws[half:])] if ws.numel() > half else \
        [cdb.cdb_read_device_error(ws)]


def _check_table_uploads(st, n_seqs, shape, max_pages):
    """After the first whole-table upload, only changed sequences' blocks travel."""
    full = n_seqs * (shape.r_max + 2) * max_pages * 4
    assert st["pt_uploads"] >= 1
    assert st["pt_upload_bytes"] == full + (st["pt_uploads"] - 1) * full // n_seqs


def _decode_on_gpu(shape, gm, prompts, ndec, depths, kv_layout=drv.KV_FULL, **cfg):
    """depths[q] is None in gated mode."""
    """Prefill every prompt through the stage calls (one block per sequence),
    then let the driver decode all requests.  Returns (first tokens, decoded
    ids [seq][k], driver stats)."""
    R = shape.r_max
    n = len(prompts)
    T = [len(p) + k for p, k in zip(prompts, ndec)]
    max_pages = max(cdbgen.pages_for(t) for t in T)
    tot = sum(cdbgen.pages_for(t) for t in T)
    per = {drv.KV_FULL: R, drv.KV_SHARED: 1, drv.KV_FIRST_THEN_SHARED: min(2, R)}[kv_layout]
    d = drv.Driver(max_seqs=n, max_pages=max_pages, core_pages=tot * per, pre_pages=tot, coda_pages=tot,
                   has_prelude=shape.n_prelude > 0, has_coda=shape.n_coda > 0, r_max=R, kv_layout=kv_layout,
                   **cfg)
    for q in range(n):
        d.add_sequence(len(prompts[q]), depths[q], n_decode=ndec[q])
    assert cfg.get("max_active", 0) >= n
    first_tick = d.next()  # admits every request; the plan is kept until completed
    assert first_tick.n_rows == n
    kv = cdb.PagedKV(shape, n, max_pages, tot, tot * per, tot)
    kv.page_table.copy_(torch.from_numpy(d.page_table()))
    ws = cdb.Workspace(gm.desc, 256)
    # prefill: prompt rows use their own state slots
    pstate = cdb.State(shape, max(len(p) for p in prompts))
    first = np.zeros(n, np.int32)
    for q, p in enumerate(prompts):
        P = len(p)
        pos = np.arange(P, dtype=np.int32)
        rows = cdb.Rows(pos, np.full(P, q, np.int32), pos, None, None)
        cdb.cdb_boundary_prelude(gm.model, kv.c, pstate.c, rows.c, torch.as_tensor(p, dtype=torch.int32,
                                                                                   device="cuda"), ws.buf)
        out = cdb.StepOut(P)
        for c in range(R):
            lr = cdb.Rows(pos, np.full(P, q, np.int32), pos, np.full(P, c, np.int32), np.full(P, R, np.int32))
            cdb.cdb_loop_step(gm.model, kv.c, pstate.c, lr.c, out.c, ws.buf)
        logits = torch.zeros((P, shape.vocab), dtype=torch.float32, device="cuda")
        ids = torch.zeros(P, dtype=torch.int32, device="cuda")
        cdb.cdb_boundary_coda(gm.model, kv.c, pstate.c, rows.c, logits, ids, ws.buf)
        first[q] = int(ids[-1].item())
    state = cdb.State(shape, n)
    scratch = torch.empty(d.scratch_bytes(shape.vocab), dtype=torch.uint8, device="cuda")
    out_ids = torch.full((n, max(ndec)), -1, dtype=torch.int32, device="cuda")
    assert cdb.cdb_read_device_error(ws.buf) == 0
    rws, half = _driver_ws(gm, 256, cfg)
    secs = d.run(gm.model, kv.c, state.c, scratch, first, rws, tokens_out=out_ids)
    torch.cuda.synchronize()
    assert _ws_errors(rws, half) == [0] * (2 if cfg.get("boundary_stream") else 1)
    st = d.stats()
    _check_table_uploads(st, n, shape, max_pages)
    return first, out_ids.cpu().numpy(), st, secs


def _check_against_oracle(shape, w, prompts, ndec, depths, first, ids, kv_layout):
    m = oracle.Model(shape, w, bf16_storage=True, kv_layout=kv_layout)
    checked = 0
    for q, p in enumerate(prompts):
        P, N = len(p), ndec[q]
        dep = np.concatenate([np.full(P, shape.r_max, np.int32), depths[q]])
        # teacher-force the GPU's own tokens, so a legitimate near-tie flip does
        # not stop the comparison of the positions after it
        gpu_tokens = np.concatenate([p, [first[q]], ids[q, :N - 1]]).astype(np.int32)
        ref = m.ref_sequence(gpu_tokens, dep, n_given=P + N, n_prefill=P)
        gpu_next = np.concatenate([[first[q]], ids[q, :N]])  # id after positions P-1 .. P+N-1
        for k, t in enumerate(range(P - 1, P + N)):
            lg = ref["logits"][t]
            top2 = np.sort(lg)[-2:]
            if top2[1] - top2[0] > GAP:
                assert gpu_next[k] == int(np.argmax(lg)), f"seq {q} position {t}"
                checked += 1
            else:
                assert lg[gpu_next[k]] >= top2[1] - GAP
    return checked


@pytest.mark.parametrize("kv_layout", [drv.KV_FULL, drv.KV_SHARED, drv.KV_FIRST_THEN_SHARED],
                         ids=["full", "shared", "first-then-shared"])
def test_driver_decode_is_schedule_invariant_and_follows_oracle(kv_layout):
    s = cdbgen.TINY
    _say(f"[gpu] driver decode {s.name} layout {kv_layout}")
    w = cdbgen.model_weights(s)
    gm = cdb.DeviceModel(s, w)
    prompts, ndec, depths = _requests(s)
    n = len(prompts)
    runs = {}
    for name, cfg in (("refill", dict(max_batch=4, max_active=n)),
                      ("no-refill", dict(max_batch=3, max_active=n, refill=False)),
                      ("refill-coda3", dict(max_batch=6, max_active=n, min_coda_batch=3)),
                      ("refill-boundary-stream-1", dict(max_batch=4, max_active=n, boundary_stream=1)),
                      ("refill-boundary-stream-2", dict(max_batch=4, max_active=n, boundary_stream=2)),
                      ("refill-graph", dict(max_batch=4, max_active=n, graph_loop=True)),
                      ("no-refill-graph-boundary-stream", dict(max_batch=3, max_active=n, refill=False,
                                                               boundary_stream=1, graph_loop=True))):
        first, ids, st, secs = _decode_on_gpu(s, gm, prompts, ndec, depths, kv_layout, **cfg)
        _say(f"[gpu]   {name}: {st} in {secs * 1e3:.1f} ms")
        assert st["tokens"] == sum(ndec)
        assert st["graph_launches"] == (st["loop_steps"] if cfg.get("graph_loop") else 0)
        assert st["loop_rows"] == sum(int(x.sum()) for x in depths)
        runs[name] = (first, ids)
    base = runs["refill"]
    for name, (first, ids) in runs.items():
        assert np.array_equal(first, base[0]) and np.array_equal(ids, base[1]), name
    checked = _check_against_oracle(s, w, prompts, ndec, depths, base[0], base[1], kv_layout)
    _say(f"[gpu]   {checked} greedy ids checked against the oracle")
    assert checked >= 0.3 * (sum(ndec) + n)  # not vacuous: about half the positions have a clear gap


# the Huginn-shaped features at small widths: the input-injection adapter
# (W_a [h; e] before every core pass) and the convergence exit score
INJ = cdbgen.ModelShape(name="inj-1-2-1", d=192, n_heads=3, head_dim=64, d_ff=256, vocab=160, n_prelude=1,
                        n_core=2, n_coda=1, r_max=3, injection=1, exit_kind=1)


@pytest.mark.parametrize("kv_layout", [drv.KV_FULL, drv.KV_SHARED], ids=["full", "shared"])
def test_driver_decode_with_injection_is_schedule_invariant_and_follows_oracle(kv_layout):
    s = INJ
    _say(f"[gpu] driver decode {s.name} layout {kv_layout}")
    w = cdbgen.model_weights(s)
    gm = cdb.DeviceModel(s, w)
    prompts, ndec, depths = _requests(s, seed=44)
    n = len(prompts)
    runs = {}
    for name, cfg in (("refill", dict(max_batch=4, max_active=n)),
                      ("no-refill", dict(max_batch=5, max_active=n, refill=False)),
                      ("refill-boundary-stream", dict(max_batch=4, max_active=n, min_coda_batch=2,
                                                      boundary_stream=2)),
                      ("refill-graph", dict(max_batch=4, max_active=n, graph_loop=True))):
        first, ids, st, secs = _decode_on_gpu(s, gm, prompts, ndec, depths, kv_layout, **cfg)
        _say(f"[gpu]   {name}: {st} in {secs * 1e3:.1f} ms")
        assert st["tokens"] == sum(ndec)
        assert st["loop_rows"] == sum(int(x.sum()) for x in depths)
        runs[name] = (first, ids)
    for name in runs:
        assert np.array_equal(runs["refill"][0], runs[name][0]), name
        assert np.array_equal(runs["refill"][1], runs[name][1]), name
    checked = _check_against_oracle(s, w, prompts, ndec, depths, *runs["refill"], kv_layout)
    _say(f"[gpu]   {checked} greedy ids checked against the oracle")
    assert checked >= 0.3 * (sum(ndec) + n)


@pytest.mark.parametrize("kv_layout", [1, 2], ids=["shared", "first-then-shared"])
def test_shared_layouts_call_by_call(kv_layout):
    from lockstep import Lockstep
    s = cdbgen.TINY
    _say(f"[gpu] lockstep {s.name} kv layout {kv_layout}")
    w = cdbgen.model_weights(s)
    prompts, ndec, depths = _requests(s, seed=50)
    deps = [np.concatenate([np.full(len(p), s.r_max, np.int32), d]) for p, d in zip(prompts, depths)]
    ls = Lockstep(s, w, [len(p) + k for p, k in zip(prompts, ndec)], max_batch=4, kv_layout=kv_layout)
    ls.run(prompts, ndec, deps)
    _say(f"[gpu]   errors {ls.errors} calls {ls.calls} argmax checked {ls.argmax_checked}")
    assert ls.device_error() == 0


def test_driver_rejects_short_token_table():
    s = cdbgen.TINY
    gm = cdb.DeviceModel(s, cdbgen.model_weights(s))
    d = drv.Driver(max_batch=2, max_active=1, r_max=s.r_max, max_seqs=1, max_pages=2, core_pages=8,
                   pre_pages=2, coda_pages=2, has_prelude=True, has_coda=True)
    d.add_sequence(4, [1, 2, 3])
    kv = cdb.PagedKV(s, 1, 2, 2, 8, 2)
    ws = cdb.Workspace(gm.desc, 4)
    st = cdb.State(s, 1)
    scratch = torch.empty(d.scratch_bytes(s.vocab), dtype=torch.uint8, device="cuda")
    short = torch.zeros((1, 2), dtype=torch.int32, device="cuda")
    with pytest.raises(cdb.CdbError):
        d.run(gm.model, kv.c, st.c, scratch, np.zeros(1, np.int32), ws.buf, tokens_out=short)
    assert d.stats()["loop_steps"] == 0


def _gate_threshold(shape, w, prompts):
    """A threshold the model's exit scores straddle: the median, over the first
    prompt under the oracle, of the loop-1 gate scores, or for the convergence
    criterion (first applied after loop 2) of the loop-2 distances."""
    m = oracle.Model(shape, w, bf16_storage=True)
    p = prompts[0]
    ref = m.ref_sequence(p, np.full(len(p), shape.r_max, np.int32))
    return float(np.median(ref["scores"][:, 1 if shape.exit_kind == 1 else 0]))


# the learned gate (the tiny model) and the convergence criterion (the d = 192
# model with the adapter, at r_max 4 so that its earliest lookahead exit, after
# loop 3, comes before r_max)
@pytest.mark.parametrize("shape_name", ["tiny", "inj"], ids=["tiny-gate", "inj-convergence"])
def test_lookahead_gate_call_by_call(shape_name):
    from lockstep import Lockstep
    s = cdbgen.TINY if shape_name == "tiny" else dataclasses.replace(INJ, name="inj-1-2-1-r4", r_max=4)
    w = cdbgen.model_weights(s)
    prompts, ndec, depths = _requests(s, seed=70)
    thr = _gate_threshold(s, w, prompts)
    _say(f"[gpu] lockstep {s.name} lookahead gate, threshold {thr:.4f}")
    deps = [np.concatenate([np.full(len(p), s.r_max, np.int32), np.full(k, s.r_max, np.int32)])
            for p, k in zip(prompts, ndec)]
    ls = Lockstep(s, w, [len(p) + k for p, k in zip(prompts, ndec)], max_batch=4, gate=(thr, True))
    ls.run(prompts, ndec, deps)
    _say(f"[gpu]   errors {ls.errors} calls {ls.calls} gate {ls.gate_stats}")
    assert ls.device_error() == 0
    assert ls.gate_stats["exits_before_r_max"] > 0 and ls.gate_stats["decisions"] > 0


@pytest.mark.parametrize("lookahead", [True, False], ids=["lookahead", "same-step"])
def test_gated_driver_decode_is_schedule_invariant(lookahead):
    s = cdbgen.TINY
    w = cdbgen.model_weights(s)
    gm = cdb.DeviceModel(s, w)
    prompts, ndec, _ = _requests(s, seed=71)
    n = len(prompts)
    thr = _gate_threshold(s, w, prompts)
    _say(f"[gpu] gated driver decode {s.name}, lookahead {lookahead}, threshold {thr:.4f}")
    runs = {}
    for name, cfg in (("refill", dict(max_batch=4, max_active=n)),
                      ("no-refill", dict(max_batch=3, max_active=n, refill=False)),
                      ("refill-boundary-stream", dict(max_batch=4, max_active=n, boundary_stream=1)),
                      ("refill-graph", dict(max_batch=4, max_active=n, graph_loop=True))):
        first, ids, st, secs = _decode_on_gpu(s, gm, prompts, ndec, [None] * n, gated=True, lookahead=lookahead,
                                              threshold=thr, **cfg)
        _say(f"[gpu]   {name}: {st} in {secs * 1e3:.1f} ms")
        assert st["tokens"] == sum(ndec)
        runs[name] = (first, ids, st["loop_rows"])
    a = runs["refill"]
    for name, b in runs.items():
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]) and a[2] == b[2], name
    lo = sum(ndec) * (2 if lookahead else 1)
    assert lo <= a[2] < sum(ndec) * s.r_max  # some tokens exit early, none before the minimum depth


def _first_ids_by_prefill(shape, gm, prompts, chunk):
    """Each prompt through cdb_prefill in the driver's chunking on a pool of its
    own: the last chunk's greedy id (last-row-only mode) is the first decode
    input the driver computes (a chunk's rows do not depend on other
    sequences).  The full-logits mode must give the same id."""
    R = shape.r_max
    first = np.zeros(len(prompts), np.int32)
    for q, p in enumerate(prompts):
        pages = cdbgen.pages_for(len(p))
        kv = cdb.PagedKV(shape, 1, pages, pages, pages * R, pages)
        pt = np.full((1, R + 2, pages), -1, np.int32)
        for plane in range(R + 2):
            pt[0, plane, :] = np.arange(pages) + (plane - 1) * pages if 1 <= plane <= R else np.arange(pages)
        kv.page_table.copy_(torch.from_numpy(pt))
        ws = cdb.Workspace(gm.desc, chunk)
        nxt = torch.zeros(chunk, dtype=torch.int32, device="cuda")
        for p0 in range(0, len(p), chunk):
            tok = torch.as_tensor(p[p0:p0 + chunk], dtype=torch.int32, device="cuda")
            cdb.cdb_prefill(gm.model, kv.c, 0, p0, tok, None, nxt, ws.buf)
        torch.cuda.synchronize()
        first[q] = int(nxt[0].item())
        # full logits for the last chunk again (same cache contents): same argmax
        p0 = (len(p) - 1) // chunk * chunk
        tok = torch.as_tensor(p[p0:], dtype=torch.int32, device="cuda")
        lg = torch.empty((len(tok), shape.vocab), dtype=torch.float32, device="cuda")
        ids = torch.empty(len(tok), dtype=torch.int32, device="cuda")
        cdb.cdb_prefill(gm.model, kv.c, 0, p0, tok, lg, ids, ws.buf)
        torch.cuda.synchronize()
        assert int(ids[-1].item()) == first[q]
        assert cdb.cdb_read_device_error(ws.buf) == 0
    return first


def _decode_with_driver_prefill(shape, gm, prompts, ndec, depths, chunk, arrivals=None, **cfg):
    R = shape.r_max
    n = len(prompts)
    T = [len(p) + k for p, k in zip(prompts, ndec)]
    max_pages = max(cdbgen.pages_for(t) for t in T)
    tot = sum(cdbgen.pages_for(t) for t in T)
    d = drv.Driver(max_seqs=n, max_pages=max_pages, core_pages=tot * R, pre_pages=tot, coda_pages=tot,
                   has_prelude=shape.n_prelude > 0, has_coda=shape.n_coda > 0, r_max=R, prefill_chunk=chunk, **cfg)
    for q in range(n):
        d.add_request(prompts[q], depths[q], arrival=0.0 if arrivals is None else arrivals[q])
    kv = cdb.PagedKV(shape, n, max_pages, tot, tot * R, tot)
    ws, half = _driver_ws(gm, max(256, chunk), cfg)
    state = cdb.State(shape, n)
    scratch = torch.empty(d.scratch_bytes(shape.vocab), dtype=torch.uint8, device="cuda")
    out_ids = torch.full((n, max(ndec)), -1, dtype=torch.int32, device="cuda")
    secs = d.run(gm.model, kv.c, state.c, scratch, None, ws, tokens_out=out_ids)
    torch.cuda.synchronize()
    assert _ws_errors(ws, half) == [0] * (2 if cfg.get("boundary_stream") else 1)
    if arrivals is not None:
        # every request finished after it arrived, and the run lasted past the last arrival
        lat = d.latencies(n)
        assert len(lat) == n and (lat > 0).all() and secs >= max(arrivals)
    return out_ids.cpu().numpy(), d.stats(), secs


def test_driver_prefill_chunks_decode_like_the_oracle():
    s = cdbgen.TINY
    chunk = 16
    _say(f"[gpu] driver-run prefill {s.name}, chunks of {chunk}")
    w = cdbgen.model_weights(s)
    gm = cdb.DeviceModel(s, w)
    prompts, ndec, depths = _requests(s)
    n = len(prompts)
    first = _first_ids_by_prefill(s, gm, prompts, chunk)
    runs = {}
    for name, cfg in (("refill", dict(max_batch=4, max_active=n)),
                      ("no-refill", dict(max_batch=3, max_active=n, refill=False)),
                      ("two-at-a-time", dict(max_batch=2, max_active=2)),
                      ("boundary-stream", dict(max_batch=4, max_active=3, boundary_stream=2)),
                      ("graph", dict(max_batch=4, max_active=n, graph_loop=True)),
                      # requests arriving while others decode (wall-clock seconds from the run's start):
                      # admissions mid-run and waits for the next arrival, as in the serving trace
                      ("arrivals", dict(max_batch=4, max_active=n, arrivals=[0.0, 0.0, 0.004, 0.008, 0.016, 0.03]))):
        ids, st, secs = _decode_with_driver_prefill(s, gm, prompts, ndec, depths, chunk, **cfg)
        _say(f"[gpu]   {name}: {st} in {secs * 1e3:.1f} ms")
        assert st["tokens"] == sum(ndec)
        assert st["prefill_tokens"] == sum(len(p) for p in prompts)
        assert st["prefill_calls"] == sum(-(-len(p) // chunk) for p in prompts)
        runs[name] = ids
    for name, ids in runs.items():
        assert np.array_equal(ids, runs["refill"]), name
    checked = _check_against_oracle(s, w, prompts, ndec, depths, first, runs["refill"], drv.KV_FULL)
    _say(f"[gpu]   {checked} greedy ids checked against the oracle")
    assert checked >= 0.3 * (sum(ndec) + n)


def test_driver_decode_at_ouro_width_follows_oracle():
    # the real projection widths (d 2048, 16 x 128 heads, SwiGLU 5632) with a
    # 2-layer core: skinny GEMMs of every row count the schedule produces
    s = cdbgen.shrink(cdbgen.OURO, n_core=2)
    w = cdbgen.model_weights(cdbgen.OURO)
    w = dict(w, layers=w["layers"][:2])
    _say(f"[gpu] driver decode at Ouro widths, 2 core layers")
    gm = cdb.DeviceModel(s, w)
    plens, ndec = [12, 5, 20, 9], [6, 8, 5, 7]
    prompts = [cdbgen.prompt_ids(s.vocab, 1, p, seed=46, stream=q)[0] for q, p in enumerate(plens)]
    depths = [cdbgen.draw_depths(cdbgen.OURO_DEPTHS, n, s.r_max, seed=47, stream=q) for q, n in enumerate(ndec)]
    runs = {}
    for name, cfg in (("refill", dict(max_batch=3, max_active=4)),
                      ("no-refill", dict(max_batch=4, max_active=4, refill=False)),
                      ("refill-boundary-stream", dict(max_batch=3, max_active=4, boundary_stream=1)),
                      ("refill-graph", dict(max_batch=3, max_active=4, graph_loop=True))):
        first, ids, st, secs = _decode_on_gpu(s, gm, prompts, ndec, depths, drv.KV_FULL, **cfg)
        _say(f"[gpu]   {name}: {st} in {secs * 1e3:.1f} ms")
        assert st["tokens"] == sum(ndec)
        runs[name] = (first, ids)
    for name in runs:
        assert np.array_equal(runs["refill"][0], runs[name][0]), name
        assert np.array_equal(runs["refill"][1], runs[name][1]), name
    checked = _check_against_oracle(s, w, prompts, ndec, depths, *runs["refill"], drv.KV_FULL)
    _say(f"[gpu]   {checked} greedy ids checked against the oracle")
    assert checked >= 0.3 * (sum(ndec) + len(plens))
