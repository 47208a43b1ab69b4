"""GPU: a loop step captured once in a HIP graph at its row capacity, with the
row count in device memory (cdb_rows.d_n_rows), replays for any count up to
that capacity and gives, bit for bit, what an eager call of exactly that many
rows gives (states, exit scores and decisions, compaction, every K/V entry).
Section 4.3: static shapes let the scheduler replay captured steps."""
import sys

import numpy as np
import pytest
import torch

import cdbgen
import paper_2608_09444_amd as cdb

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _own_pages(shape, rows_np):
    R = shape.r_max
    n = len(rows_np["pos"])
    max_pages = cdbgen.pages_for(int(rows_np["pos"].max()) + 1)
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
    return pt, max_pages, nxt


def test_captured_loop_step_replays_for_any_row_count():
    s = cdbgen.shrink(cdbgen.OURO, n_core=2)
    w = cdbgen.model_weights(cdbgen.OURO)
    w = dict(w, layers=w["layers"][:2])
    cap = 64
    rows_np = cdbgen.decode_snapshot(cap, cdbgen.OURO_DEPTHS, s.r_max, 512, 767, stream=90)
    gm = cdb.DeviceModel(s, w)
    pt, max_pages, n_pages = _own_pages(s, rows_np)
    kv = cdb.PagedKV(s, cap, max_pages, 0, n_pages, 0, fill="random")
    g = torch.Generator(device="cuda")
    g.manual_seed(31)
    kv.core.normal_(0.0, 1.0, generator=g)
    kv.page_table.copy_(torch.from_numpy(pt))
    state = cdb.State(s, cap)
    state.h.normal_(0.0, 1.0, generator=g)
    h0, kv0 = state.h.clone(), kv.core.clone()
    ar = np.arange(cap, dtype=np.int32)

    def restore():
        state.h.copy_(h0)
        kv.core.copy_(kv0)

    d_n = torch.full((1,), cap, dtype=torch.int32, device="cuda")
    rows_g = cdb.Rows(ar, ar, rows_np["pos"], rows_np["c"], rows_np["depth"], d_n_rows=d_n)
    out_g = cdb.StepOut(cap)
    ws_g = cdb.Workspace(gm.desc, cap)
    ws_e = cdb.Workspace(gm.desc, cap)
    # one eager call of the captured shape first (kernel attributes are set on first use)
    cdb.cdb_loop_step(gm.model, kv.c, state.c, rows_g.c, out_g.c, ws_g.buf)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            cdb.cdb_loop_step(gm.model, kv.c, state.c, rows_g.c, out_g.c, ws_g.buf, stream=side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for n in (17, 40, 64, 17):
        _say(f"[gpu] graph captured at {cap} rows, replayed at {n} rows, against an eager call of {n} rows")
        restore()
        sl = slice(0, n)
        rows_e = cdb.Rows(ar[sl], ar[sl], rows_np["pos"][sl], rows_np["c"][sl], rows_np["depth"][sl])
        out_e = cdb.StepOut(n)
        cdb.cdb_loop_step(gm.model, kv.c, state.c, rows_e.c, out_e.c, ws_e.buf)
        torch.cuda.synchronize()
        assert cdb.cdb_read_device_error(ws_e.buf) == 0
        want = (state.h.clone(), kv.core.clone())
        restore()
        d_n.fill_(n)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert cdb.cdb_read_device_error(ws_g.buf) == 0
        assert torch.equal(state.h, want[0])  # rows past n leave their slots alone
        assert torch.equal(kv.core, want[1])
        cnt = out_e.counts.cpu().tolist()
        assert out_g.counts.cpu().tolist() == cnt
        for a, b in ((out_g.score, out_e.score), (out_g.mask, out_e.mask), (out_g.exit_next, out_e.exit_next)):
            assert torch.equal(a[:n], b[:n])
        assert torch.equal(out_g.cont[:cnt[0]], out_e.cont[:cnt[0]])
        assert torch.equal(out_g.exited[:cnt[1]], out_e.exited[:cnt[1]])
    del graph
    torch.cuda.empty_cache()


def test_device_row_count_in_eager_loop_step():
    """An eager (uncaptured) loop step of 64 rows of capacity with a device row
    count: for live counts below and at a 32-row tile and up to the capacity,
    every row's results equal those of a call of exactly that many rows, and
    outputs past the count are left alone."""
    s = cdbgen.shrink(cdbgen.OURO, n_core=2)
    w = cdbgen.model_weights(cdbgen.OURO)
    w = dict(w, layers=w["layers"][:2])
    cap = 64
    rows_np = cdbgen.decode_snapshot(cap, cdbgen.OURO_DEPTHS, s.r_max, 512, 767, stream=91)
    gm = cdb.DeviceModel(s, w)
    pt, max_pages, n_pages = _own_pages(s, rows_np)
    kv = cdb.PagedKV(s, cap, max_pages, 0, n_pages, 0, fill="random")
    g = torch.Generator(device="cuda")
    g.manual_seed(33)
    kv.core.normal_(0.0, 1.0, generator=g)
    kv.page_table.copy_(torch.from_numpy(pt))
    state = cdb.State(s, cap)
    state.h.normal_(0.0, 1.0, generator=g)
    h0, kv0 = state.h.clone(), kv.core.clone()
    ar = np.arange(cap, dtype=np.int32)
    d_n = torch.full((1,), cap, dtype=torch.int32, device="cuda")
    rows_d = cdb.Rows(ar, ar, rows_np["pos"], rows_np["c"], rows_np["depth"], d_n_rows=d_n)
    out_d = cdb.StepOut(cap)
    ws_d = cdb.Workspace(gm.desc, cap)
    ws_e = cdb.Workspace(gm.desc, cap)
    for n in (20, 32, 56, 64):
        _say(f"[gpu] eager loop step at {cap} rows of capacity with {n} live rows, against a call of {n} rows")
        state.h.copy_(h0)
        kv.core.copy_(kv0)
        sl = slice(0, n)
        rows_e = cdb.Rows(ar[sl], ar[sl], rows_np["pos"][sl], rows_np["c"][sl], rows_np["depth"][sl])
        out_e = cdb.StepOut(n)
        cdb.cdb_loop_step(gm.model, kv.c, state.c, rows_e.c, out_e.c, ws_e.buf)
        torch.cuda.synchronize()
        assert cdb.cdb_read_device_error(ws_e.buf) == 0
        want = (state.h.clone(), kv.core.clone())
        state.h.copy_(h0)
        kv.core.copy_(kv0)
        d_n.fill_(n)
        out_d.score.fill_(-1.0)
        cdb.cdb_loop_step(gm.model, kv.c, state.c, rows_d.c, out_d.c, ws_d.buf)
        torch.cuda.synchronize()
        assert cdb.cdb_read_device_error(ws_d.buf) == 0
        assert torch.equal(state.h, want[0])
        assert torch.equal(kv.core, want[1])
        cnt = out_e.counts.cpu().tolist()
        assert out_d.counts.cpu().tolist() == cnt
        for a, b in ((out_d.score, out_e.score), (out_d.mask, out_e.mask), (out_d.exit_next, out_e.exit_next)):
            assert torch.equal(a[:n], b[:n])
        assert bool((out_d.score[n:] == -1.0).all())
        assert torch.equal(out_d.cont[:cnt[0]], out_e.cont[:cnt[0]])
        assert torch.equal(out_d.exited[:cnt[1]], out_e.exited[:cnt[1]])


def test_device_row_count_in_boundary_calls():
    """Prelude and coda with a device row count: the first n rows' states,
    logits and greedy ids equal an eager call of n rows; the other rows'
    outputs are untouched."""
    s = cdbgen.TINY
    w = cdbgen.model_weights(s)
    gm = cdb.DeviceModel(s, w)
    cap, n = 12, 7
    R = s.r_max
    pos = np.arange(cap, dtype=np.int32) + 3
    ar = np.arange(cap, dtype=np.int32)
    max_pages = cdbgen.pages_for(int(pos.max()) + 1)
    pt = np.full((cap, R + 2, max_pages), -1, np.int32)
    pt[:, 0, :] = np.arange(cap * max_pages).reshape(cap, max_pages)
    pt[:, R + 1, :] = np.arange(cap * max_pages).reshape(cap, max_pages)
    kv = cdb.PagedKV(s, cap, max_pages, cap * max_pages, 1, cap * max_pages, fill="random")
    g = torch.Generator(device="cuda")
    g.manual_seed(32)
    kv.pre.normal_(0.0, 1.0, generator=g)
    kv.coda.normal_(0.0, 1.0, generator=g)
    kv.page_table.copy_(torch.from_numpy(pt))
    toks = torch.as_tensor(np.arange(cap) * 37 % s.vocab, dtype=torch.int32, device="cuda")
    ws = cdb.Workspace(gm.desc, cap)
    pre0, coda0 = kv.pre.clone(), kv.coda.clone()
    results = []
    for dev_count in (False, True):
        kv.pre.copy_(pre0)
        kv.coda.copy_(coda0)
        state = cdb.State(s, cap)
        state.h.fill_(7.0)
        d_n = torch.full((1,), n, dtype=torch.int32, device="cuda") if dev_count else None
        m = cap if dev_count else n
        rows = cdb.Rows(ar[:m], ar[:m], pos[:m], d_n_rows=d_n)
        cdb.cdb_boundary_prelude(gm.model, kv.c, state.c, rows.c, toks[:m], ws.buf)
        logits = torch.full((cap, s.vocab), -5.0, dtype=torch.float32, device="cuda")
        ids = torch.full((cap,), -1, dtype=torch.int32, device="cuda")
        cdb.cdb_boundary_coda(gm.model, kv.c, state.c, rows.c, logits[:m], ids[:m], ws.buf)
        torch.cuda.synchronize()
        assert cdb.cdb_read_device_error(ws.buf) == 0
        results.append((state.h.clone(), logits, ids, kv.pre.clone(), kv.coda.clone()))
    (h_e, l_e, i_e, p_e, c_e), (h_g, l_g, i_g, p_g, c_g) = results
    _say(f"[gpu] prelude + coda at {cap} rows of capacity with {n} live rows")
    assert torch.equal(h_g, h_e)  # slots past n keep their 7.0
    assert torch.equal(l_g, l_e) and torch.equal(i_g, i_e)  # logits and ids past n untouched
    assert torch.equal(p_g, p_e) and torch.equal(c_g, c_e)
