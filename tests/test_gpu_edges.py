"""GPU: edge cases of the stage calls.

* Empty calls are no-ops (a loop step over zero rows still reports zero counts);
  an empty prefill chunk is refused.
* Row counts that leave ragged 32-row tiles in every skinny-GEMM tile size
  (1, 31, 33, 100, 255 rows) at the Ouro widths, checked like the full-batch
  parity tests: integer outputs for the whole batch, sampled rows against the
  oracle.
* Degenerate exit patterns: every row exits (depth = c + 1, depths 1..r_max, so
  every exiting row below r_max copies its entry into the deeper planes), and no
  row exits.
* The benchmark's loop step run twice from the same state and cache is
  bit-identical (determinism).
* Conditions the device detects are reported through the sticky error word and
  never make a kernel touch memory outside its buffers: an unmapped page inside a
  row's context, an unmapped write page, a slot outside the state pool.  They are
  forced from the host through the page table and the row arrays.
"""
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


def _ouro_two_layers():
    s = cdbgen.shrink(cdbgen.OURO, n_core=2)
    w = cdbgen.model_weights(cdbgen.OURO)
    w = dict(w, layers=w["layers"][:2])
    return s, w


def _sample_rows(rows_np, r_max):
    from lockstep import sample_rows
    return sample_rows(rows_np, r_max)


def test_empty_stage_calls():
    s = cdbgen.TINY
    R = s.r_max
    gm = cdb.DeviceModel(s, cdbgen.model_weights(s))
    kv = cdb.PagedKV(s, 2, 4, 8, 8 * R, 8, fill="random")
    pt = np.arange(2 * (R + 2) * 4, dtype=np.int32).reshape(2, R + 2, 4) % 8
    kv.page_table.copy_(torch.from_numpy(pt))
    state = cdb.State(s, 2)
    state.h.normal_(0.0, 1.0)
    pools = [kv.pre.clone(), kv.core.clone(), kv.coda.clone()]
    h0 = state.h.clone()
    ws = cdb.Workspace(gm.desc, 4)
    empty = np.zeros(0, np.int32)
    rows = cdb.Rows(empty, empty, empty, empty, empty)
    out = cdb.StepOut(1)
    out.counts.fill_(7)
    tokens = torch.zeros(1, dtype=torch.int32, device="cuda")
    logits = torch.zeros((1, s.vocab), dtype=torch.float32, device="cuda")
    ids = torch.zeros(1, dtype=torch.int32, device="cuda")
    _say("[gpu] empty prelude / loop step / coda / attention calls on the tiny model")
    cdb.cdb_boundary_prelude(gm.model, kv.c, state.c, rows.c, tokens, ws.buf)
    cdb.cdb_loop_step(gm.model, kv.c, state.c, rows.c, out.c, ws.buf)
    cdb.cdb_boundary_coda(gm.model, kv.c, state.c, rows.c, logits, ids, ws.buf)
    q = torch.zeros((1, s.d), dtype=torch.float32, device="cuda")
    o = torch.zeros((1, s.d), dtype=torch.bfloat16, device="cuda")
    cdb.cdb_paged_attention(gm.desc, kv.c, rows.c, 1, 0, q, o, ws.buf)
    torch.cuda.synchronize()
    assert out.counts.cpu().tolist() == [0, 0]
    assert torch.equal(state.h, h0)
    for a, b in zip(pools, (kv.pre, kv.core, kv.coda)):
        assert torch.equal(a, b)
    assert cdb.cdb_read_device_error(ws.buf) == cdb.CDB_DEV_OK
    with pytest.raises(cdb.CdbError):
        cdb.cdb_prefill(gm.model, kv.c, 0, 0, tokens[:0], logits, ids, ws.buf)


@pytest.mark.parametrize("n_rows", [1, 31, 33, 100, 255])
def test_ragged_row_counts_at_ouro_width(n_rows):
    from lockstep import injected_loop_step
    s, w = _ouro_two_layers()
    rows = cdbgen.decode_snapshot(n_rows, cdbgen.OURO_DEPTHS, s.r_max, 512, 767, stream=60 + n_rows)
    sample = _sample_rows(rows, s.r_max)
    _say(f"[gpu] Ouro widths, 2 core layers, {n_rows} rows; sampled rows {sample}")
    err = injected_loop_step(s, w, rows, sample, sensitivity=True)
    _say(f"[gpu]   errors {err}")


@pytest.mark.parametrize("pattern", ["all_exit", "none_exit"])
def test_degenerate_exit_patterns(pattern):
    from lockstep import injected_loop_step
    s, w = _ouro_two_layers()
    R = s.r_max
    rows = cdbgen.decode_snapshot(64, cdbgen.OURO_DEPTHS, R, 512, 767, stream=70)
    g = np.random.default_rng(5)
    if pattern == "all_exit":
        rows["c"] = g.integers(0, R, 64).astype(np.int32)
        rows["depth"] = rows["c"] + 1
    else:
        rows["depth"] = np.full(64, R, np.int32)
        rows["c"] = g.integers(0, R - 1, 64).astype(np.int32)
    sample = _sample_rows(rows, R)
    _say(f"[gpu] {pattern}: c {rows['c'][:8]} depth {rows['depth'][:8]}; sampled rows {sample}")
    err = injected_loop_step(s, w, rows, sample, sensitivity=True)
    _say(f"[gpu]   errors {err}")


def _tiny_step_setup(n=4, seed=3):
    s = cdbgen.TINY
    R = s.r_max
    gm = cdb.DeviceModel(s, cdbgen.model_weights(s))
    pos = np.array([40, 47, 52, 60], np.int32)[:n]
    c = np.array([0, 1, 2, 3], np.int32)[:n]
    depth = np.array([1, 3, 4, 4], np.int32)[:n]
    max_pages = cdbgen.pages_for(int(pos.max()) + 1)
    n_pages = n * max_pages * R
    pt = np.full((n, R + 2, max_pages), -1, np.int32)
    pt[:, 1:R + 1, :] = np.arange(n_pages, dtype=np.int32).reshape(n, R, max_pages)
    kv = cdb.PagedKV(s, n, max_pages, 0, n_pages, 0, fill="random")
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    kv.core.normal_(0.0, 1.0, generator=g)
    state = cdb.State(s, n)
    state.h.normal_(0.0, 1.0, generator=g)
    return s, gm, kv, pt, state, pos, c, depth


@pytest.mark.parametrize("case", ["context_page", "write_page"])
def test_unmapped_page_is_reported(case):
    s, gm, kv, pt, state, pos, c, depth = _tiny_step_setup()
    i = 2
    if case == "context_page":
        pt[i, c[i] + 1, 1] = -1  # positions 16..31 of row 2's plane
    else:
        pt[i, c[i] + 1, pos[i] // 16] = -1  # the page row 2 writes its new entry to
    kv.page_table.copy_(torch.from_numpy(pt))
    n = len(pos)
    rows = cdb.Rows(np.arange(n, dtype=np.int32), np.arange(n, dtype=np.int32), pos, c, depth)
    out = cdb.StepOut(n)
    ws = cdb.Workspace(gm.desc, n)
    _say(f"[gpu] tiny loop step with an unmapped {case.replace('_', ' ')} in row {i}")
    cdb.cdb_loop_step(gm.model, kv.c, state.c, rows.c, out.c, ws.buf)
    torch.cuda.synchronize()
    assert cdb.cdb_read_device_error(ws.buf) == cdb.CDB_DEV_UNMAPPED_PAGE
    assert out.counts.cpu().tolist() == [int((c + 1 < depth).sum()), int((c + 1 == depth).sum())]


def test_bad_loop_index_writes_no_other_page():
    """A row whose loop index c is r_max (past its last core plane) is reported
    as a bad depth, and its K/V write does not land in the page its sequence's
    coda-plane entry names (here another row's context page, which must stay
    unchanged)."""
    s, gm, kv, pt, state, pos, c, depth = _tiny_step_setup()
    R = s.r_max
    i, victim = 2, int(pt[0, 1, 0])  # row 0's plane-1 positions 0..15: read-only in this step
    c = c.copy()
    c[i] = R
    pt[i, R + 1, pos[i] // 16] = victim
    kv.page_table.copy_(torch.from_numpy(pt))
    before = kv.core[:, victim].clone()
    n = len(pos)
    rows = cdb.Rows(np.arange(n, dtype=np.int32), np.arange(n, dtype=np.int32), pos, c, depth)
    out = cdb.StepOut(n)
    ws = cdb.Workspace(gm.desc, n)
    _say(f"[gpu] tiny loop step with c = r_max in row {i}")
    cdb.cdb_loop_step(gm.model, kv.c, state.c, rows.c, out.c, ws.buf)
    torch.cuda.synchronize()
    assert cdb.cdb_read_device_error(ws.buf) == cdb.CDB_DEV_BAD_DEPTH
    assert torch.equal(kv.core[:, victim], before)


def test_slot_outside_the_pool_is_reported():
    s, gm, kv, pt, state, pos, c, depth = _tiny_step_setup()
    kv.page_table.copy_(torch.from_numpy(pt))
    n = len(pos)
    slots = np.arange(n, dtype=np.int32)
    slots[1] = n + 5
    h0 = state.h.clone()
    rows = cdb.Rows(slots, np.arange(n, dtype=np.int32), pos, c, depth)
    out = cdb.StepOut(n)
    ws = cdb.Workspace(gm.desc, n)
    _say("[gpu] tiny loop step with a slot outside the state pool")
    cdb.cdb_loop_step(gm.model, kv.c, state.c, rows.c, out.c, ws.buf)
    torch.cuda.synchronize()
    assert cdb.cdb_read_device_error(ws.buf) == cdb.CDB_DEV_BAD_INDEX
    # the valid rows' states were written, the pool has no row for the bad one
    assert not torch.equal(state.h[0], h0[0])


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


def _batch_invariance(shape, w, rows_np, n_small):
    """The first n_small rows run alone give bit-identical states and exit scores
    to the same rows run inside the whole batch (same pages, same inputs)."""
    n = len(rows_np["pos"])
    gm = cdb.DeviceModel(shape, w)
    pt, max_pages, n_pages = _own_pages(shape, rows_np)
    kv = cdb.PagedKV(shape, n, max_pages, 0, n_pages, 0, fill="random")
    g = torch.Generator(device="cuda")
    g.manual_seed(21)
    kv.core.normal_(0.0, 1.0, generator=g)
    kv.page_table.copy_(torch.from_numpy(pt))
    state = cdb.State(shape, n)
    state.h.normal_(0.0, 1.0, generator=g)
    if shape.injection:
        state.e.normal_(0.0, 1.0, generator=g)
    h0 = state.h.clone()
    ws = cdb.Workspace(gm.desc, n)
    results = {}
    for m in (n, n_small):
        state.h.copy_(h0)
        sl = {k: rows_np[k][:m] for k in ("pos", "c", "depth")}
        rows = cdb.Rows(np.arange(m, dtype=np.int32), np.arange(m, dtype=np.int32), sl["pos"], sl["c"], sl["depth"])
        out = cdb.StepOut(m)
        cdb.cdb_loop_step(gm.model, kv.c, state.c, rows.c, out.c, ws.buf)
        torch.cuda.synchronize()
        assert cdb.cdb_read_device_error(ws.buf) == 0
        results[m] = (state.h[:n_small].clone(), out.score[:n_small].clone())
    hb, sb = results[n]
    hs, ss = results[n_small]
    diff = float((hb - hs).abs().max())
    _say(f"[gpu]   {n} vs {n_small} rows: max |h difference| {diff}")
    assert torch.equal(hb, hs) and torch.equal(sb, ss)


def test_row_results_do_not_depend_on_the_batch_ouro_width():
    s, w = _ouro_two_layers()
    rows = cdbgen.decode_snapshot(100, cdbgen.OURO_DEPTHS, s.r_max, 512, 767, stream=80)
    _say("[gpu] batch invariance, Ouro widths, 2 core layers: 100 rows (4 row tiles) vs their first 30 (1)")
    _batch_invariance(s, w, rows, 30)


def test_row_results_do_not_depend_on_the_batch_huginn_width():
    # O and down take two stripes per workgroup at 128 rows and one at 50
    s = cdbgen.shrink(cdbgen.HUGINN, n_core=1)
    w = cdbgen.model_weights(cdbgen.HUGINN)
    P = cdbgen.HUGINN.n_prelude
    w = dict(w, layers=w["layers"][:P + 1] + w["layers"][P + cdbgen.HUGINN.n_core:])
    wl = cdbgen.WORKLOADS[3]
    rows = cdbgen.decode_snapshot(128, wl.depth, s.r_max, 256, 767, stream=81)
    _say("[gpu] batch invariance, Huginn widths, 1 core layer: 128 rows vs their first 50")
    _batch_invariance(s, w, rows, 50)


def test_loop_step_is_deterministic_as_benched():
    """The benchmark's batch (64 mixed-depth rows of the 24-layer Ouro-shaped
    model at positions 512..767) run twice from the same state and cache: the
    states, exit scores, integer outputs and every written K/V entry are
    bit-identical between the runs."""
    s = cdbgen.OURO
    rows_np = cdbgen.decode_snapshot(64, cdbgen.OURO_DEPTHS, s.r_max, 512, 767, stream=7)
    n = 64
    gm = cdb.DeviceModel(s, cdbgen.model_weights(s))
    pt, max_pages, n_pages = _own_pages(s, rows_np)
    kv = cdb.PagedKV(s, n, max_pages, 0, n_pages, 0, fill="random")
    g = torch.Generator(device="cuda")
    g.manual_seed(23)
    kv.core.normal_(0.0, 1.0, generator=g)
    kv.page_table.copy_(torch.from_numpy(pt))
    state = cdb.State(s, n)
    state.h.normal_(0.0, 1.0, generator=g)
    h0 = state.h.clone()
    rows = cdb.Rows(np.arange(n, dtype=np.int32), np.arange(n, dtype=np.int32), rows_np["pos"], rows_np["c"],
                    rows_np["depth"])
    ws = cdb.Workspace(gm.desc, n)
    _say("[gpu] determinism: the benchmark's 64-row, 24-layer loop step twice")
    runs = []
    for _ in range(2):
        state.h.copy_(h0)
        out = cdb.StepOut(n)
        cdb.cdb_loop_step(gm.model, kv.c, state.c, rows.c, out.c, ws.buf)
        torch.cuda.synchronize()
        assert cdb.cdb_read_device_error(ws.buf) == 0
        runs.append((state.h.clone(), out.score.clone(), out.mask.clone(), out.cont.clone(), out.exited.clone(),
                     out.counts.clone(), kv.core.clone()))
    for a, b in zip(runs[0], runs[1]):
        assert torch.equal(a, b)
    del runs
    torch.cuda.empty_cache()


def test_coda_argmax_takes_the_lowest_index_on_exact_ties():
    """Greedy ties on the device (reading 9: the lowest index wins).  Two
    identical LM-head rows at the same position of their 32-column stripes go
    through the same arithmetic and give bit-identical logits; copying the
    winning row r to a lower such index must move the winner there, and
    copying it to a higher one must leave r."""
    s = cdbgen.TINY
    w = cdbgen.model_weights(s)
    n, R, V = 6, s.r_max, s.vocab
    pos = np.arange(n, dtype=np.int32) * 5 + 3
    ar = np.arange(n, dtype=np.int32)
    max_pages = cdbgen.pages_for(int(pos.max()) + 1)
    pt = np.full((n, R + 2, max_pages), -1, np.int32)
    pt[:, R + 1, :] = np.arange(n * max_pages).reshape(n, max_pages)
    kv = cdb.PagedKV(s, n, max_pages, 1, 1, n * max_pages, fill="random")
    g = torch.Generator(device="cuda")
    g.manual_seed(91)
    kv.coda.normal_(0.0, 1.0, generator=g)
    kv.page_table.copy_(torch.from_numpy(pt))
    coda0 = kv.coda.clone()
    state = cdb.State(s, n)
    state.h.normal_(0.0, 1.0, generator=g)
    rows = cdb.Rows(ar, ar, pos)
    gm = cdb.DeviceModel(s, w)
    ws = cdb.Workspace(gm.desc, n)

    def coda(model):
        kv.coda.copy_(coda0)  # the coda rewrites its own K/V entries; start each call from the same cache
        logits = torch.empty((n, V), dtype=torch.float32, device="cuda")
        ids = torch.empty(n, dtype=torch.int32, device="cuda")
        cdb.cdb_boundary_coda(model.model, kv.c, state.c, rows.c, logits, ids, ws.buf)
        torch.cuda.synchronize()
        assert cdb.cdb_read_device_error(ws.buf) == 0
        return logits.cpu().numpy(), ids.cpu().numpy()

    lg, ids = coda(gm)
    assert (ids == lg.argmax(axis=1)).all()  # random logits, no ties: the plain argmax
    # a row whose winner has a lower and a higher index at the same stripe position
    row = next(i for i in range(n) if 32 <= int(ids[i]) < V - 32)
    r = int(ids[row])
    head = np.asarray(w["lm_head"])
    h2d = head.reshape(V, s.d)
    for j in (r % 32, r + 32 * max(1, (V - 1 - r) // 64)):
        h2 = h2d.copy()
        h2[j] = h2d[r]
        lg2, ids2 = coda(cdb.DeviceModel(s, dict(w, lm_head=h2.reshape(head.shape))))
        _say(f"[gpu] LM-head row {r} copied to row {j}: greedy id {int(ids2[row])}")
        assert np.array_equal(lg2[:, j], lg2[:, r])  # an exact tie in every row
        assert int(ids2[row]) == min(j, r)
