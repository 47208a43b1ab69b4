"""The host driver's scheduler and page allocator (Section 4.1, Fig. 1;
Section 4.2, Table 1) and the FLOP bound (Section 5, Eq. 2), stepped without a
device.  CPU only."""
import json
import os

import numpy as np
import pytest

import cdbgen
import paper_2608_09444_amd as cdb
from paper_2608_09444_amd import cost
from paper_2608_09444_amd.driver import (KV_FIRST_THEN_SHARED, KV_FULL, KV_SHARED, TICK_CODA, TICK_LOOP,
                                         TICK_PREFILL, TICK_PRELUDE_FIRST, Driver)

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def fig1_driver(refill):
    g = json.load(open(os.path.join(GOLD, "fig1_slot_grid.json")))
    d = Driver(max_batch=g["batch_slots"], max_active=2, r_max=3, max_seqs=3, max_pages=1, core_pages=64,
               refill=refill)
    for q in ("1", "2", "3"):
        d.add_sequence(1, g["depth_tables"][q])
    return d, g


def loop_cells(ticks):
    """(sequence, token, loop) cells of every loop step, numbered from 1 as in Fig. 1."""
    out = []
    for t in ticks:
        if t.stage == TICK_LOOP:
            out.append(sorted((t.seq[i] + 1, t.decode_index[i] + 1, t.c[i] + 1) for i in range(t.n_rows)))
    return out


@pytest.mark.parametrize("mode", ["refill", "no_refill"])
def test_fig1_slot_grid(mode):
    d, g = fig1_driver(mode == "refill")
    cells = loop_cells(d.step())
    want = g[mode]
    assert len(cells) == want["passes"]
    for p, got in enumerate(cells):
        exp = sorted(tuple(c) for c in (want["slot_1"][p], want["slot_2"][p]) if c is not None)
        assert got == exp, f"pass {p + 1}"
    st = d.stats()
    assert st["loop_steps"] == want["passes"]
    assert st["idle_rows"] == want.get("idle_cells", 0)
    assert st["tokens"] == 6 and st["loop_rows"] == 12  # every token ran exactly its depth
    assert d.pages_in_use() == {"pre": 0, "core": 0, "coda": 0}


def test_fixed_depth_runs_every_token_r_max_loops():
    d, g = fig1_driver(True)
    d2 = Driver(max_batch=2, max_active=2, r_max=3, max_seqs=3, max_pages=1, core_pages=64, fixed_depth=True)
    for q in ("1", "2", "3"):
        d2.add_sequence(1, g["depth_tables"][q])
    d2.step()
    st = d2.stats()
    assert st["loop_rows"] == 6 * 3 and st["tokens"] == 6
    assert st["loop_steps"] >= 9


@pytest.mark.parametrize("refill", [True, False])
def test_refill_never_idles_while_loop_work_waits(refill):
    rng = np.random.default_rng(0)
    d = Driver(max_batch=8, max_active=12, r_max=4, max_seqs=12, max_pages=2, core_pages=12 * 2 * 4,
               refill=refill)
    for q in range(12):
        d.add_sequence(5, rng.integers(1, 5, size=int(rng.integers(1, 9))))
    in_core = set()  # sequences whose token is in the core (in the batch or waiting for it)
    short_steps = 0
    for t in d.step():
        rows = [t.seq[i] for i in range(t.n_rows)]
        if t.stage == TICK_PRELUDE_FIRST:
            in_core.update(rows)
        elif t.stage == TICK_CODA:
            in_core.update(rows[:t.n_continue])
        elif t.stage == TICK_LOOP:
            assert len(set(rows)) == len(rows) and set(rows) <= in_core
            assert all(0 <= t.c[i] < t.depth[i] for i in range(t.n_rows))
            if refill:
                assert len(rows) == min(8, len(in_core))
            short_steps += len(rows) < min(8, len(in_core))
            in_core -= {t.seq[i] for i in range(t.n_rows) if t.c[i] + 1 == t.depth[i]}
    assert refill or short_steps > 0  # no-refill lets the batch shrink
    assert d.pages_in_use()["core"] == 0


def test_loop_rows_equal_sum_of_depths_and_codas_follow_exits():
    rng = np.random.default_rng(1)
    tables = [rng.integers(1, 5, size=int(rng.integers(1, 7))) for _ in range(9)]
    d = Driver(max_batch=4, max_active=5, r_max=4, max_seqs=9, max_pages=1, core_pages=5 * 4)
    for tb in tables:
        d.add_sequence(3, tb)
    in_core = {}
    for t in d.step():
        for i in range(t.n_rows):
            key = (t.seq[i], t.decode_index[i])
            if t.stage == TICK_LOOP:
                assert in_core.get(key, 0) == t.c[i]  # loops run in order, one at a time
                in_core[key] = t.c[i] + 1
            elif t.stage == TICK_CODA:
                assert in_core[key] == tables[t.seq[i]][t.decode_index[i]]  # coda only after the last loop
    st = d.stats()
    assert st["loop_rows"] == sum(int(x.sum()) for x in tables)
    assert st["tokens"] == sum(len(x) for x in tables)


def test_min_coda_batch_accumulates_exits():
    rng = np.random.default_rng(2)
    d = Driver(max_batch=16, max_active=16, r_max=8, max_seqs=16, max_pages=1, core_pages=16 * 8,
               min_coda_batch=6)
    for q in range(16):
        d.add_sequence(2, rng.integers(1, 9, size=4))
    ticks = d.step()
    codas = [t for t in ticks if t.stage == TICK_CODA]
    assert codas
    # every coda but the ones that drain the core waits for 6 exits
    loop_work_after = []
    for k, t in enumerate(ticks):
        if t.stage == TICK_CODA:
            more = any(u.stage == TICK_LOOP for u in ticks[k + 1:])
            loop_work_after.append((t.n_rows, more))
    small = [n for n, more in loop_work_after if n < 6]
    assert len(small) < len(codas)
    assert d.stats()["tokens"] == 64


def test_admission_waits_for_kv_capacity_and_reuses_lowest_pages():
    # room for two 2-page sequences at r_max 2 (8 core pages); the third waits
    d = Driver(max_batch=4, max_active=8, r_max=2, max_seqs=3, max_pages=2, core_pages=8)
    for q in range(3):
        d.add_sequence(20, [2, 1, 2])
    first = d.next()
    assert first.stage == TICK_PRELUDE_FIRST and first.n_rows == 2
    pt = d.page_table()
    # (sequence, page, plane) order, lowest free id first
    assert pt[0, 1:3, :].T.tolist() == [[0, 1], [2, 3]]
    assert pt[1, 1:3, :].T.tolist() == [[4, 5], [6, 7]]
    assert (pt[2] == -1).all()
    d.complete(first)
    ticks = d.step()
    assert any(t.stage == TICK_PRELUDE_FIRST and t.seq[0] == 2 for t in ticks)
    assert d.pages_in_use()["core"] == 0


def test_arrivals_are_respected():
    d = Driver(max_batch=4, max_active=4, r_max=2, max_seqs=2, max_pages=1, core_pages=8)
    d.add_sequence(4, [1, 2], arrival=0.0)
    d.add_sequence(4, [2], arrival=5.0)
    t = d.next()
    assert t.stage == TICK_PRELUDE_FIRST and t.n_rows == 1
    d.complete(t)
    while True:
        t = d.next()
        if t.stage == 0:
            assert t.wait_until == 5.0
            break
        d.complete(t)
    d.set_time(5.0)
    t = d.next()
    assert t.stage == TICK_PRELUDE_FIRST and t.seq[0] == 1


@pytest.mark.parametrize("layout,core_per_page", [(KV_FULL, 3), (KV_SHARED, 1), (KV_FIRST_THEN_SHARED, 2)])
def test_page_aliasing_layouts(layout, core_per_page):
    d = Driver(max_batch=2, max_active=2, r_max=3, max_seqs=2, max_pages=2, core_pages=12, kv_layout=layout)
    d.add_sequence(20, [1, 3])
    d.add_sequence(5, [2])
    t = d.next()
    assert d.pages_in_use()["core"] == (2 + 1) * core_per_page
    pt = d.page_table()
    for q, n in ((0, 2), (1, 1)):
        for pg in range(n):
            ids = pt[q, 1:4, pg].tolist()
            assert len(set(ids)) == core_per_page
            if layout == KV_FIRST_THEN_SHARED:
                assert ids[1] == ids[2] != ids[0]
    d.complete(t)
    d.step()
    assert d.pages_in_use()["core"] == 0


def footprint(shape, layout, tokens=4096):
    """KiB per token and GiB for one sequence from the driver's page mapping
    and the library's page sizes."""
    desc = cdb.make_desc(shape)
    pages = (tokens + 15) // 16
    d = Driver(max_batch=1, max_active=1, r_max=shape.r_max, max_seqs=1, max_pages=pages,
               core_pages=pages * shape.r_max, pre_pages=pages, coda_pages=pages,
               has_prelude=shape.n_prelude > 0, has_coda=shape.n_coda > 0, kv_layout=layout)
    d.add_sequence(tokens - 1, [shape.r_max])
    d.next()
    use = d.pages_in_use()
    nbytes = sum(use[k] * cdb.cdb_kv_page_bytes(desc, i) for i, k in enumerate(("pre", "core", "coda")))
    slots = use["core"] // pages
    return slots, nbytes / tokens / 1024, nbytes / 2 ** 30


@pytest.mark.parametrize("model,shape,r", [("ouro_r4", cdbgen.OURO, 4), ("huginn_r32", cdbgen.HUGINN, 32)])
def test_kv_footprint_matches_table1(model, shape, r):
    gold = json.load(open(os.path.join(GOLD, "kv_footprint.json")))[model]
    shape = cdbgen.shrink(shape, r_max=r)
    for name, layout in (("full_depth_indexed", KV_FULL), ("single_shared", KV_SHARED),
                         ("first_then_shared", KV_FIRST_THEN_SHARED)):
        slots, kib, gib = footprint(shape, layout)
        w_slots, w_kib, w_gib = gold[name]
        assert slots == w_slots
        assert abs(kib - w_kib) <= 0.5, (name, kib)
        # the table prints two decimals; its Huginn entries sit up to 0.006 above
        # slots x KiB/tok x 4096 (10.635 -> 10.64, 0.645 -> 0.65)
        assert abs(gib - w_gib) <= 0.01, (name, gib)


# ------------------------------------------------------------ Eq. 2 FLOP bound

def test_flop_bound_ordering_and_paper_ratios():
    for shape, dbar in ((cdbgen.OURO, 2.3), (cdbgen.HUGINN, 13.45), (cdbgen.TINY, 2.5)):
        b = cost.flop_bound(shape, dbar)
        assert 1.0 < b <= shape.r_max / dbar <= shape.r_max / 1
        assert cost.flop_bound(shape, shape.r_max) == pytest.approx(1.0)
    # Section 5: Ouro's boundary work is small next to the core; Huginn's is about 1.2 F_r
    o, h = cdbgen.OURO, cdbgen.HUGINN
    assert cost.boundary_flops(o) / cost.core_flops(o) < 0.1
    assert cost.boundary_flops(h) / cost.core_flops(h) == pytest.approx(1.2, abs=0.05)
    # one loop fewer saves about 25% (Ouro, r_max 4) and about 6% (Huginn, r_max 16)
    assert cost.core_flops(o) / (cost.boundary_flops(o) + 4 * cost.core_flops(o)) == pytest.approx(0.25, abs=0.01)
    assert cost.core_flops(h) / (cost.boundary_flops(h) + 16 * cost.core_flops(h)) == pytest.approx(0.06, abs=0.005)


def test_flop_bound_at_the_workloads():
    # decode workload at Ouro, categorical depths with mean 2.3
    assert cost.flop_bound(cdbgen.OURO, 2.3) == pytest.approx(1.714, abs=2e-3)
    # 50% depth 1, 50% depth 4
    assert cost.flop_bound(cdbgen.OURO, 2.5) == pytest.approx(1.581, abs=2e-3)


# ------------------------------------------------------ driver-run prefill

def _prefill_driver(chunk, plens, ndec, arrivals=None, max_active=8, refill=True, r=3):
    d = Driver(max_batch=4, max_active=max_active, r_max=r, max_seqs=len(plens), max_pages=16,
               core_pages=16 * r * len(plens), refill=refill, prefill_chunk=chunk)
    rng = np.random.default_rng(11)
    for q, (p, n) in enumerate(zip(plens, ndec)):
        d.add_request(rng.integers(0, 100, p), rng.integers(1, r + 1, n),
                      arrival=0.0 if arrivals is None else arrivals[q])
    return d


@pytest.mark.parametrize("refill", [True, False])
def test_prompts_run_as_ordered_chunks_before_their_first_input(refill):
    plens, ndec, chunk = [37, 5, 16, 64], [3, 4, 2, 5], 16
    d = _prefill_driver(chunk, plens, ndec, refill=refill)
    ticks = d.step()
    done = {q: 0 for q in range(len(plens))}
    first_prelude = {}
    for k, t in enumerate(ticks):
        if t.stage == TICK_PREFILL:
            q = t.seq[0]
            assert t.pos[0] == done[q] and 1 <= t.n_rows <= chunk  # chunks in order, none longer than the limit
            done[q] += t.n_rows
            assert t.n_continue == int(done[q] == plens[q])
        elif t.stage == TICK_PRELUDE_FIRST:
            for i in range(t.n_rows):
                q = t.seq[i]
                assert done[q] == plens[q] and t.pos[i] == plens[q]  # the prompt is complete first
                first_prelude[q] = k
        elif t.stage == TICK_LOOP:
            for i in range(t.n_rows):
                assert t.seq[i] in first_prelude  # no decode work before the first input's prelude
    assert done == dict(enumerate(plens))
    st = d.stats()
    assert st["prefill_tokens"] == sum(plens)
    assert st["prefill_calls"] == sum(-(-p // chunk) for p in plens)
    assert st["tokens"] == sum(ndec)


def test_prefill_takes_priority_over_loop_steps_but_not_over_the_coda():
    # a second request arrives while the first decodes: its chunks run before
    # the next loop step, after any coda that is due
    d = _prefill_driver(8, [8, 24], [6, 2], arrivals=[0.0, 1.0])
    seen_second_arrival = False
    ticks = []
    while True:
        t = d.next()
        if t is None:
            break
        if t.stage == 0:
            d.set_time(t.wait_until)
            continue
        if t.stage == TICK_LOOP and not seen_second_arrival and ticks.count(TICK_LOOP) >= 3:
            d.set_time(1.0)  # the second request is now due
            seen_second_arrival = True
        assert d.complete(t) == 0
        ticks.append(t.stage)
    # after the arrival time, the three chunks of the second prompt run back to back
    i = ticks.index(TICK_PREFILL, 1)
    assert ticks[i:i + 3] == [TICK_PREFILL] * 3


def test_prefill_requests_need_the_chunk_setting():
    d = Driver(max_batch=2, max_active=2, r_max=2, max_seqs=2, max_pages=4, core_pages=16)
    with pytest.raises(ValueError):
        d.add_request([1, 2, 3], [1, 2])
    with pytest.raises(ValueError):
        Driver(max_batch=2, max_active=2, r_max=2, max_seqs=2, max_pages=4, core_pages=16, prefill_chunk=513)


def test_prefill_completion_must_follow_the_plan():
    d = _prefill_driver(4, [10], [2])
    t = d.next()
    assert t.stage == TICK_PREFILL and t.pos[0] == 0 and t.n_rows == 4
    bad = type(t).from_buffer_copy(t)
    bad.pos[0] = 4  # a chunk that is not the next one
    assert d.complete(bad) == -1
    assert d.complete(t) == 0


def test_add_sequence_rejects_what_could_never_run():
    """Bad depths, a zero-length prompt, too many sequences, out-of-order
    arrivals, and sequences longer than the page table or the pool are refused
    when added (a sequence that could never be admitted would stall the queue)."""
    d = Driver(max_batch=2, max_active=2, r_max=2, max_seqs=2, max_pages=2, core_pages=8)
    for prompt, depths in ((4, [0, 1]), (4, [1, 3]), (0, [1]), (4, [])):
        with pytest.raises(ValueError):
            d.add_sequence(prompt, depths)
    with pytest.raises(ValueError):
        d.add_sequence(30, [1, 2, 1])  # 33 positions: 3 pages > max_pages 2
    assert d.add_sequence(30, [1, 2]) == 0  # 32 positions fit 2 pages
    small = Driver(max_batch=2, max_active=2, r_max=4, max_seqs=2, max_pages=4, core_pages=7)
    with pytest.raises(ValueError):
        small.add_sequence(20, [1])  # 2 pages x 4 planes = 8 > 7 core pages
    shared = Driver(max_batch=2, max_active=2, r_max=4, max_seqs=2, max_pages=4, core_pages=7, kv_layout=KV_SHARED)
    assert shared.add_sequence(20, [1]) == 0  # 2 pages when all planes share one
    one = Driver(max_batch=2, max_active=2, r_max=2, max_seqs=1, max_pages=4, core_pages=16)
    one.add_sequence(4, [1], arrival=1.0)
    with pytest.raises(ValueError):
        one.add_sequence(4, [1], arrival=2.0)  # beyond max_seqs
    two = Driver(max_batch=2, max_active=2, r_max=2, max_seqs=2, max_pages=4, core_pages=16)
    two.add_sequence(4, [1], arrival=1.0)
    with pytest.raises(ValueError):
        two.add_sequence(4, [1], arrival=0.5)  # before the previous arrival


def test_boundary_stream_holds_new_tokens_back_one_loop_step():
    """With boundary stages on their own stream (refill), tokens whose prelude
    was just planned are held back from the next loop step.  Mode 2: they join
    the step after next, so a step holds such tokens only when it holds nothing
    else.  Mode 1: they still fill rows the loop queue leaves free, so no row
    idles while loop work waits.  Every token still runs exactly its depth,
    loops in order."""
    rng = np.random.default_rng(7)
    tables = [rng.integers(1, 5, size=int(rng.integers(2, 7))) for _ in range(10)]
    totals = {}
    for bs in (0, 1, 2):
        d = Driver(max_batch=4, max_active=6, r_max=4, max_seqs=10, max_pages=1, core_pages=6 * 4,
                   boundary_stream=bs)
        for tb in tables:
            d.add_sequence(3, tb)
        prelude_at = {}  # token -> index of the tick that ran its prelude
        last_loop = -1
        in_core = {}
        mixed = 0  # loop steps holding both just-prelude'd tokens and others
        for k, t in enumerate(d.step()):
            if t.stage == TICK_PRELUDE_FIRST:
                for i in range(t.n_rows):
                    prelude_at[(t.seq[i], 0)] = k
            elif t.stage == TICK_CODA:
                for i in range(t.n_continue):
                    prelude_at[(t.seq[i], t.decode_index[i] + 1)] = k
            elif t.stage == TICK_LOOP:
                keys = [(t.seq[i], t.decode_index[i]) for i in range(t.n_rows)]
                # tokens whose prelude ran and which have not exited
                live = {x for x in prelude_at if in_core.get(x, 0) < tables[x[0]][x[1]]}
                if bs == 1:  # no row idles while such tokens wait
                    assert len(keys) == min(4, len(live)), (k, keys, live)
                fresh = [x for x in keys if in_core.get(x, 0) == 0 and prelude_at[x] > last_loop]
                mixed += 0 < len(fresh) < len(keys)
                for i, x in enumerate(keys):
                    assert in_core.get(x, 0) == t.c[i]
                    in_core[x] = t.c[i] + 1
                last_loop = k
        st = d.stats()
        assert st["loop_rows"] == sum(int(x.sum()) for x in tables)
        assert st["tokens"] == sum(len(x) for x in tables)
        totals[bs] = st["loop_steps"]
        assert (mixed == 0) == (bs == 2) or bs == 1
    assert totals[2] >= totals[1] >= totals[0] - 1


def test_gated_lookahead_last_decisions_are_checked():
    """Gated mode with the lookahead: the last loop step's device decisions,
    given after the run, must match the exits the scheduler applied."""
    for mask, want in (([1], 0), ([0], -1)):
        d = Driver(max_batch=2, max_active=1, r_max=2, max_seqs=1, max_pages=1, core_pages=2, gated=True,
                   lookahead=True, threshold=0.5)
        d.add_sequence(1, None, n_decode=1)
        t = d.next()
        assert t.stage == TICK_PRELUDE_FIRST
        d.complete(t)
        first = d.next()
        assert first.stage == TICK_LOOP and first.c[0] == 0
        assert d.complete(first) == 0
        second = d.next()
        assert second.stage == TICK_LOOP and second.c[0] == 1
        assert d.loop_result(first, [0], [1]) == 0  # loop 1 did not end the token
        assert d.complete(second) == 0  # loop r_max ends it
        coda = d.next()
        assert coda.stage == TICK_CODA
        d.complete(coda)
        assert d.next() is None
        assert d.loop_result(second, mask, [0]) == want
