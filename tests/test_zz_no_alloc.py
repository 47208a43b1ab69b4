"""GPU: cdb_loop_step_noalloc (scratch in a static device array, nothing
allocated) against cdb_loop_step (caller's workspace) on the same inputs:
bit-identical states, exit scores and decisions, compaction and K/V, over two
calls in a row, the second with fewer rows; and the scratch limit refused on
the host."""
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


def test_noalloc_loop_step_equals_workspace_call():
    s = cdbgen.shrink(cdbgen.OURO, n_core=2)
    w = cdbgen.model_weights(cdbgen.OURO)
    w = dict(w, layers=w["layers"][:2])
    n_big, n_small = 64, 40
    rows_np = cdbgen.decode_snapshot(n_big, cdbgen.OURO_DEPTHS, s.r_max, 512, 767, stream=95)
    gm = cdb.DeviceModel(s, w)
    pt, max_pages, n_pages = _own_pages(s, rows_np)
    kv = cdb.PagedKV(s, n_big, max_pages, 0, n_pages, 0, fill="random")
    g = torch.Generator(device="cuda")
    g.manual_seed(41)
    kv.core.normal_(0.0, 1.0, generator=g)
    kv.page_table.copy_(torch.from_numpy(pt))
    state = cdb.State(s, n_big)
    state.h.normal_(0.0, 1.0, generator=g)
    h0, kv0 = state.h.clone(), kv.core.clone()
    ws = cdb.Workspace(gm.desc, n_big)
    d_err = torch.zeros(1, dtype=torch.int32, device="cuda")
    ar = np.arange(n_big, dtype=np.int32)

    def run(noalloc):
        state.h.copy_(h0)
        kv.core.copy_(kv0)
        res = []
        for n in (n_big, n_small):  # two calls in a row, the second smaller
            sl = slice(0, n)
            rows = cdb.Rows(ar[sl], ar[sl], rows_np["pos"][sl], rows_np["c"][sl], rows_np["depth"][sl])
            out = cdb.StepOut(n)
            if noalloc:
                cdb.cdb_loop_step_noalloc(gm.model, kv.c, state.c, rows.c, out.c, d_err)
            else:
                cdb.cdb_loop_step(gm.model, kv.c, state.c, rows.c, out.c, ws.buf)
            torch.cuda.synchronize()
            cnt = out.counts.cpu().tolist()
            res.append((state.h.clone(), out.score[:n].clone(), out.mask[:n].clone(), out.exit_next[:n].clone(),
                        out.cont[:cnt[0]].clone(), out.exited[:cnt[1]].clone(), out.counts.clone(), kv.core.clone()))
        return res

    _say(f"[gpu] no-alloc loop step: Ouro widths, 2 core layers, {n_big} then {n_small} rows")
    want = run(False)
    assert cdb.cdb_read_device_error(ws.buf) == 0
    got = run(True)
    assert int(d_err.item()) == 0
    for k, (a, b) in enumerate(zip(got, want)):
        for x, y in zip(a, b):
            assert torch.equal(x, y), f"call {k}"


def test_noalloc_refuses_rows_beyond_its_scratch():
    # d = 10240, d_ff = 32768: the workspace of 256 rows exceeds the 48 MiB scratch
    big = cdbgen.shrink(cdbgen.OURO, d=10240, n_heads=80, d_ff=32768, n_core=1)
    desc = cdb.make_desc(big)
    assert cdb.cdb_workspace_bytes(desc, 256) > 48 << 20
    dummy = torch.zeros(64, dtype=torch.int32, device="cuda")
    model = cdb.cdb_model(dummy.data_ptr(), desc)
    rows = cdb.cdb_rows(256, dummy.data_ptr(), dummy.data_ptr(), dummy.data_ptr(), dummy.data_ptr(),
                        dummy.data_ptr(), None)
    with pytest.raises(cdb.CdbError) as e:
        cdb.cdb_loop_step_noalloc(model, cdb.cdb_kv(), cdb.cdb_state(dummy.data_ptr(), None, 1), rows,
                                  cdb.cdb_step_out(), dummy)
    assert e.value.status == cdb.CDB_ERR_CAPACITY
