"""The C-ABI library: it loads, exports every symbol include/libcdb.h declares,
and rejects host-checkable bad arguments before enqueuing anything.  CPU only
(no call here reaches a kernel launch)."""
import ctypes as C
import os
import re

import pytest

import cdbgen
import paper_2608_09444_amd as cdb
from paper_2608_09444_amd import driver as cdb_driver

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions(header):
    text = open(os.path.join(ROOT, "include", header)).read()
    ret = r"(?:cdb_status|size_t|const char\*|int32_t|void|cdb_driver\*|const int32_t\*)"
    return sorted(set(re.findall(r"^\s*" + ret + r"\s+(cdb_\w+)\s*\(", text, re.M)))


def test_library_exports_every_declared_symbol():
    names = declared_functions("libcdb.h")
    assert len(names) == 14
    assert set(names) == set(cdb.EXPORTED)
    dnames = declared_functions("libcdb_driver.h")
    assert len(dnames) == 14
    assert set(dnames) == set(cdb_driver.EXPORTED)
    L = cdb.lib()
    for n in names + dnames:
        assert hasattr(L, n), n


@pytest.mark.parametrize("shape", [cdbgen.TINY, cdbgen.OURO, cdbgen.HUGINN], ids=lambda s: s.name)
def test_layout_sizes(shape):
    desc = cdb.make_desc(shape)
    nb = cdb.cdb_packed_weight_bytes(desc)
    pc = cdbgen.param_counts(shape)
    params = shape.n_layers * pc["per_layer"] + pc["embed"] + pc["lm_head"] + shape.d + \
        (2 * shape.d * shape.d if shape.injection else 0)
    assert 2 * params <= nb <= 2 * params + 256 * (4 * shape.n_layers + 8)
    ws = cdb.cdb_workspace_bytes(desc, 64)
    assert ws > 64 * shape.d * 4 * 3
    assert cdb.cdb_workspace_bytes(desc, cdb.MAX_PREFILL_ROWS) > cdb.cdb_workspace_bytes(desc, cdb.MAX_ROWS)
    assert cdb.cdb_workspace_bytes(desc, cdb.MAX_PREFILL_ROWS + 1) == 0


def test_unsupported_shapes_are_rejected():
    for kw in ({"head_dim": 80, "n_heads": 4, "d": 320}, {"d": 250}, {"vocab": 1000}):
        desc = cdb.make_desc(cdbgen.shrink(cdbgen.TINY, **kw))
        assert cdb.cdb_packed_weight_bytes(desc) == 0
        assert cdb.cdb_workspace_bytes(desc, 8) == 0


def test_host_checks_return_errors_without_launching():
    desc = cdb.make_desc(cdbgen.TINY)
    L = cdb.lib()
    model = cdb.cdb_model(None, desc)
    kv = cdb.cdb_kv()
    st = cdb.cdb_state()
    rows = cdb.cdb_rows()
    out = cdb.cdb_step_out()
    # null packed weights / workspace
    assert L.cdb_loop_step(C.byref(model), C.byref(kv), C.byref(st), C.byref(rows), C.byref(out), None, 0,
                           None) == cdb.CDB_ERR_INVALID_ARG
    # too many rows for one call
    model = cdb.cdb_model(1, desc)
    st = cdb.cdb_state(1, None, 4)
    rows = cdb.cdb_rows(cdb.MAX_ROWS + 1, 1, 1, 1, 1, 1)
    assert L.cdb_loop_step(C.byref(model), C.byref(kv), C.byref(st), C.byref(rows), C.byref(out), 1, 1 << 30,
                           None) == cdb.CDB_ERR_CAPACITY
    # workspace smaller than the rows need
    rows = cdb.cdb_rows(8, 1, 1, 1, 1, 1)
    assert L.cdb_boundary_coda(C.byref(model), C.byref(kv), C.byref(st), C.byref(rows), 1, 1, 1, 16,
                               None) == cdb.CDB_ERR_CAPACITY
    # unsupported descriptor
    bad = cdb.cdb_model(1, cdb.make_desc(cdbgen.shrink(cdbgen.TINY, head_dim=80, n_heads=4, d=320)))
    assert L.cdb_boundary_prelude(C.byref(bad), C.byref(kv), C.byref(st), C.byref(rows), 1, 1, 1 << 30,
                                  None) == cdb.CDB_ERR_UNSUPPORTED
    assert cdb.cdb_status_str(cdb.CDB_ERR_CAPACITY) == "capacity exceeded"


def test_workspace_size_covers_every_smaller_call():
    # a workspace sized for max_rows serves every call of fewer rows, although
    # the per-call layout is not monotonic (the tile GEMM's split-K factor
    # shrinks as its grid grows)
    for shape in (cdbgen.TINY, cdbgen.OURO, cdbgen.HUGINN):
        desc = cdb.make_desc(shape)
        sizes = [cdb.cdb_workspace_bytes(desc, r) for r in range(1, cdb.MAX_PREFILL_ROWS + 1)]
        assert all(b >= a for a, b in zip(sizes, sizes[1:])), shape.name
