"""Python binding of the libcdb host driver (include/libcdb_driver.h): the
continuous-depth-batching scheduler (paper Section 4.1) and its runner.

Argument marshalling only; scheduling, page allocation and the stage calls run
in libcdb.so.
"""
from __future__ import annotations

import ctypes as C
from typing import Dict, List, Optional, Sequence

import numpy as np

from . import _ptr, _stream, cdb_kv, cdb_model, cdb_state, lib as _lib

EXPORTED = ("cdb_driver_create", "cdb_driver_destroy", "cdb_driver_add_sequence", "cdb_driver_add_request",
            "cdb_driver_page_table",
            "cdb_driver_next", "cdb_driver_complete", "cdb_driver_loop_result", "cdb_driver_set_time",
            "cdb_driver_get_stats",
            "cdb_driver_pages_in_use", "cdb_driver_latencies", "cdb_driver_scratch_bytes", "cdb_driver_run")

KV_FULL, KV_SHARED, KV_FIRST_THEN_SHARED = 0, 1, 2
TICK_NONE, TICK_PRELUDE_FIRST, TICK_LOOP, TICK_CODA, TICK_PREFILL = 0, 1, 2, 3, 4
MAX_ROWS = 256


class cdb_driver_config(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("max_batch", "max_active", "refill", "fixed_depth", "min_coda_batch",
                                          "r_max", "has_prelude", "has_coda", "max_seqs", "max_pages",
                                          "pre_pages", "core_pages", "coda_pages", "kv_layout", "gated",
                                          "lookahead")] + [("threshold", C.c_float), ("prefill_chunk", C.c_int32),
                                                           ("sync_steps", C.c_int32), ("boundary_stream", C.c_int32),
                                                           ("graph_loop", C.c_int32)]


class cdb_driver_tick(C.Structure):
    _fields_ = [("stage", C.c_int32), ("n_rows", C.c_int32), ("n_continue", C.c_int32)] + \
               [(n, C.c_int32 * MAX_ROWS) for n in ("slot", "seq", "pos", "c", "depth", "decode_index")] + \
               [("wait_until", C.c_double)]


class cdb_driver_stats(C.Structure):
    _fields_ = [(n, C.c_int64) for n in ("loop_steps", "loop_rows", "idle_rows", "coda_calls", "coda_rows",
                                          "prelude_calls", "prelude_rows", "tokens", "prefill_calls",
                                          "prefill_tokens", "host_wait_us", "pt_uploads", "pt_upload_bytes",
                                          "graph_launches")]


_bound = False


def lib() -> C.CDLL:
    global _bound
    L = _lib()
    if not _bound:
        P, I, S, D = C.c_void_p, C.c_int32, C.c_size_t, C.c_double
        L.cdb_driver_create.argtypes = [P]
        L.cdb_driver_create.restype = P
        L.cdb_driver_destroy.argtypes = [P]
        L.cdb_driver_destroy.restype = None
        L.cdb_driver_add_sequence.argtypes = [P, I, I, P, D]
        L.cdb_driver_add_request.argtypes = [P, I, P, I, P, D]
        L.cdb_driver_page_table.argtypes = [P]
        L.cdb_driver_page_table.restype = C.POINTER(C.c_int32)
        L.cdb_driver_next.argtypes = [P, P]
        L.cdb_driver_complete.argtypes = [P, P]
        L.cdb_driver_loop_result.argtypes = [P, P, P, P]
        L.cdb_driver_set_time.argtypes = [P, D]
        L.cdb_driver_set_time.restype = None
        L.cdb_driver_get_stats.argtypes = [P, P]
        L.cdb_driver_pages_in_use.argtypes = [P, P, P, P]
        L.cdb_driver_latencies.argtypes = [P, P, I]
        L.cdb_driver_scratch_bytes.argtypes = [P, I]
        L.cdb_driver_scratch_bytes.restype = S
        L.cdb_driver_run.argtypes = [P, P, P, P, P, S, P, P, I, P, S, P, P]
        for f in ("cdb_driver_add_sequence", "cdb_driver_add_request", "cdb_driver_next", "cdb_driver_complete",
                  "cdb_driver_loop_result", "cdb_driver_get_stats", "cdb_driver_pages_in_use",
                  "cdb_driver_latencies", "cdb_driver_run"):
            getattr(L, f).restype = C.c_int32
        _bound = True
    return L




class Driver:
    """One scheduler instance.  Sequences are added in arrival order; step()
    plans and applies calls without a device, run() executes them on it."""

    def __init__(self, max_batch: int, max_active: int, r_max: int, max_seqs: int, max_pages: int,
                 core_pages: int, pre_pages: int = 0, coda_pages: int = 0, has_prelude: bool = False,
                 has_coda: bool = False, refill: bool = True, fixed_depth: bool = False, min_coda_batch: int = 1,
                 kv_layout: int = KV_FULL, gated: bool = False, lookahead: bool = False, threshold: float = 0.0,
                 prefill_chunk: int = 0, sync_steps: bool = False, boundary_stream: int = 0,
                 graph_loop: bool = False):
        """boundary_stream: 1 or 2 puts prelude, coda and prefill on a second
        stream (libcdb_driver.h); run() then needs a workspace holding two
        (each half of ws).  graph_loop: loop steps replay one captured graph."""
        self.cfg = cdb_driver_config(max_batch, max_active, int(refill), int(fixed_depth), min_coda_batch, r_max,
                                     int(has_prelude), int(has_coda), max_seqs, max_pages, pre_pages, core_pages,
                                     coda_pages, kv_layout, int(gated), int(lookahead), threshold, prefill_chunk,
                                     int(sync_steps), int(boundary_stream), int(graph_loop))
        self.h = lib().cdb_driver_create(C.byref(self.cfg))
        if not self.h:
            raise ValueError("cdb_driver_create: invalid configuration")

    def __del__(self):
        h = getattr(self, "h", None)
        if h:
            lib().cdb_driver_destroy(h)
            self.h = None

    def add_sequence(self, prompt_len: int, depths: Optional[Sequence[int]], arrival: float = 0.0,
                     n_decode: Optional[int] = None) -> int:
        """depths: exit depth per decode input (None in gated mode, with n_decode)."""
        if depths is None:
            q = lib().cdb_driver_add_sequence(self.h, prompt_len, int(n_decode), None, arrival)
        else:
            dep = np.ascontiguousarray(depths, dtype=np.int32)
            q = lib().cdb_driver_add_sequence(self.h, prompt_len, len(dep), dep.ctypes.data, arrival)
        if q < 0:
            raise ValueError("cdb_driver_add_sequence: rejected")
        return q

    def add_request(self, prompt_ids: Sequence[int], depths: Optional[Sequence[int]], arrival: float = 0.0,
                    n_decode: Optional[int] = None) -> int:
        """A request whose prompt the driver prefills (prefill_chunk > 0)."""
        pr = np.ascontiguousarray(prompt_ids, dtype=np.int32)
        if depths is None:
            q = lib().cdb_driver_add_request(self.h, len(pr), pr.ctypes.data, int(n_decode), None, arrival)
        else:
            dep = np.ascontiguousarray(depths, dtype=np.int32)
            q = lib().cdb_driver_add_request(self.h, len(pr), pr.ctypes.data, len(dep), dep.ctypes.data, arrival)
        if q < 0:
            raise ValueError("cdb_driver_add_request: rejected")
        return q

    def page_table(self) -> np.ndarray:
        c = self.cfg
        n = c.max_seqs * (c.r_max + 2) * c.max_pages
        p = lib().cdb_driver_page_table(self.h)
        return np.ctypeslib.as_array(p, shape=(n,)).reshape(c.max_seqs, c.r_max + 2, c.max_pages).copy()

    def next(self) -> Optional[cdb_driver_tick]:
        """The next planned call, None when all work is done; a tick with stage
        TICK_NONE means nothing can run before tick.wait_until."""
        t = cdb_driver_tick()
        r = lib().cdb_driver_next(self.h, C.byref(t))
        return None if r == 0 else t

    def complete(self, t: cdb_driver_tick) -> int:
        return lib().cdb_driver_complete(self.h, C.byref(t))

    def loop_result(self, t: cdb_driver_tick, exit_mask, exit_next) -> int:
        m = np.ascontiguousarray(exit_mask, dtype=np.uint8)
        n = np.ascontiguousarray(exit_next, dtype=np.uint8)
        return lib().cdb_driver_loop_result(self.h, C.byref(t), m.ctypes.data, n.ctypes.data)

    def scratch_bytes(self, vocab: int) -> int:
        return lib().cdb_driver_scratch_bytes(self.h, vocab)

    def set_time(self, now: float):
        lib().cdb_driver_set_time(self.h, now)

    def stats(self) -> Dict[str, int]:
        s = cdb_driver_stats()
        lib().cdb_driver_get_stats(self.h, C.byref(s))
        return {n: int(getattr(s, n)) for n, _ in s._fields_}

    def pages_in_use(self) -> Dict[str, int]:
        a, b, c = C.c_int32(), C.c_int32(), C.c_int32()
        lib().cdb_driver_pages_in_use(self.h, C.byref(a), C.byref(b), C.byref(c))
        return {"pre": a.value, "core": b.value, "coda": c.value}

    def latencies(self, n: int) -> np.ndarray:
        out = np.zeros(n, dtype=np.float64)
        k = lib().cdb_driver_latencies(self.h, out.ctypes.data, n)
        return out[:k]

    def step(self) -> List[cdb_driver_tick]:
        """Plan and apply every call (no device); returns the ticks in order."""
        ticks = []
        while True:
            t = self.next()
            if t is None:
                return ticks
            if t.stage == TICK_NONE:
                self.set_time(t.wait_until)
                continue
            self.complete(t)
            ticks.append(t)

    def run(self, model: cdb_model, kv: cdb_kv, state: cdb_state, scratch, first_tokens, ws, tokens_out=None,
            stream=None) -> float:
        """Runs all added requests on the device; returns the wall time in
        seconds.  first_tokens: host ids per sequence, or None when every
        request was added with add_request.  tokens_out: optional device int32
        [max_seqs][stride]."""
        from . import CDB_OK, CdbError
        tok = None if first_tokens is None else np.ascontiguousarray(first_tokens, dtype=np.int32)
        secs = C.c_double()
        stride = 0 if tokens_out is None else int(tokens_out.shape[1])
        r = lib().cdb_driver_run(self.h, C.byref(model), C.byref(kv), C.byref(state), _ptr(scratch),
                                 scratch.numel() * scratch.element_size(), None if tok is None else tok.ctypes.data,
                                 _ptr(tokens_out), stride,
                                 _ptr(ws), ws.numel() * ws.element_size(), _stream(stream), C.byref(secs))
        if r != CDB_OK:
            raise CdbError("cdb_driver_run", r)
        return secs.value
