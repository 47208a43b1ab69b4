"""Python binding of libcdb (continuous depth batching on MI355X).

Argument marshalling only: every step of the stage calls runs in the HIP
kernels of libcdb.so.  PyTorch provides device memory and the stream.  The
library must have been built (``python -m paper_2608_09444_amd.build`` or
``__graft_entry__.build()``); importing this package without it raises.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcdb.so")

CDB_OK, CDB_ERR_INVALID_ARG, CDB_ERR_CAPACITY, CDB_ERR_HIP, CDB_ERR_UNSUPPORTED = range(5)
CDB_DEV_OK, CDB_DEV_UNMAPPED_PAGE, CDB_DEV_BAD_DEPTH, CDB_DEV_BAD_INDEX = range(4)
PAGE_TOKENS = 16
MAX_ROWS = 256
MAX_PREFILL_ROWS = 512

EXPORTED = ("cdb_packed_weight_bytes", "cdb_pack_weights", "cdb_kv_page_bytes", "cdb_workspace_bytes",
            "cdb_workspace_init", "cdb_boundary_prelude", "cdb_loop_step", "cdb_loop_step_gated", "cdb_boundary_coda",
            "cdb_prefill", "cdb_paged_attention", "cdb_read_device_error", "cdb_status_str", "cdb_loop_step_noalloc")


class CdbError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn}: {cdb_status_str(status)} ({status})")
        self.status = status


class cdb_model_desc(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("d", "n_heads", "head_dim", "d_ff", "vocab", "n_prelude", "n_core",
                                          "n_coda", "r_max", "injection", "exit_kind", "page_tokens")] + \
               [("rms_eps", C.c_float), ("rope_base", C.c_float)]


class cdb_plain_weights(C.Structure):
    _fields_ = [("embed", C.c_void_p), ("lm_head", C.c_void_p), ("w_exit", C.c_void_p), ("adapter", C.c_void_p),
                ("layer", C.POINTER(C.c_void_p))]


class cdb_model(C.Structure):
    _fields_ = [("packed", C.c_void_p), ("desc", cdb_model_desc)]


class cdb_kv(C.Structure):
    _fields_ = [("pre_pool", C.c_void_p), ("core_pool", C.c_void_p), ("coda_pool", C.c_void_p),
                ("pre_pages", C.c_int32), ("core_pages", C.c_int32), ("coda_pages", C.c_int32),
                ("page_table", C.c_void_p), ("max_seqs", C.c_int32), ("max_pages", C.c_int32)]


class cdb_state(C.Structure):
    _fields_ = [("h", C.c_void_p), ("e", C.c_void_p), ("n_slots", C.c_int32)]


class cdb_rows(C.Structure):
    _fields_ = [("n_rows", C.c_int32), ("slot", C.c_void_p), ("seq", C.c_void_p), ("pos", C.c_void_p),
                ("c", C.c_void_p), ("depth", C.c_void_p), ("d_n_rows", C.c_void_p)]


class cdb_step_out(C.Structure):
    _fields_ = [("exit_score", C.c_void_p), ("exit_mask", C.c_void_p), ("cont", C.c_void_p),
                ("exited", C.c_void_p), ("counts", C.c_void_p), ("exit_next", C.c_void_p)]


class cdb_gate(C.Structure):
    _fields_ = [("threshold", C.c_float), ("lookahead", C.c_int32), ("pending", C.c_void_p)]


_lib = None


def lib() -> C.CDLL:
    """The loaded libcdb.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"libcdb.so not built at {LIB_PATH}; run __graft_entry__.build()")
        L = C.CDLL(LIB_PATH)
        P, I, S = C.c_void_p, C.c_int32, C.c_size_t
        L.cdb_packed_weight_bytes.argtypes = [P]
        L.cdb_packed_weight_bytes.restype = S
        L.cdb_pack_weights.argtypes = [P, P, P, S, P]
        L.cdb_kv_page_bytes.argtypes = [P, I]
        L.cdb_kv_page_bytes.restype = S
        L.cdb_workspace_bytes.argtypes = [P, I]
        L.cdb_workspace_bytes.restype = S
        L.cdb_workspace_init.argtypes = [P, S, P]
        L.cdb_boundary_prelude.argtypes = [P, P, P, P, P, P, S, P]
        L.cdb_loop_step.argtypes = [P, P, P, P, P, P, S, P]
        L.cdb_loop_step_gated.argtypes = [P, P, P, P, P, P, P, S, P]
        L.cdb_loop_step_noalloc.argtypes = [P, P, P, P, P, P, P]
        L.cdb_boundary_coda.argtypes = [P, P, P, P, P, P, P, S, P]
        L.cdb_paged_attention.argtypes = [P, P, P, I, I, P, P, P, P, S, P]
        L.cdb_prefill.argtypes = [P, P, I, I, I, P, P, P, P, S, P]
        L.cdb_read_device_error.argtypes = [P, P, P]
        L.cdb_status_str.argtypes = [C.c_int]
        L.cdb_status_str.restype = C.c_char_p
        for f in ("cdb_pack_weights", "cdb_workspace_init", "cdb_boundary_prelude", "cdb_loop_step", "cdb_loop_step_gated",
                  "cdb_boundary_coda", "cdb_paged_attention", "cdb_prefill", "cdb_read_device_error",
                  "cdb_loop_step_noalloc"):
            getattr(L, f).restype = C.c_int
        _lib = L
    return _lib


def cdb_status_str(status: int) -> str:
    return lib().cdb_status_str(status).decode()


def _check(fn: str, status: int):
    if status != CDB_OK:
        raise CdbError(fn, status)


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def make_desc(shape) -> cdb_model_desc:
    """Descriptor from any object with the model-shape attributes."""
    return cdb_model_desc(shape.d, shape.n_heads, shape.head_dim, shape.d_ff, shape.vocab, shape.n_prelude,
                          shape.n_core, shape.n_coda, shape.r_max, shape.injection, shape.exit_kind, PAGE_TOKENS,
                          shape.rms_eps, shape.rope_base)


# ---------------------------------------------------------------- C ABI, same names

def cdb_packed_weight_bytes(desc: cdb_model_desc) -> int:
    return lib().cdb_packed_weight_bytes(C.byref(desc))


def cdb_pack_weights(desc: cdb_model_desc, w: cdb_plain_weights, packed, stream=None):
    _check("cdb_pack_weights", lib().cdb_pack_weights(C.byref(desc), C.byref(w), _ptr(packed),
                                                      packed.numel() * packed.element_size(), _stream(stream)))


def cdb_kv_page_bytes(desc: cdb_model_desc, stage: int) -> int:
    return lib().cdb_kv_page_bytes(C.byref(desc), stage)


def cdb_workspace_bytes(desc: cdb_model_desc, max_rows: int) -> int:
    return lib().cdb_workspace_bytes(C.byref(desc), max_rows)


def cdb_workspace_init(ws, stream=None):
    _check("cdb_workspace_init", lib().cdb_workspace_init(_ptr(ws), ws.numel(), _stream(stream)))


def cdb_boundary_prelude(model: cdb_model, kv: cdb_kv, state: cdb_state, rows: cdb_rows, tokens, ws, stream=None):
    _check("cdb_boundary_prelude", lib().cdb_boundary_prelude(C.byref(model), C.byref(kv), C.byref(state),
                                                              C.byref(rows), _ptr(tokens), _ptr(ws), ws.numel(),
                                                              _stream(stream)))


def cdb_loop_step(model: cdb_model, kv: cdb_kv, state: cdb_state, rows: cdb_rows, out: cdb_step_out, ws,
                  stream=None):
    _check("cdb_loop_step", lib().cdb_loop_step(C.byref(model), C.byref(kv), C.byref(state), C.byref(rows),
                                                C.byref(out), _ptr(ws), ws.numel(), _stream(stream)))


def cdb_loop_step_gated(model: cdb_model, kv: cdb_kv, state: cdb_state, rows: cdb_rows, gate: cdb_gate,
                        out: cdb_step_out, ws, stream=None):
    _check("cdb_loop_step_gated", lib().cdb_loop_step_gated(C.byref(model), C.byref(kv), C.byref(state),
                                                            C.byref(rows), C.byref(gate), C.byref(out), _ptr(ws),
                                                            ws.numel(), _stream(stream)))


def cdb_loop_step_noalloc(model: cdb_model, kv: cdb_kv, state: cdb_state, rows: cdb_rows, out: cdb_step_out,
                          d_error, stream=None):
    """d_error: device int32 tensor of one element (zeroed by the caller)."""
    _check("cdb_loop_step_noalloc", lib().cdb_loop_step_noalloc(C.byref(model), C.byref(kv), C.byref(state),
                                                                C.byref(rows), C.byref(out), _ptr(d_error),
                                                                _stream(stream)))


def cdb_boundary_coda(model: cdb_model, kv: cdb_kv, state: cdb_state, rows: cdb_rows, logits, next_ids, ws,
                      stream=None):
    _check("cdb_boundary_coda", lib().cdb_boundary_coda(C.byref(model), C.byref(kv), C.byref(state), C.byref(rows),
                                                        _ptr(logits), _ptr(next_ids), _ptr(ws), ws.numel(),
                                                        _stream(stream)))


def cdb_prefill(model: cdb_model, kv: cdb_kv, seq: int, pos0: int, tokens, logits, next_ids, ws, stream=None):
    """tokens: device int32 [n]; logits: device fp32 [n][vocab], or None (only the
    last row's greedy id, into next_ids[0]); next_ids: device int32 [n] (or [1])."""
    n = int(tokens.numel())
    _check("cdb_prefill", lib().cdb_prefill(C.byref(model), C.byref(kv), seq, pos0, n, _ptr(tokens), _ptr(logits),
                                            _ptr(next_ids), _ptr(ws), ws.numel(), _stream(stream)))


def cdb_paged_attention(desc: cdb_model_desc, kv: cdb_kv, rows: cdb_rows, stage: int, layer: int, q, out, ws,
                        stream=None, order=None):
    """order: None (computed into ws[256:]) or an int32 device tensor / address of a
    previous call's order."""
    optr = order if isinstance(order, int) else _ptr(order)
    _check("cdb_paged_attention", lib().cdb_paged_attention(C.byref(desc), C.byref(kv), C.byref(rows), stage, layer,
                                                            _ptr(q), optr, _ptr(out), _ptr(ws), ws.numel(),
                                                            _stream(stream)))


def cdb_read_device_error(ws, stream=None) -> int:
    code = C.c_int32(0)
    _check("cdb_read_device_error", lib().cdb_read_device_error(_ptr(ws), _stream(stream), C.byref(code)))
    return code.value


# ---------------------------------------------------------------- device-memory holders (torch)

def _bf16_tensor(bits, device):
    """A numpy uint16 (bf16 bit pattern) array as a device bf16 tensor."""
    import numpy as np
    import torch
    a = np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16)
    return torch.from_numpy(a).to(device).view(torch.bfloat16)


class DeviceModel:
    """Packed weights of one model on the device (plain weights are uploaded,
    packed by cdb_pack_weights, then released)."""

    def __init__(self, shape, weights, device="cuda", stream=None):
        import torch
        self.shape = shape
        self.desc = make_desc(shape)
        nbytes = cdb_packed_weight_bytes(self.desc)
        if nbytes == 0:
            raise CdbError("cdb_packed_weight_bytes", CDB_ERR_UNSUPPORTED)
        self.packed = torch.empty(nbytes, dtype=torch.uint8, device=device)
        self._pack_from(weights, device, stream)
        self.model = cdb_model(self.packed.data_ptr(), self.desc)

    def _pack_from(self, w, device, stream):
        import torch
        names = ("q", "k", "v", "o", "gate", "up", "down")
        keep = []
        ptrs = []
        # upload and pack layer by layer to bound the plain-weight footprint
        tops = {k: (_bf16_tensor(w[k], device) if w.get(k) is not None else None)
                for k in ("embed", "lm_head", "w_exit", "adapter")}
        for lw in w["layers"]:
            for n in names:
                t = _bf16_tensor(lw[n], device)
                keep.append(t)
                ptrs.append(t.data_ptr())
        arr = (C.c_void_p * max(1, len(ptrs)))(*ptrs)
        pw = cdb_plain_weights(_ptr(tops["embed"]), _ptr(tops["lm_head"]), _ptr(tops["w_exit"]),
                               _ptr(tops["adapter"]), C.cast(arr, C.POINTER(C.c_void_p)))
        cdb_pack_weights(self.desc, pw, self.packed, stream)
        torch.cuda.current_stream().synchronize() if stream is None else stream.synchronize()
        del keep, tops


class PagedKV:
    """Device KV pools (bf16, layer-major [layers][pages][2][H][16][hd] per stage)
    and the int32 page table [max_seqs][r_max + 2][max_pages] (-1 = unmapped)."""

    def __init__(self, shape, max_seqs, max_pages, pre_pages, core_pages, coda_pages, device="cuda", fill=None):
        import torch
        s = shape
        H, hd = s.n_heads, s.head_dim

        def pool(nl, n):
            if nl == 0 or n == 0:
                return torch.zeros(1, dtype=torch.bfloat16, device=device)
            t = torch.empty((nl, n, 2, H, PAGE_TOKENS, hd), dtype=torch.bfloat16, device=device)
            if fill is None:
                t.zero_()
            return t

        self.shape = s
        self.pre, self.core, self.coda = pool(s.n_prelude, pre_pages), pool(s.n_core, core_pages), \
            pool(s.n_coda, coda_pages)
        self.page_table = torch.full((max_seqs, s.r_max + 2, max_pages), -1, dtype=torch.int32, device=device)
        self.c = cdb_kv(self.pre.data_ptr(), self.core.data_ptr(), self.coda.data_ptr(),
                        pre_pages if s.n_prelude else 0, core_pages, coda_pages if s.n_coda else 0,
                        self.page_table.data_ptr(), max_seqs, max_pages)


class State:
    def __init__(self, shape, n_slots, device="cuda"):
        import torch
        self.h = torch.zeros((n_slots, shape.d), dtype=torch.float32, device=device)
        self.e = torch.zeros((n_slots, shape.d), dtype=torch.float32, device=device) if shape.injection else None
        self.c = cdb_state(self.h.data_ptr(), _ptr(self.e), n_slots)


class Workspace:
    def __init__(self, desc: cdb_model_desc, max_rows: int, device="cuda", stream=None):
        import torch
        n = cdb_workspace_bytes(desc, max_rows)
        if n == 0:
            raise CdbError("cdb_workspace_bytes", CDB_ERR_CAPACITY)
        self.buf = torch.empty(n, dtype=torch.uint8, device=device)
        cdb_workspace_init(self.buf, stream)


class Rows:
    """Device row arrays for one stage call.  d_n_rows: optional device int32
    tensor holding the live row count (the arrays' length is then the
    capacity)."""

    def __init__(self, slot, seq, pos, c=None, depth=None, device="cuda", d_n_rows=None):
        import torch

        def dev(a):
            if a is None:
                return None
            return torch.as_tensor(a, dtype=torch.int32).to(device).contiguous()

        self.slot, self.seq, self.pos, self.cc, self.depth = dev(slot), dev(seq), dev(pos), dev(c), dev(depth)
        self.d_n_rows = d_n_rows
        self.n = int(self.slot.numel())
        self.c = cdb_rows(self.n, _ptr(self.slot), _ptr(self.seq), _ptr(self.pos), _ptr(self.cc), _ptr(self.depth),
                          _ptr(d_n_rows))


class StepOut:
    def __init__(self, n, device="cuda"):
        import torch
        m = max(n, 1)
        self.score = torch.zeros(m, dtype=torch.float32, device=device)
        self.mask = torch.zeros(m, dtype=torch.uint8, device=device)
        self.cont = torch.zeros(m, dtype=torch.int32, device=device)
        self.exited = torch.zeros(m, dtype=torch.int32, device=device)
        self.counts = torch.zeros(2, dtype=torch.int32, device=device)
        self.exit_next = torch.zeros(m, dtype=torch.uint8, device=device)
        self.c = cdb_step_out(self.score.data_ptr(), self.mask.data_ptr(), self.cont.data_ptr(),
                              self.exited.data_ptr(), self.counts.data_ptr(), self.exit_next.data_ptr())


class Gate:
    """Threshold exits (cdb_gate) with the per-slot lookahead flags on the device."""

    def __init__(self, threshold: float, lookahead: bool, n_slots: int, device="cuda"):
        import torch
        self.pending = torch.zeros(max(n_slots, 1), dtype=torch.uint8, device=device)
        self.c = cdb_gate(threshold, 1 if lookahead else 0, self.pending.data_ptr())
