"""ctypes binding of the CPU oracle (oracle/cdb_oracle.c).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the CPU-baseline leg of
the benchmark use it; the product path never imports it.  Floating point is
fp64 throughout; weights are the same bf16 bit patterns the device receives.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
LIB32_PATH = os.path.join(_HERE, "liboracle_acc32.so")
# fp32-accumulator builds that sum the projections' dot products in another
# order (reverse, blocks of 32): further fp32 realizations for tolerance sizing
LIB32_ORDER_PATHS = {1: os.path.join(_HERE, "liboracle_acc32_rev.so"),
                     2: os.path.join(_HERE, "liboracle_acc32_blk32.so")}
_SRC = os.path.join(_HERE, "cdb_oracle.c")

ORC_OK, ORC_ERR_ARG, ORC_ERR_UNMAPPED = 0, 1, 2


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain C, OpenMP over independent rows): the
    fp64 oracle, and the same source with fp32 accumulators (used only to size
    tolerances)."""
    builds = [(LIB_PATH, []), (LIB32_PATH, ["-DORC_ACC=float"])] + \
        [(p, ["-DORC_ACC=float", f"-DORC_SUM_ORDER={k}"]) for k, p in LIB32_ORDER_PATHS.items()]
    for path, extra in builds:
        if force or not os.path.exists(path):
            tmp = path + ".tmp"
            subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", *extra, "-o", tmp, _SRC,
                                   "-lm"])
            os.replace(tmp, path)
    return LIB_PATH


_libs = {}


def lib(acc32: bool = False, sum_order: int = 0):
    """The fp64 oracle, or with acc32 an fp32-accumulator build summing in
    sum_order (0 index order, 1 reverse, 2 blocks of 32)."""
    if sum_order and not acc32:
        raise ValueError("other summation orders exist only as fp32 builds")
    key = (bool(acc32), int(sum_order))
    if key not in _libs:
        path = LIB32_ORDER_PATHS[sum_order] if sum_order else (LIB32_PATH if acc32 else LIB_PATH)
        if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_SRC):
            build()
        L = C.CDLL(path)
        _declare(L)
        _libs[key] = L
    return _libs[key]


class OrcDesc(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("d", "n_heads", "head_dim", "d_ff", "vocab", "n_prelude", "n_core",
                                          "n_coda", "r_max", "injection", "exit_kind", "bf16_storage")] + \
               [("rms_eps", C.c_double), ("rope_base", C.c_double), ("kv_layout", C.c_int32)]

KV_FULL, KV_SHARED, KV_FIRST_THEN_SHARED = 0, 1, 2


class OrcWeights(C.Structure):
    _fields_ = [("embed", C.c_void_p), ("lm_head", C.c_void_p), ("w_exit", C.c_void_p), ("adapter", C.c_void_p),
                ("layer", C.POINTER(C.c_void_p))]


class OrcPaged(C.Structure):
    _fields_ = [("pre_pool", C.c_void_p), ("core_pool", C.c_void_p), ("coda_pool", C.c_void_p),
                ("pre_pages", C.c_int32), ("core_pages", C.c_int32), ("coda_pages", C.c_int32),
                ("page_table", C.c_void_p), ("max_seqs", C.c_int32), ("max_pages", C.c_int32),
                ("r_max", C.c_int32)]


_P = C.c_void_p
_I = C.c_int32


def _declare(L):
    L.orc_ref_sequence.argtypes = [_P, _P, _I, _P, _I, _I, _P, _P, _P, _P, _P]
    L.orc_brute_force.argtypes = [_P, _P, _I, _P, _I, _P, _P, _P, _P]
    L.orc_ref_sequence_gated.argtypes = [_P, _P, _I, _P, _I, _I, C.c_double, _I, _P, _P, _P, _P]
    L.orc_gate_decide.argtypes = [_P, _I, _P, _P, C.c_double, _I, _P, _P, _P]
    L.orc_prelude.argtypes = [_P, _P, _P, _P, _P, _I, _I, _P, _P, _P, _P]
    L.orc_loop_step.argtypes = [_P, _P, _P, _P, _P, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]
    L.orc_coda.argtypes = [_P, _P, _P, _P, _I, _I, _P, _P, _P, _P, _P]
    L.orc_exit_compact.argtypes = [_I, _P, _P, _I, _P, _P, _P, _P]
    L.orc_set_threads.argtypes = [_I]
    L.orc_set_threads.restype = _I
    L.orc_rmsnorm.argtypes = [_P, _I, C.c_double, _P]
    L.orc_rope.argtypes = [_P, _I, _I, _I, C.c_double]
    L.orc_attend.argtypes = [_P, _P, _P, _I, _I, _P]
    L.orc_silu.argtypes = [C.c_double]
    L.orc_silu.restype = C.c_double
    L.orc_to_bf16.argtypes = [C.c_double]
    L.orc_to_bf16.restype = C.c_double
    for f in ("orc_ref_sequence", "orc_ref_sequence_gated", "orc_gate_decide", "orc_brute_force", "orc_prelude",
              "orc_loop_step", "orc_coda",
              "orc_exit_compact"):
        getattr(L, f).restype = C.c_int


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


class Model:
    """Oracle model: a shape (cdbgen.ModelShape), bf16-bit weights, and the
    storage mode (bf16_storage=True rounds what the model keeps in bf16)."""

    def __init__(self, shape, weights: Dict[str, object], bf16_storage: bool = True, acc32: bool = False,
                 kv_layout: int = KV_FULL, sum_order: int = 0):
        """acc32: run the same steps with fp32 accumulators (tolerance sizing
        only), summing the projections in sum_order (0, 1 reverse, 2 blocks of 32).
        kv_layout: the core KV layout the dense references follow (the paged
        operators follow whatever the page table maps)."""
        self.shape = shape
        self.L = lib(acc32, sum_order)
        self.desc = OrcDesc(shape.d, shape.n_heads, shape.head_dim, shape.d_ff, shape.vocab, shape.n_prelude,
                            shape.n_core, shape.n_coda, shape.r_max, shape.injection, shape.exit_kind,
                            1 if bf16_storage else 0, shape.rms_eps, shape.rope_base, kv_layout)
        self._keep = []
        names = ("q", "k", "v", "o", "gate", "up", "down")
        ptrs = []
        for lw in weights["layers"]:
            for n in names:
                a = _c(lw[n], np.uint16)
                self._keep.append(a)
                ptrs.append(a.ctypes.data)
        self._layer_ptrs = (C.c_void_p * max(1, len(ptrs)))(*ptrs)
        tops = {}
        for n in ("embed", "lm_head", "w_exit", "adapter"):
            a = weights.get(n)
            if a is not None:
                a = _c(a, np.uint16)
                self._keep.append(a)
            tops[n] = _ptr(a)
        self.w = OrcWeights(tops["embed"], tops["lm_head"], tops["w_exit"], tops["adapter"],
                            C.cast(self._layer_ptrs, C.POINTER(C.c_void_p)))

    # -- dense references -------------------------------------------------
    def ref_sequence(self, tokens, depth, n_given: Optional[int] = None, want_kv: bool = False,
                     n_prefill: Optional[int] = None):
        """n_given: leading tokens taken as given (the rest are greedy);
        n_prefill: leading tokens run as one prefill block (default n_given)."""
        s = self.shape
        tok = _c(tokens, np.int32).copy()
        dep = _c(depth, np.int32)
        T = len(tok)
        n_given = T if n_given is None else n_given
        n_prefill = n_given if n_prefill is None else n_prefill
        logits = np.zeros((T, s.vocab))
        h = np.zeros((T, s.d))
        scores = np.zeros((T, s.r_max))
        kv = np.zeros((T, s.r_max, s.n_core, 2, s.d)) if want_kv else None
        rc = self.L.orc_ref_sequence(C.byref(self.desc), C.byref(self.w), T, _ptr(tok), n_given, n_prefill,
                                    _ptr(dep), _ptr(logits), _ptr(h), _ptr(scores), _ptr(kv))
        if rc != ORC_OK:
            raise ValueError(f"orc_ref_sequence: {rc}")
        return {"tokens": tok, "logits": logits, "h": h, "scores": scores, "core_kv": kv}

    def ref_sequence_gated(self, tokens, n_given: int, threshold: float, lookahead: bool,
                           n_prefill: Optional[int] = None):
        """Decode tokens take the depth the threshold rule gives on their own
        scores; the first n_prefill (default n_given) tokens are one prefill
        block at r_max."""
        s = self.shape
        tok = _c(tokens, np.int32).copy()
        T = len(tok)
        n_prefill = n_given if n_prefill is None else n_prefill
        logits = np.zeros((T, s.vocab))
        h = np.zeros((T, s.d))
        scores = np.zeros((T, s.r_max))
        depth = np.zeros(T, np.int32)
        rc = self.L.orc_ref_sequence_gated(C.byref(self.desc), C.byref(self.w), T, _ptr(tok), n_given, n_prefill,
                                          float(threshold), 1 if lookahead else 0, _ptr(depth), _ptr(logits),
                                          _ptr(h), _ptr(scores))
        if rc != ORC_OK:
            raise ValueError(f"orc_ref_sequence_gated: {rc}")
        return {"tokens": tok, "logits": logits, "h": h, "scores": scores, "depth": depth}

    def gate_decide(self, c, score, threshold: float, lookahead: bool, pending):
        """One loop step's threshold decisions (exit_mask, exit_next); pending
        (uint8 per row) is updated in place."""
        c = _c(c, np.int32)
        sc = _c(score, np.float64)
        assert pending.dtype == np.uint8 and pending.flags.c_contiguous
        n = len(c)
        mask = np.zeros(n, np.uint8)
        nxt = np.zeros(n, np.uint8)
        rc = self.L.orc_gate_decide(C.byref(self.desc), n, _ptr(c), _ptr(sc), float(threshold),
                                    1 if lookahead else 0, _ptr(pending), _ptr(mask), _ptr(nxt))
        if rc != ORC_OK:
            raise ValueError(f"orc_gate_decide: {rc}")
        return mask, nxt

    def brute_force(self, tokens, depth, n_prefill: Optional[int] = None):
        """n_prefill: leading tokens run as one prefill block (default all)."""
        s = self.shape
        tok = _c(tokens, np.int32)
        dep = _c(depth, np.int32)
        T = len(tok)
        n_prefill = T if n_prefill is None else n_prefill
        logits = np.zeros((T, s.vocab))
        h = np.zeros((T, s.d))
        scores = np.zeros((T, s.r_max))
        rc = self.L.orc_brute_force(C.byref(self.desc), C.byref(self.w), T, _ptr(tok), n_prefill, _ptr(dep),
                                   _ptr(logits), _ptr(h), _ptr(scores))
        if rc != ORC_OK:
            raise ValueError(f"orc_brute_force: {rc}")
        return {"logits": logits, "h": h, "scores": scores}


class Paged:
    """The oracle's own paged KV pools (fp64) and page table
    [max_seqs][r_max + 2][max_pages]; -1 marks an unmapped page."""

    PAGE = 16

    def __init__(self, shape, max_seqs: int, max_pages: int, pre_pages: int, core_pages: int, coda_pages: int):
        s = shape
        self.shape = s
        H, hd = s.n_heads, s.head_dim

        def pool(nl, n):
            return np.zeros((max(n, 1), max(nl, 1), 2, H, self.PAGE, hd))

        self.pre = pool(s.n_prelude, pre_pages)
        self.core = pool(s.n_core, core_pages)
        self.coda = pool(s.n_coda, coda_pages)
        self.page_table = np.full((max_seqs, s.r_max + 2, max_pages), -1, dtype=np.int32)
        self.c = OrcPaged(self.pre.ctypes.data, self.core.ctypes.data, self.coda.ctypes.data, pre_pages,
                          core_pages, coda_pages, self.page_table.ctypes.data, max_seqs, max_pages, s.r_max)

    def pool_of_plane(self, plane: int):
        if plane == 0:
            return self.pre
        if plane == self.shape.r_max + 1:
            return self.coda
        return self.core


def prelude(model: Model, paged: Paged, state_h, state_e, slot, seq, pos, tokens):
    n = len(slot)
    rc = model.L.orc_prelude(C.byref(model.desc), C.byref(model.w), C.byref(paged.c), _ptr(state_h),
                           _ptr(state_e), state_h.shape[0], n, _ptr(_c(slot, np.int32)), _ptr(_c(seq, np.int32)),
                           _ptr(_c(pos, np.int32)), _ptr(_c(tokens, np.int32)))
    if rc != ORC_OK:
        raise ValueError(f"orc_prelude: {rc}")


def loop_step(model: Model, paged: Paged, state_h, state_e, slot, seq, pos, c, depth):
    n = len(slot)
    score = np.zeros(n)
    mask = np.zeros(n, dtype=np.uint8)
    cont = np.zeros(max(n, 1), dtype=np.int32)
    exited = np.zeros(max(n, 1), dtype=np.int32)
    counts = np.zeros(2, dtype=np.int32)
    rc = model.L.orc_loop_step(C.byref(model.desc), C.byref(model.w), C.byref(paged.c), _ptr(state_h),
                             _ptr(state_e), state_h.shape[0], n, _ptr(_c(slot, np.int32)),
                             _ptr(_c(seq, np.int32)), _ptr(_c(pos, np.int32)), _ptr(_c(c, np.int32)),
                             _ptr(_c(depth, np.int32)), _ptr(score), _ptr(mask), _ptr(cont), _ptr(exited),
                             _ptr(counts))
    if rc != ORC_OK:
        raise ValueError(f"orc_loop_step: {rc}")
    return {"score": score, "exit_mask": mask, "cont": cont[:counts[0]].copy(),
            "exited": exited[:counts[1]].copy(), "counts": counts}


def coda(model: Model, paged: Paged, state_h, slot, seq, pos):
    n = len(slot)
    logits = np.zeros((n, model.shape.vocab))
    ids = np.zeros(max(n, 1), dtype=np.int32)
    rc = model.L.orc_coda(C.byref(model.desc), C.byref(model.w), C.byref(paged.c), _ptr(state_h), state_h.shape[0],
                        n, _ptr(_c(slot, np.int32)), _ptr(_c(seq, np.int32)), _ptr(_c(pos, np.int32)),
                        _ptr(logits), _ptr(ids))
    if rc != ORC_OK:
        raise ValueError(f"orc_coda: {rc}")
    return logits, ids[:n].copy()


def exit_compact(c, depth, r_max: int):
    c = _c(c, np.int32)
    depth = _c(depth, np.int32)
    n = len(c)
    mask = np.zeros(max(n, 1), dtype=np.uint8)
    cont = np.zeros(max(n, 1), dtype=np.int32)
    exited = np.zeros(max(n, 1), dtype=np.int32)
    counts = np.zeros(2, dtype=np.int32)
    rc = lib().orc_exit_compact(n, _ptr(c), _ptr(depth), r_max, _ptr(mask), _ptr(cont), _ptr(exited),
                                _ptr(counts))
    if rc != ORC_OK:
        raise ValueError(f"orc_exit_compact: {rc}")
    return {"exit_mask": mask[:n].copy(), "cont": cont[:counts[0]].copy(), "exited": exited[:counts[1]].copy(),
            "counts": counts}


# -- small pieces exported for closed-form pins ------------------------------

def rmsnorm(x, eps):
    x = _c(x, np.float64)
    y = np.zeros_like(x)
    lib().orc_rmsnorm(_ptr(x), len(x), eps, _ptr(y))
    return y


def rope(v, n_heads, hd, pos, base):
    v = _c(v, np.float64).copy()
    lib().orc_rope(_ptr(v), n_heads, hd, pos, base)
    return v


def attend(q, k, v):
    q = _c(q, np.float64)
    k = _c(k, np.float64)
    v = _c(v, np.float64)
    out = np.zeros(q.shape[0])
    lib().orc_attend(_ptr(q), _ptr(k), _ptr(v), k.shape[0], q.shape[0], _ptr(out))
    return out


def silu(x: float) -> float:
    return lib().orc_silu(x)


def to_bf16(x: float) -> float:
    return lib().orc_to_bf16(x)


def set_threads(n: int) -> int:
    """Threads of the oracle's OpenMP loops over rows (for timing runs)."""
    return int(lib().orc_set_threads(n))
