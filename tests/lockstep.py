"""Drives the HIP stage calls and the CPU oracle side by side on identical row
batches, so every call's outputs can be compared.  Used by the GPU parity tests.

The schedule and the oracle's side live in oracle_side (refill policy; decode
inputs teacher-forced with the oracle's greedy ids).

Bounds.  Integer outputs are compared exactly.  Hidden states, exit scores and
logits must lie within max-abs 2e-2 / mean-abs 2e-3, or, where the oracle's own
arithmetic cannot be reproduced that closely, within DRIFT_FACTOR times the
largest distance of fp32-level realizations of the oracle from the fp64 oracle
(same steps with fp32 accumulators; the state rounded to fp32; fp32-sized noise
on the state).  A random-init core turns any rounding-level difference into
bf16 rounding flips that cascade layer after layer, so no fp32 implementation
sits closer to the fp64 oracle than these realizations do.  The realizations
are run per call from the oracle's state (`sensitivity`), or taken from a stored
envelope of a free-running run (`envelope`).  Relative errors
||got - want||_2 / ||want||_2 per row are recorded next to the absolute ones.
"""
from __future__ import annotations

from typing import Dict, List

import numpy as np
import torch

import cdbgen
import oracle
import paper_2608_09444_amd as cdb
from oracle_side import OracleSide, row_rel, run_schedule

PAGE = 16
TOL_MAX, TOL_MEAN = 2e-2, 2e-3
DRIFT_FACTOR = 1.25


def bf16_pool_to_f64(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


class Lockstep:
    def __init__(self, shape, weights, seq_lens: List[int], max_batch: int, bf16_storage: bool = True,
                 extra_pages: int = 0, resync: bool = False, sensitivity: bool = False, kv_layout: int = 0,
                 gate=None, envelope=None):
        """resync: after every call, copy the oracle's states and newly written
        K/V entries into the device buffers, so that each call is checked from
        identical inputs.  sensitivity: bound each call by fp32-level
        realizations of the oracle run from the oracle's state before the call.
        envelope: a stored free-running drift envelope (tests/golden/drift_*.json)
        whose per-call distances bound the calls of a free-running run in order.
        kv_layout: 0 full, 1 single shared slot, 2 first-then-shared (core planes
        aliased in the page table).  gate: (threshold, lookahead) for threshold
        exits decided on the device (lookahead only: each step's exits are fixed
        by the previous step, so both sides run the same rows); the loop-step
        depths are then ignored."""
        self.resync = resync
        self.sensitivity = sensitivity
        self.envelope = envelope["calls"] if envelope else None
        # free-running envelopes: how far one of the oracle's realizations exceeds
        # the largest of the others (per output kind), for the report
        self.spread = envelope.get("spread", {}) if envelope else {}
        self.rec = None  # this call's envelope record (free-running runs)
        self.single_row = {"calls": 0, "max_ratio": 0.0}
        self.tol = (TOL_MAX, TOL_MEAN)
        self.score_tol = TOL_MAX
        self.w_exit = (np.asarray(weights["w_exit"], np.uint16).astype(np.uint32) << 16).view(np.float32).astype(
            np.float64)
        self.self_diff = {"max": 0.0, "mean": 0.0}
        self.s = s = shape
        self.R = s.r_max
        self.max_batch = max_batch
        self.o = OracleSide(s, weights, seq_lens, kv_layout=kv_layout, extra_pages=extra_pages,
                            bf16_storage=bf16_storage)
        self.om, self.op, self.oh, self.oe, self.base = self.o.om, self.o.op, self.o.oh, self.o.oe, self.o.base
        self.om32 = oracle.Model(s, weights, bf16_storage=bf16_storage, acc32=True) if sensitivity else None
        self.gm = cdb.DeviceModel(s, weights)
        n_seq = len(seq_lens)
        self.max_pages = self.o.max_pages
        self.gkv = cdb.PagedKV(s, n_seq, self.max_pages, *self.o.pages)
        self.gkv.page_table.copy_(torch.from_numpy(self.op.page_table))
        n_slots = int(self.base[-1])
        self.gstate = cdb.State(s, n_slots)
        self.ws = cdb.Workspace(self.gm.desc, max(max_batch, max(seq_lens)))
        self.errors: Dict[str, float] = {"h_max": 0.0, "h_mean": 0.0, "h_rel": 0.0, "logit_max": 0.0,
                                         "logit_mean": 0.0, "logit_rel": 0.0, "kv_max": 0.0, "score_max": 0.0}
        # the largest error of each kind relative to its call's bound
        self.ratio: Dict[str, float] = {}
        self.calls = {"prelude": 0, "loop": 0, "coda": 0}
        self.n_calls = 0
        self.argmax_checked = 0
        self.gate = gate
        if gate is not None:
            assert gate[1], "the lockstep gate runs with lookahead"
            self.ggate = cdb.Gate(gate[0], True, n_slots)
            self.opending = np.zeros(n_slots, np.uint8)
            self.gate_stats = {"decisions": 0, "near_threshold": 0, "overridden": 0, "exits_before_r_max": 0}
        # mean-abs bookkeeping per output kind over the whole run: sum of |error|,
        # element count, and the per-call mean bound weighted by elements
        self.run_sums: Dict[str, List[float]] = {}

    # -------------------------------------------------------------- compare helpers
    def _cmp(self, key_max, key_mean, got, want, what, key_rel=None):
        """max-abs is checked per call; mean-abs is a statistic of the whole
        result, checked over the run by check_means() (a call of two rows is
        dominated by single bf16 rounding flips).  In a free-running run a call
        of one row is bounded instead by the row's relative L2 error and its
        mean-abs error, each at DRIFT_FACTOR times the realizations': the largest
        of one row's d errors is too heavy-tailed a statistic for a sample of
        realizations to bound (its ratio to that bound is reported)."""
        d = np.abs(np.asarray(got, np.float64) - want)
        mx, mn = float(d.max()) if d.size else 0.0, float(d.mean()) if d.size else 0.0
        self.errors[key_max] = max(self.errors[key_max], mx)
        rel = row_rel(got, want) if key_rel else 0.0
        if key_rel:
            self.errors[key_rel] = max(self.errors[key_rel], rel)
        one_row = self.rec is not None and np.atleast_2d(want).shape[0] == 1 and key_rel is not None
        if one_row:
            self.single_row["calls"] += 1
            self.single_row["max_ratio"] = max(self.single_row["max_ratio"], mx / self.tol[0])
            rb = max(DRIFT_FACTOR * self.rec[key_rel], 1e-12)
            self.ratio[key_rel] = max(self.ratio.get(key_rel, 0.0), rel / rb)
            assert rel <= rb and mn <= self.tol[1], \
                f"{what} (one row): rel {rel:.3e} (bound {rb:.3e}), mean abs {mn:.3e} (bound {self.tol[1]:.3e})"
        else:
            self.ratio[key_max] = max(self.ratio.get(key_max, 0.0), mx / self.tol[0])
        if key_mean:
            self.errors[key_mean] = max(self.errors[key_mean], mn)
            acc = self.run_sums.setdefault(key_mean, [0.0, 0, 0.0])
            acc[0] += float(d.sum())
            acc[1] += d.size
            acc[2] += self.tol[1] * d.size
        tmax = self.tol[0]
        assert one_row or mx <= tmax, f"{what}: max abs {mx:.3e}, mean abs {mn:.3e} (max bound {tmax:.3e})"

    def check_means(self):
        """Mean-abs error of each output kind over the run against the
        element-weighted mean of the per-call bounds."""
        for key, (tot, n, bound) in self.run_sums.items():
            if n:
                self.ratio[key] = (tot / n) / (bound / n)
                assert tot / n <= bound / n, f"{key}: run mean abs {tot / n:.3e} > bound {bound / n:.3e}"

    def _oracle_bound(self, run32, out_of):
        """Run the call through several fp32-level realizations of the oracle's
        arithmetic on copies of the oracle's buffers, restoring them after each:
        the same steps with fp32 accumulators; the fp64 steps from the residual
        state rounded to fp32 (as the device keeps it); and the fp64 steps from
        the state under two draws of fp32-sized relative noise.  This call's
        bound is the larger of the absolute tolerance and DRIFT_FACTOR times the
        largest distance of any of them from the oracle's own outputs (in a call
        of a few rows the error is set by a handful of bf16 rounding flips, which
        one realization undersamples).  `out_of(result)` picks the compared output."""
        self.tol = (TOL_MAX, TOL_MEAN)
        if not self.sensitivity:
            return None
        bufs = [self.oh, self.op.pre, self.op.core, self.op.coda] + ([self.oe] if self.oe is not None else [])
        saved = [a.copy() for a in bufs]

        def restore():
            for a, b in zip(bufs, saved):
                a[...] = b

        got = [out_of(run32(self.om32))]
        restore()
        rng = np.random.default_rng(1000 + sum(self.calls.values()))
        for k in range(3):
            for a in ([self.oh] + ([self.oe] if self.oe is not None else [])):
                if k == 0:
                    a[...] = a.astype(np.float32)
                else:
                    a *= 1.0 + 2.0 ** -24 * rng.standard_normal(a.shape)
            got.append(out_of(run32(self.om)))
            restore()
        return got

    def _set_bound(self, variants, got64, stage):
        """This call's (max, mean) bound: the absolute tolerance, widened to
        DRIFT_FACTOR times the realizations' distance from the oracle, either
        run now (variants) or stored for this call of a free-running run."""
        k = self.n_calls
        self.n_calls += 1
        mx = mn = None
        if variants is not None:
            mx = max(float(np.abs(v - got64).max()) for v in variants)
            mn = max(float(np.abs(v - got64).mean()) for v in variants)
        self.rec = None
        if variants is None and self.envelope is not None:
            rec = self.rec = self.envelope[k]
            assert rec["stage"] == stage and rec["rows"] == len(got64), (k, rec, stage, len(got64))
            key = "logit" if stage == "coda" else "h"
            mx, mn = rec[key + "_max"], rec[key + "_mean"]
            if stage == "loop":
                self.score_tol = max(TOL_MAX, DRIFT_FACTOR * rec["score_max"])
        if mx is None:
            return
        self.self_diff["max"] = max(self.self_diff["max"], mx)
        self.self_diff["mean"] = max(self.self_diff["mean"], mn)
        self.tol = (max(TOL_MAX, DRIFT_FACTOR * mx), max(TOL_MEAN, DRIFT_FACTOR * mn))

    def _cmp_state(self, slots, what):
        idx = torch.as_tensor(slots, dtype=torch.long, device="cuda")
        g = self.gstate.h[idx].cpu().numpy()
        self._cmp("h_max", "h_mean", g, self.oh[slots], what, key_rel="h_rel")
        if self.resync:
            self.gstate.h[idx] = torch.from_numpy(self.oh[slots].astype(np.float32)).to("cuda")
            if self.oe is not None:
                self.gstate.e[idx] = torch.from_numpy(self.oe[slots].astype(np.float32)).to("cuda")

    def _cmp_kv(self, seqs, poss, planes, what):
        """K/V entries of (seq, pos) in each listed plane, every layer of that stage."""
        for q, t in zip(seqs, poss):
            for plane in planes:
                pid = int(self.op.page_table[q, plane, t // PAGE])
                if plane == 0:
                    gp, opool = self.gkv.pre, self.op.pre
                elif plane == self.R + 1:
                    gp, opool = self.gkv.coda, self.op.coda
                else:
                    gp, opool = self.gkv.core, self.op.core
                g = gp[:, pid, :, :, t % PAGE, :].float().cpu().numpy()  # device pools are layer-major
                o = opool[pid, :, :, :, t % PAGE, :]
                d = np.abs(g - o)
                self.errors["kv_max"] = max(self.errors["kv_max"], float(d.max()))
                # bf16 entries: at most one bf16 step apart (2^-7 relative), or the absolute bound
                bad = d > np.maximum(self.tol[0], np.abs(o) * 2.0 ** -7 * 1.001)
                assert not bad.any() and float(d.mean()) <= self.tol[1], \
                    f"{what}: kv plane {plane} seq {q} pos {t}: max {d.max():.3e} mean {d.mean():.3e}"
                if self.resync:  # oracle entries are bf16 values in bf16-storage mode
                    gp[:, pid, :, :, t % PAGE, :] = torch.from_numpy(o.astype(np.float32)).to("cuda").to(torch.bfloat16)

    # -------------------------------------------------------------- stages
    def prelude(self, seqs, poss, toks):
        slots = self.o.slots(seqs, poss)
        g32 = self._oracle_bound(lambda m: oracle.prelude(m, self.op, self.oh, self.oe, slots, seqs, poss, toks),
                                 lambda _: self.oh[slots].copy())
        self.o.prelude(seqs, poss, toks)
        self._set_bound(g32, self.oh[slots], "prelude")
        rows = cdb.Rows(slots, seqs, poss)
        cdb.cdb_boundary_prelude(self.gm.model, self.gkv.c, self.gstate.c, rows.c,
                                 torch.as_tensor(toks, dtype=torch.int32, device="cuda"), self.ws.buf)
        torch.cuda.synchronize()
        self.calls["prelude"] += 1
        self._cmp_state(slots, "prelude state")
        if self.s.n_prelude:
            self._cmp_kv(seqs, poss, [0], "prelude kv")

    def loop(self, seqs, poss, cs, deps, replay=False):
        """replay: run the given depths even in gated mode (prompt tokens run r_max loops)."""
        slots = self.o.slots(seqs, poss)
        gated = self.gate is not None and not replay
        if gated:
            # this step's exits were decided by the previous one (or loop r_max)
            pend = self.opending[slots].copy()
            exit_now = (pend != 0) | (cs + 1 == self.R)
            deps = np.where(exit_now, cs + 1, self.R).astype(np.int32)
        # states before the call on both sides (the exit score of the
        # convergence criterion is a distance from them)
        idx = torch.as_tensor(slots, dtype=torch.long, device="cuda")
        o_in = self.oh[slots].copy()
        g_in = self.gstate.h[idx].double().cpu().numpy()
        # each realization gives its states and its exit scores: the score takes
        # its own bound from the realizations' scores
        g32 = self._oracle_bound(lambda m: oracle.loop_step(m, self.op, self.oh, self.oe, slots, seqs, poss, cs, deps),
                                 lambda r: (self.oh[slots].copy(), np.array(r["score"], np.float64)))
        o = self.o.loop(seqs, poss, cs, deps)
        self.score_tol = TOL_MAX
        if g32 is not None:
            dscore = max(float(np.abs(sc - o["score"]).max()) for _, sc in g32)
            self.score_tol = max(TOL_MAX, DRIFT_FACTOR * dscore)
            g32 = [h for h, _ in g32]
        self._set_bound(g32, self.oh[slots], "loop")
        rows = cdb.Rows(slots, seqs, poss, cs, None if gated else deps)
        out = cdb.StepOut(len(seqs))
        if gated:
            cdb.cdb_loop_step_gated(self.gm.model, self.gkv.c, self.gstate.c, rows.c, self.ggate.c, out.c,
                                    self.ws.buf)
        else:
            cdb.cdb_loop_step(self.gm.model, self.gkv.c, self.gstate.c, rows.c, out.c, self.ws.buf)
        torch.cuda.synchronize()
        self.calls["loop"] += 1
        n = len(seqs)
        cnt = out.counts.cpu().numpy()
        assert cnt.tolist() == o["counts"].tolist(), (cnt, o["counts"])
        assert out.mask[:n].cpu().numpy().tolist() == o["exit_mask"].tolist()
        assert out.cont[:cnt[0]].cpu().numpy().tolist() == o["cont"].tolist()
        assert out.exited[:cnt[1]].cpu().numpy().tolist() == o["exited"].tolist()
        g_out = self.gstate.h[idx].double().cpu().numpy()
        o_out = self.oh[slots].copy()
        self._cmp_state(slots, "loop-step state")
        sc = out.score[:n].cpu().numpy().astype(np.float64)
        # the device's score is the exit signal of the device's own states
        own = self._exit_signal(g_out, g_in)
        assert (np.abs(sc - own) <= 1e-4 + 1e-5 * np.abs(own)).all(), \
            f"exit score against the device's own states: {np.abs(sc - own).max():.3e}"
        # against the oracle: the realizations' score drift; for the convergence
        # distance ||h - h_in||_2 also what the state differences on both sides
        # allow (triangle inequality), which the state bounds above already limit
        d = np.abs(sc - o["score"])
        bound = np.full(n, self.score_tol)
        if self.s.exit_kind == 1:
            derived = np.linalg.norm((g_out - o_out) - (g_in - o_in), axis=1)
            bound = np.maximum(bound, derived * (1 + 1e-6) + 1e-4 + 1e-5 * np.abs(o["score"]))
        self.score_bound = bound
        self.errors["score_max"] = max(self.errors["score_max"], float(d.max()))
        self.ratio["score_max"] = max(self.ratio.get("score_max", 0.0), float((d / bound).max()))
        assert (d <= bound).all(), f"exit score max abs {d.max():.3e} (bound {bound[np.argmax(d / bound)]:.3e})"
        dev_next = out.exit_next[:n].cpu().numpy()
        if not gated:
            # replayed depths: the next loop is the last one exactly when c + 2 == depth
            assert dev_next.tolist() == ((o["exit_mask"] == 0) & (cs + 2 == deps)).astype(np.uint8).tolist()
        else:
            self._gate_next(cs, slots, o, dev_next, pend)
        for i in range(n):
            planes = [int(cs[i]) + 1]
            if o["exit_mask"][i]:
                planes += list(range(int(deps[i]) + 1, self.R + 1))
            self._cmp_kv([seqs[i]], [poss[i]], planes, "core kv")
        if self.calls["loop"] % 10 == 0:
            print(f"[lockstep] {self.calls} max errors {self.errors}", flush=True)
        return o

    def _exit_signal(self, h, h_in):
        """The exit signal of states h (rows) after a loop from h_in, in fp64:
        ||h - h_in||_2, or sigmoid(w_exit . RMSNorm(h)) (Section 4.3; App. C.2)."""
        if self.s.exit_kind == 1:
            return np.linalg.norm(h - h_in, axis=1)
        nrm = h / np.sqrt(np.mean(h * h, axis=1, keepdims=True) + self.s.rms_eps)
        return 1.0 / (1.0 + np.exp(-(nrm @ self.w_exit)))

    def _gate_next(self, cs, slots, o, dev_next, pend):
        """The oracle's decisions for the next loop from its own scores; a
        device decision may differ only where the oracle's score lies within
        the score tolerance of the threshold, and is then adopted by both."""
        thr = self.gate[0]
        _, o_next = self.om.gate_decide(cs, o["score"], thr, True, pend)
        exited = o["exit_mask"] != 0
        self.gate_stats["decisions"] += int((~exited).sum())
        self.gate_stats["exits_before_r_max"] += int((exited & (cs + 1 < self.R)).sum())
        near = np.abs(o["score"] - thr) <= self.score_bound
        self.gate_stats["near_threshold"] += int((near & ~exited).sum())
        diff = (dev_next != o_next) & ~exited
        assert not (diff & ~near).any(), f"exit decisions differ away from the threshold: {o['score'][diff]}"
        self.gate_stats["overridden"] += int(diff.sum())
        final = np.where(diff, dev_next, o_next).astype(np.uint8)
        self.opending[slots] = np.where(exited, 0, final)

    def coda(self, seqs, poss):
        slots = self.o.slots(seqs, poss)
        g32 = self._oracle_bound(lambda m: oracle.coda(m, self.op, self.oh, slots, seqs, poss), lambda r: r[0].copy())
        ol, oid = self.o.coda(seqs, poss)
        self._set_bound(g32, ol, "coda")
        rows = cdb.Rows(slots, seqs, poss)
        n = len(seqs)
        logits = torch.zeros((n, self.s.vocab), dtype=torch.float32, device="cuda")
        ids = torch.zeros(n, dtype=torch.int32, device="cuda")
        cdb.cdb_boundary_coda(self.gm.model, self.gkv.c, self.gstate.c, rows.c, logits, ids, self.ws.buf)
        torch.cuda.synchronize()
        self.calls["coda"] += 1
        gl = logits.cpu().numpy()
        self._cmp("logit_max", "logit_mean", gl, ol, "coda logits", key_rel="logit_rel")
        gid = ids.cpu().numpy()
        # logits within b of the oracle's: a top-2 gap above 2b fixes the argmax
        gap = max(4 * TOL_MAX, 2 * self.tol[0])
        for i in range(n):
            top2 = np.sort(ol[i])[-2:]
            if top2[1] - top2[0] > gap:
                assert gid[i] == oid[i], f"argmax {gid[i]} vs oracle {oid[i]}"
                self.argmax_checked += 1
            else:  # near-tie: the GPU's choice must be (near) maximal under the oracle
                assert ol[i][gid[i]] >= top2[1] - gap
        if self.s.n_coda:
            self._cmp_kv(seqs, poss, [self.R + 1], "coda kv")
        return ol, oid

    def device_error(self) -> int:
        return cdb.cdb_read_device_error(self.ws.buf)

    # -------------------------------------------------------------- whole schedule
    def run(self, prompts: List[np.ndarray], n_decode: List[int], depths: List[np.ndarray]):
        toks = run_schedule(self, prompts, n_decode, depths, self.R, self.max_batch)
        self.check_means()
        return toks


def oracle_realizations(s, weights, op_args):
    """The oracle's loop step on the same inputs under fp32-level realizations
    of its arithmetic (same bf16 storage points): fp32 accumulators; the fp64
    steps from the state rounded to fp32; the fp64 steps from the state under
    two draws of fp32-sized relative noise.  Returns (states, scores) per
    realization; the oracle's buffers are restored after each."""
    op, oh, oe, oslot, pos, cs, deps = op_args
    saved = op.core.copy()
    out = []
    rng = np.random.default_rng(1234)
    for k in range(4):
        h, e = oh.copy(), None if oe is None else oe.copy()
        if k == 1:
            h = h.astype(np.float32).astype(np.float64)
            e = None if e is None else e.astype(np.float32).astype(np.float64)
        elif k >= 2:
            h *= 1.0 + 2.0 ** -24 * rng.standard_normal(h.shape)
            if e is not None:
                e *= 1.0 + 2.0 ** -24 * rng.standard_normal(e.shape)
        m = oracle.Model(s, weights, bf16_storage=True, acc32=(k == 0))
        o = oracle.loop_step(m, op, h, e, oslot, oslot, pos, cs, deps)
        op.core[...] = saved
        out.append((h, o["score"]))
    return out


def injected_loop_step(shape, weights, rows_np, sample, seed=11, gpu_model=None, sensitivity=False):
    """One cdb_loop_step over a full batch at the real shape, checked on sampled
    rows by the oracle from the same injected inputs (states and the sampled rows'
    K/V context come from the seeded generators; the other rows' K/V is random
    device data).  Integer outputs are checked for the whole batch.  With
    `sensitivity` the bound is DRIFT_FACTOR times the largest distance of the
    oracle's fp32-level realizations from the fp64 oracle on the same rows, where
    that exceeds the absolute tolerance.  Returns the errors, the bound, and the
    ratio of each error to its bound."""
    s = shape
    R = s.r_max
    n = len(rows_np["pos"])
    pos, cs, deps = rows_np["pos"], rows_np["c"], rows_np["depth"]
    dm = gpu_model or cdb.DeviceModel(s, weights)
    # device pages: row i owns sequence i; plane c+1 over its context, plus the
    # page at pos of every deeper plane (copy-on-exit destinations)
    pages = [cdbgen.pages_for(int(p) + 1) for p in pos]
    max_pages = max(pages)
    pt = np.full((n, R + 2, max_pages), -1, np.int32)
    nxt = 0
    for i in range(n):
        for pg in range(pages[i]):
            pt[i, cs[i] + 1, pg] = nxt
            nxt += 1
        for pl in range(cs[i] + 2, R + 1):
            pt[i, pl, pages[i] - 1] = nxt
            nxt += 1
    gkv = cdb.PagedKV(s, n, max_pages, 0, nxt, 0, fill="random")
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    gkv.core.normal_(0.0, 1.0, generator=g)
    gkv.page_table.copy_(torch.from_numpy(pt))
    # oracle pages for the sampled rows only, with their own ids
    ns = len(sample)
    opages = sum(pages[i] + (R - cs[i] - 1) for i in sample)
    op = oracle.Paged(s, ns, max_pages, 0, opages, 0)
    nxt_o = 0
    for j, i in enumerate(sample):
        for pl in range(cs[i] + 1, R + 1):
            for pg in range(pages[i]):
                if pt[i, pl, pg] < 0:
                    continue
                op.page_table[j, pl, pg] = nxt_o
                bits = cdbgen.random_kv_bf16(op.core.shape[1:], seed, stream=int(i) * 1000 + pl * 100 + pg)
                op.core[nxt_o] = cdbgen.bf16_to_f32(bits)
                gkv.core[:, int(pt[i, pl, pg])].copy_(
                    torch.from_numpy(bits.view(np.int16)).to("cuda").view(torch.bfloat16))
                nxt_o += 1
    # states
    h = cdbgen.random_state(n, s.d, seed, stream=1)
    state = cdb.State(s, n)
    state.h.copy_(torch.from_numpy(h))
    oh = h[sample].astype(np.float64)
    oe = None
    if s.injection:
        e = cdbgen.random_state(n, s.d, seed, stream=2)
        state.e.copy_(torch.from_numpy(e))
        oe = e[sample].astype(np.float64)
    rows = cdb.Rows(rows_np["slot"], rows_np["seq"], pos, cs, deps)
    out = cdb.StepOut(n)
    ws = cdb.Workspace(dm.desc, n)
    torch.cuda.synchronize()
    cdb.cdb_loop_step(dm.model, gkv.c, state.c, rows.c, out.c, ws.buf)
    torch.cuda.synchronize()
    assert cdb.cdb_read_device_error(ws.buf) == 0
    # integer outputs, whole batch
    want = oracle.exit_compact(cs, deps, R)
    cnt = out.counts.cpu().numpy()
    assert cnt.tolist() == want["counts"].tolist()
    assert out.mask[:n].cpu().numpy().tolist() == want["exit_mask"].tolist()
    assert out.cont[:cnt[0]].cpu().numpy().tolist() == want["cont"].tolist()
    assert out.exited[:cnt[1]].cpu().numpy().tolist() == want["exited"].tolist()
    # the oracle's step on the sampled rows
    oslot = np.arange(ns, dtype=np.int32)
    tol_max, tol_mean, tol_score = TOL_MAX, TOL_MEAN, TOL_MAX
    err = {"rows": ns}
    reals = None
    if sensitivity:
        reals = oracle_realizations(s, weights, (op, oh, oe, oslot, pos[sample], cs[sample], deps[sample]))
    o = oracle.loop_step(oracle.Model(s, weights, bf16_storage=True), op, oh, oe, oslot, oslot, pos[sample],
                         cs[sample], deps[sample])
    if reals:
        dmax = max(float(np.abs(h - oh).max()) for h, _ in reals)
        dmean = max(float(np.abs(h - oh).mean()) for h, _ in reals)
        dscore = max(float(np.abs(sc - o["score"]).max()) for _, sc in reals)
        err["drift_max"], err["drift_mean"], err["drift_score"] = dmax, dmean, dscore
        err["drift_rel"] = max(row_rel(h, oh) for h, _ in reals)
        tol_max, tol_mean = max(TOL_MAX, DRIFT_FACTOR * dmax), max(TOL_MEAN, DRIFT_FACTOR * dmean)
        tol_score = max(TOL_MAX, DRIFT_FACTOR * dscore)
    gh = state.h.cpu().numpy()[sample]
    d = np.abs(gh - oh)
    err["h_max"], err["h_mean"], err["h_rel"] = float(d.max()), float(d.mean()), row_rel(gh, oh)
    err["bound"] = (tol_max, tol_mean)
    err["ratio_max"], err["ratio_mean"] = err["h_max"] / tol_max, err["h_mean"] / tol_mean
    err["abs_bound_met"] = bool(err["h_max"] <= TOL_MAX and err["h_mean"] <= TOL_MEAN)
    assert d.max() <= tol_max and d.mean() <= tol_mean, err
    sc = out.score.cpu().numpy()[sample]
    err["score_max"] = float(np.abs(sc - o["score"]).max())
    assert err["score_max"] <= tol_score, (err, tol_score)
    kv_max = 0.0
    for j, i in enumerate(sample):
        planes = [int(cs[i]) + 1]
        if cs[i] + 1 == deps[i]:
            planes += list(range(int(deps[i]) + 1, R + 1))
        t = int(pos[i])
        for pl in planes:
            gpage = gkv.core[:, int(pt[i, pl, t // PAGE])][:, :, :, t % PAGE, :].float().cpu().numpy()
            opage = op.core[int(op.page_table[j, pl, t // PAGE])][:, :, :, t % PAGE, :]
            dd = np.abs(gpage - opage)
            kv_max = max(kv_max, float(dd.max()))
            assert not (dd > np.maximum(tol_max, np.abs(opage) * 2.0 ** -7 * 1.001)).any(), (i, pl, dd.max())
            assert dd.mean() <= tol_mean
    err["kv_max"] = kv_max
    return err


def sample_rows(rows_np, r_max, k=16, seed=0):
    """Up to k rows of a batch to check against the oracle: both members of
    several of the attention's row pairs (the kernel pairs the p-th longest
    context with the p-th shortest, ranking by descending position, ties by
    index: pairs 0, 1, a quarter and the middle), one row of every loop index
    present, exiting rows with copy-on-exit (depth < r_max) and continuing rows,
    then seeded picks."""
    c, dep, pos = rows_np["c"], rows_np["depth"], rows_np["pos"]
    n = len(pos)
    order = sorted(range(n), key=lambda i: (-int(pos[i]), i))
    picks = []

    def add(i):
        if i not in picks and len(picks) < k:
            picks.append(int(i))

    for p in sorted({0, 1, n // 4, (n + 1) // 2 - 1}):
        if 0 <= p < (n + 1) // 2:
            add(order[p])
            add(order[n - 1 - p])
    for cv in sorted(set(int(x) for x in c)):
        add(int(np.flatnonzero(c == cv)[0]))
    ex = [i for i in range(n) if c[i] + 1 == dep[i] and dep[i] < r_max]
    co = [i for i in range(n) if c[i] + 1 < dep[i]]
    for i in ex[:2] + co[:2]:
        add(i)
    rest = [i for i in np.random.default_rng(seed).permutation(n) if i not in picks]
    for i in rest:
        add(i)
    return picks
