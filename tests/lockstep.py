"""Drives the HIP stage calls and the CPU oracle side by side on identical row
batches, so every call's outputs can be compared.  Used by the GPU parity tests.

The schedule is the refill policy: prompt tokens go through prelude, r_max loop
steps and coda; decode tokens run coda -> prelude -> loop queue, and every loop
step takes up to `max_batch` work items from the loop queue, mixing loop
indices.  Decode inputs are teacher-forced with the oracle's greedy ids.
"""
from __future__ import annotations

from collections import deque
from typing import Dict, List

import numpy as np
import torch

import cdbgen
import oracle
import paper_2608_09444_amd as cdb

PAGE = 16
TOL_MAX, TOL_MEAN = 2e-2, 2e-3


def bf16_pool_to_f64(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


class Lockstep:
    def __init__(self, shape, weights, seq_lens: List[int], max_batch: int, bf16_storage: bool = True,
                 extra_pages: int = 0, resync: bool = False, sensitivity: bool = False, kv_layout: int = 0,
                 gate=None):
        """resync: after every call, copy the oracle's states and newly written
        K/V entries into the device buffers, so that each call is checked from
        identical inputs (deep random-init models amplify rounding-level
        differences from call to call).  kv_layout: 0 full, 1 single shared
        slot, 2 first-then-shared (core planes aliased in the page table).
        gate: (threshold, lookahead) for threshold exits decided on the device
        (lookahead only: each step's exits are fixed by the previous step, so
        both sides run the same rows); the loop-step depths are then ignored."""
        self.resync = resync
        self.sensitivity = sensitivity
        self.tol = (TOL_MAX, TOL_MEAN)
        self.self_diff = {"max": 0.0, "mean": 0.0}
        self.s = s = shape
        self.R = s.r_max
        self.max_batch = max_batch
        self.om = oracle.Model(s, weights, bf16_storage=bf16_storage)
        self.om32 = oracle.Model(s, weights, bf16_storage=bf16_storage, acc32=True) if sensitivity else None
        self.gm = cdb.DeviceModel(s, weights)
        n_seq = len(seq_lens)
        self.max_pages = max(cdbgen.pages_for(t) for t in seq_lens)
        tot = sum(cdbgen.pages_for(t) for t in seq_lens) + extra_pages
        per = {0: self.R, 1: 1, 2: min(2, self.R)}[kv_layout]
        pre_p, core_p, coda_p = (tot if s.n_prelude else 0), tot * per, (tot if s.n_coda else 0)
        self.op = oracle.Paged(s, n_seq, self.max_pages, pre_p, core_p, coda_p)
        self.gkv = cdb.PagedKV(s, n_seq, self.max_pages, pre_p, core_p, coda_p)
        # one page table for both sides: lowest free id first, (seq, page, plane)
        # order; aliased core planes share the page of the first plane they alias
        nxt = {0: 0, 1: 0, 2: 0}
        for q, T in enumerate(seq_lens):
            for pg in range(cdbgen.pages_for(T)):
                shared = -1
                for plane in range(self.R + 2):
                    st = 0 if plane == 0 else (2 if plane == self.R + 1 else 1)
                    if st == 0 and not s.n_prelude or st == 2 and not s.n_coda:
                        continue
                    if st == 1 and (kv_layout == 1 or (kv_layout == 2 and plane >= 2)):
                        if shared < 0:
                            shared = nxt[1]
                            nxt[1] += 1
                        self.op.page_table[q, plane, pg] = shared
                        continue
                    self.op.page_table[q, plane, pg] = nxt[st]
                    nxt[st] += 1
        self.gkv.page_table.copy_(torch.from_numpy(self.op.page_table))
        self.base = np.cumsum([0] + list(seq_lens))
        n_slots = int(self.base[-1])
        self.oh = np.zeros((n_slots, s.d))
        self.oe = np.zeros((n_slots, s.d)) if s.injection else None
        self.gstate = cdb.State(s, n_slots)
        self.ws = cdb.Workspace(self.gm.desc, max(max_batch, max(seq_lens)))
        self.errors: Dict[str, float] = {"h_max": 0.0, "h_mean": 0.0, "logit_max": 0.0, "logit_mean": 0.0,
                                         "kv_max": 0.0, "score_max": 0.0}
        self.calls = {"prelude": 0, "loop": 0, "coda": 0}
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
    def _cmp(self, key_max, key_mean, got, want, what):
        """max-abs is checked per call; mean-abs is a statistic of the whole
        result, checked over the run by check_means() (a call of two rows is
        dominated by single bf16 rounding flips)."""
        d = np.abs(np.asarray(got, np.float64) - want)
        mx, mn = float(d.max()) if d.size else 0.0, float(d.mean()) if d.size else 0.0
        self.errors[key_max] = max(self.errors[key_max], mx)
        if key_mean:
            self.errors[key_mean] = max(self.errors[key_mean], mn)
            acc = self.run_sums.setdefault(key_mean, [0.0, 0, 0.0])
            acc[0] += float(d.sum())
            acc[1] += d.size
            acc[2] += self.tol[1] * d.size
        tmax = self.tol[0]
        assert mx <= tmax, f"{what}: max abs {mx:.3e}, mean abs {mn:.3e} (max bound {tmax:.3e})"

    def check_means(self):
        """Mean-abs error of each output kind over the run against the
        element-weighted mean of the per-call bounds."""
        for key, (tot, n, bound) in self.run_sums.items():
            if n:
                assert tot / n <= bound / n, f"{key}: run mean abs {tot / n:.3e} > bound {bound / n:.3e}"

    def _oracle_bound(self, run32, out_of):
        """Run the call through several fp32-level realizations of the oracle's
        arithmetic on copies of the oracle's buffers, restoring them after each:
        the same steps with fp32 accumulators; the fp64 steps from the residual
        state rounded to fp32 (as the device keeps it); and the fp64 steps from
        the state under two draws of fp32-sized relative noise.  This call's
        bound is the larger of the absolute tolerance and twice the largest
        distance of any of them from the oracle's own outputs: in a call of a
        few rows the error is set by a handful of bf16 rounding flips, which one
        realization undersamples.  `out_of(result)` picks the compared output."""
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

    def _set_bound(self, variants, got64):
        if variants is None:
            return
        mx = max(float(np.abs(v - got64).max()) for v in variants)
        mn = max(float(np.abs(v - got64).mean()) for v in variants)
        self.self_diff["max"] = max(self.self_diff["max"], mx)
        self.self_diff["mean"] = max(self.self_diff["mean"], mn)
        self.tol = (max(TOL_MAX, 2 * mx), max(TOL_MEAN, 2 * mn))

    def _cmp_state(self, slots, what):
        idx = torch.as_tensor(slots, dtype=torch.long, device="cuda")
        g = self.gstate.h[idx].cpu().numpy()
        self._cmp("h_max", "h_mean", g, self.oh[slots], what)
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
        slots = (self.base[seqs] + poss).astype(np.int32)
        g32 = self._oracle_bound(lambda m: oracle.prelude(m, self.op, self.oh, self.oe, slots, seqs, poss, toks),
                                 lambda _: self.oh[slots].copy())
        oracle.prelude(self.om, self.op, self.oh, self.oe, slots, seqs, poss, toks)
        self._set_bound(g32, self.oh[slots])
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
        slots = (self.base[seqs] + poss).astype(np.int32)
        gated = self.gate is not None and not replay
        if gated:
            # this step's exits were decided by the previous one (or loop r_max)
            pend = self.opending[slots].copy()
            exit_now = (pend != 0) | (cs + 1 == self.R)
            deps = np.where(exit_now, cs + 1, self.R).astype(np.int32)
        g32 = self._oracle_bound(lambda m: oracle.loop_step(m, self.op, self.oh, self.oe, slots, seqs, poss, cs, deps),
                                 lambda _: self.oh[slots].copy())
        o = oracle.loop_step(self.om, self.op, self.oh, self.oe, slots, seqs, poss, cs, deps)
        self._set_bound(g32, self.oh[slots])
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
        self._cmp_state(slots, "loop-step state")
        sc = out.score[:n].cpu().numpy()
        d = np.abs(sc - o["score"])
        self.errors["score_max"] = max(self.errors["score_max"], float(d.max()))
        assert float(d.max()) <= self.tol[0], f"exit score max abs {d.max():.3e}"
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
        return o

    def _gate_next(self, cs, slots, o, dev_next, pend):
        """The oracle's decisions for the next loop from its own scores; a
        device decision may differ only where the oracle's score lies within
        the score tolerance of the threshold, and is then adopted by both."""
        thr = self.gate[0]
        _, o_next = self.om.gate_decide(cs, o["score"], thr, True, pend)
        exited = o["exit_mask"] != 0
        self.gate_stats["decisions"] += int((~exited).sum())
        self.gate_stats["exits_before_r_max"] += int((exited & (cs + 1 < self.R)).sum())
        near = np.abs(o["score"] - thr) <= self.tol[0]
        self.gate_stats["near_threshold"] += int((near & ~exited).sum())
        diff = (dev_next != o_next) & ~exited
        assert not (diff & ~near).any(), f"exit decisions differ away from the threshold: {o['score'][diff]}"
        self.gate_stats["overridden"] += int(diff.sum())
        final = np.where(diff, dev_next, o_next).astype(np.uint8)
        self.opending[slots] = np.where(exited, 0, final)

    def coda(self, seqs, poss):
        slots = (self.base[seqs] + poss).astype(np.int32)
        g32 = self._oracle_bound(lambda m: oracle.coda(m, self.op, self.oh, slots, seqs, poss), lambda r: r[0].copy())
        ol, oid = oracle.coda(self.om, self.op, self.oh, slots, seqs, poss)
        self._set_bound(g32, ol)
        rows = cdb.Rows(slots, seqs, poss)
        n = len(seqs)
        logits = torch.zeros((n, self.s.vocab), dtype=torch.float32, device="cuda")
        ids = torch.zeros(n, dtype=torch.int32, device="cuda")
        cdb.cdb_boundary_coda(self.gm.model, self.gkv.c, self.gstate.c, rows.c, logits, ids, self.ws.buf)
        torch.cuda.synchronize()
        self.calls["coda"] += 1
        gl = logits.cpu().numpy()
        self._cmp("logit_max", "logit_mean", gl, ol, "coda logits")
        gid = ids.cpu().numpy()
        for i in range(n):
            top2 = np.sort(ol[i])[-2:]
            if top2[1] - top2[0] > 4 * TOL_MAX:
                assert gid[i] == oid[i], f"argmax {gid[i]} vs oracle {oid[i]}"
                self.argmax_checked += 1
            else:  # near-tie: the GPU's choice must be (near) maximal under the oracle
                assert ol[i][gid[i]] >= top2[1] - 4 * TOL_MAX
        if self.s.n_coda:
            self._cmp_kv(seqs, poss, [self.R + 1], "coda kv")
        return ol, oid

    def device_error(self) -> int:
        return cdb.cdb_read_device_error(self.ws.buf)

    # -------------------------------------------------------------- whole schedule
    def run(self, prompts: List[np.ndarray], n_decode: List[int], depths: List[np.ndarray]):
        R = self.R
        toks = [np.zeros(len(p) + n, np.int32) for p, n in zip(prompts, n_decode)]
        for q, p in enumerate(prompts):
            P = len(p)
            toks[q][:P] = p
            pos = np.arange(P, dtype=np.int32)
            seq = np.full(P, q, np.int32)
            for a in range(0, P, cdb.MAX_ROWS):
                self.prelude(seq[a:a + cdb.MAX_ROWS], pos[a:a + cdb.MAX_ROWS], p[a:a + cdb.MAX_ROWS])
            for c in range(R):
                for a in range(0, P, cdb.MAX_ROWS):
                    b = slice(a, a + cdb.MAX_ROWS)
                    self.loop(seq[b], pos[b], np.full(len(pos[b]), c, np.int32), np.full(len(pos[b]), R, np.int32),
                              replay=True)
            for a in range(0, P, cdb.MAX_ROWS):
                _, oid = self.coda(seq[a:a + cdb.MAX_ROWS], pos[a:a + cdb.MAX_ROWS])
            if n_decode[q]:
                toks[q][P] = oid[-1]
        boundary = deque((q, len(prompts[q])) for q in range(len(prompts)) if n_decode[q])
        loopq = deque()
        while boundary or loopq:
            if boundary:
                items = list(boundary)
                boundary.clear()
                seq = np.array([q for q, _ in items], np.int32)
                pos = np.array([t for _, t in items], np.int32)
                self.prelude(seq, pos, np.array([toks[q][t] for q, t in items], np.int32))
                loopq.extend([q, t, 0] for q, t in items)
            batch = [loopq.popleft() for _ in range(min(self.max_batch, len(loopq)))]
            if not batch:
                continue
            seq = np.array([b[0] for b in batch], np.int32)
            pos = np.array([b[1] for b in batch], np.int32)
            cs = np.array([b[2] for b in batch], np.int32)
            deps = np.array([depths[b[0]][b[1]] for b in batch], np.int32)
            o = self.loop(seq, pos, cs, deps)
            if self.calls["loop"] % 10 == 0:
                print(f"[lockstep] {self.calls} max errors {self.errors}", flush=True)
            for i in o["cont"]:
                batch[i][2] += 1
                loopq.append(batch[i])
            ex = o["exited"]
            if len(ex):
                _, oid = self.coda(seq[ex], pos[ex])
                for j, i in enumerate(ex):
                    q, t = int(seq[i]), int(pos[i])
                    if t + 1 < len(toks[q]):
                        toks[q][t + 1] = oid[j]
                        boundary.append((q, t + 1))
        self.check_means()
        return toks


def oracle_fp32_drift(s, weights, op_args):
    """How far the oracle's own steps move when every sum and product is done in
    fp32 instead of fp64 (same inputs, same bf16 storage points).  A device that
    accumulates in fp32 cannot be expected to sit closer to the fp64 oracle than
    this: deep random-init cores amplify rounding-level differences through bf16
    rounding flips."""
    op, oh, oe, oslot, pos, cs, deps = op_args
    saved = op.core.copy()
    h64, h32 = oh.copy(), oh.copy()
    oracle.loop_step(oracle.Model(s, weights, bf16_storage=True), op, h64, oe, oslot, oslot, pos, cs, deps)
    op.core[...] = saved
    oracle.loop_step(oracle.Model(s, weights, bf16_storage=True, acc32=True), op, h32, oe, oslot, oslot, pos, cs,
                     deps)
    op.core[...] = saved
    d = np.abs(h32 - h64)
    return float(d.max()), float(d.mean())


def injected_loop_step(shape, weights, rows_np, sample, seed=11, gpu_model=None, sensitivity=False):
    """One cdb_loop_step over a full batch at the real shape, checked on sampled
    rows by the oracle from the same injected inputs (states and the sampled rows'
    K/V context come from the seeded generators; the other rows' K/V is random
    device data).  Integer outputs are checked for the whole batch.  Returns the
    largest errors seen."""
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
    tol_max, tol_mean = TOL_MAX, TOL_MEAN
    err = {}
    if sensitivity:
        smax, smean = oracle_fp32_drift(s, weights, (op, oh, oe, oslot, pos[sample], cs[sample], deps[sample]))
        err["oracle_fp32_max"], err["oracle_fp32_mean"] = smax, smean
        tol_max, tol_mean = max(TOL_MAX, 2 * smax), max(TOL_MEAN, 2 * smean)
    o = oracle.loop_step(oracle.Model(s, weights, bf16_storage=True), op, oh, oe, oslot, oslot, pos[sample],
                         cs[sample], deps[sample])
    gh = state.h.cpu().numpy()[sample]
    d = np.abs(gh - oh)
    err["h_max"], err["h_mean"] = float(d.max()), float(d.mean())
    assert d.max() <= tol_max and d.mean() <= tol_mean, (err, tol_max, tol_mean)
    sc = out.score.cpu().numpy()[sample]
    err["score_max"] = float(np.abs(sc - o["score"]).max())
    assert err["score_max"] <= tol_max, err
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
