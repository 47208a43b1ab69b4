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
                 extra_pages: int = 0):
        self.s = s = shape
        self.R = s.r_max
        self.max_batch = max_batch
        self.om = oracle.Model(s, weights, bf16_storage=bf16_storage)
        self.gm = cdb.DeviceModel(s, weights)
        n_seq = len(seq_lens)
        self.max_pages = max(cdbgen.pages_for(t) for t in seq_lens)
        tot = sum(cdbgen.pages_for(t) for t in seq_lens) + extra_pages
        pre_p, core_p, coda_p = (tot if s.n_prelude else 0), tot * self.R, (tot if s.n_coda else 0)
        self.op = oracle.Paged(s, n_seq, self.max_pages, pre_p, core_p, coda_p)
        self.gkv = cdb.PagedKV(s, n_seq, self.max_pages, pre_p, core_p, coda_p)
        # one page table for both sides: lowest free id first, (seq, page, plane) order
        nxt = {0: 0, 1: 0, 2: 0}
        for q, T in enumerate(seq_lens):
            for pg in range(cdbgen.pages_for(T)):
                for plane in range(self.R + 2):
                    st = 0 if plane == 0 else (2 if plane == self.R + 1 else 1)
                    if st == 0 and not s.n_prelude or st == 2 and not s.n_coda:
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

    # -------------------------------------------------------------- compare helpers
    def _cmp(self, key_max, key_mean, got, want, what):
        d = np.abs(np.asarray(got, np.float64) - want)
        mx, mn = float(d.max()) if d.size else 0.0, float(d.mean()) if d.size else 0.0
        self.errors[key_max] = max(self.errors[key_max], mx)
        if key_mean:
            self.errors[key_mean] = max(self.errors[key_mean], mn)
        assert mx <= TOL_MAX and mn <= TOL_MEAN, f"{what}: max abs {mx:.3e}, mean abs {mn:.3e}"

    def _cmp_state(self, slots, what):
        g = self.gstate.h[torch.as_tensor(slots, dtype=torch.long, device="cuda")].cpu().numpy()
        self._cmp("h_max", "h_mean", g, self.oh[slots], what)

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
                g = gp[pid, :, :, :, t % PAGE, :].float().cpu().numpy()
                o = opool[pid, :, :, :, t % PAGE, :]
                d = np.abs(g - o)
                self.errors["kv_max"] = max(self.errors["kv_max"], float(d.max()))
                # bf16 entries: at most one bf16 step apart (2^-7 relative), or the absolute bound
                bad = d > np.maximum(TOL_MAX, np.abs(o) * 2.0 ** -7 * 1.001)
                assert not bad.any() and float(d.mean()) <= TOL_MEAN, \
                    f"{what}: kv plane {plane} seq {q} pos {t}: max {d.max():.3e} mean {d.mean():.3e}"

    # -------------------------------------------------------------- stages
    def prelude(self, seqs, poss, toks):
        slots = (self.base[seqs] + poss).astype(np.int32)
        oracle.prelude(self.om, self.op, self.oh, self.oe, slots, seqs, poss, toks)
        rows = cdb.Rows(slots, seqs, poss)
        cdb.cdb_boundary_prelude(self.gm.model, self.gkv.c, self.gstate.c, rows.c,
                                 torch.as_tensor(toks, dtype=torch.int32, device="cuda"), self.ws.buf)
        torch.cuda.synchronize()
        self.calls["prelude"] += 1
        self._cmp_state(slots, "prelude state")
        if self.s.n_prelude:
            self._cmp_kv(seqs, poss, [0], "prelude kv")

    def loop(self, seqs, poss, cs, deps):
        slots = (self.base[seqs] + poss).astype(np.int32)
        o = oracle.loop_step(self.om, self.op, self.oh, self.oe, slots, seqs, poss, cs, deps)
        rows = cdb.Rows(slots, seqs, poss, cs, deps)
        out = cdb.StepOut(len(seqs))
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
        assert float(d.max()) <= TOL_MAX, f"exit score max abs {d.max():.3e}"
        for i in range(n):
            planes = [int(cs[i]) + 1]
            if o["exit_mask"][i]:
                planes += list(range(int(deps[i]) + 1, self.R + 1))
            self._cmp_kv([seqs[i]], [poss[i]], planes, "core kv")
        return o

    def coda(self, seqs, poss):
        slots = (self.base[seqs] + poss).astype(np.int32)
        ol, oid = oracle.coda(self.om, self.op, self.oh, slots, seqs, poss)
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
                    self.loop(seq[b], pos[b], np.full(len(pos[b]), c, np.int32), np.full(len(pos[b]), R, np.int32))
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
        return toks
