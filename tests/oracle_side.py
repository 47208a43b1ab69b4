"""The oracle's side of a lockstep run, and the refill schedule both sides
follow.  Imports only the oracle and the seeded generators (no HIP binding), so
the script that writes stored drift envelopes can run it without a GPU.

The schedule is the refill policy: prompt tokens go through prelude, r_max loop
steps and coda; decode tokens run coda -> prelude -> loop queue, and every loop
step takes up to `max_batch` work items from the loop queue, mixing loop
indices.  Decode inputs are teacher-forced with the fp64 oracle's greedy ids.
"""
from __future__ import annotations

from collections import deque
from typing import List

import numpy as np

import cdbgen
import oracle

MAX_ROWS = 256  # rows per stage call


class OracleSide:
    """Oracle state, paged pools and page table of one lockstep run.

    Page table: lowest free id first, (seq, page, plane) order; aliased core
    planes (kv_layout 1 single shared slot, 2 first-then-shared) share the page
    of the first plane they alias.  Slots: sequence q's position t lives in
    slot base[q] + t.
    state_hook(side, slots): called after every call that wrote states (the
    drift realizations perturb or round the state there)."""

    def __init__(self, shape, weights, seq_lens: List[int], kv_layout: int = 0, extra_pages: int = 0,
                 bf16_storage: bool = True, acc32: bool = False, state_hook=None, sum_order: int = 0):
        s = self.s = shape
        self.R = s.r_max
        self.om = oracle.Model(s, weights, bf16_storage=bf16_storage, acc32=acc32, sum_order=sum_order)
        n_seq = len(seq_lens)
        self.max_pages = max(cdbgen.pages_for(t) for t in seq_lens)
        tot = sum(cdbgen.pages_for(t) for t in seq_lens) + extra_pages
        per = {0: self.R, 1: 1, 2: min(2, self.R)}[kv_layout]
        self.pages = (tot if s.n_prelude else 0), tot * per, (tot if s.n_coda else 0)
        self.op = oracle.Paged(s, n_seq, self.max_pages, *self.pages)
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
        self.base = np.cumsum([0] + list(seq_lens))
        n_slots = int(self.base[-1])
        self.oh = np.zeros((n_slots, s.d))
        self.oe = np.zeros((n_slots, s.d)) if s.injection else None
        self.state_hook = state_hook

    def slots(self, seqs, poss):
        return (self.base[np.asarray(seqs)] + np.asarray(poss)).astype(np.int32)

    def prelude(self, seqs, poss, toks):
        slots = self.slots(seqs, poss)
        oracle.prelude(self.om, self.op, self.oh, self.oe, slots, seqs, poss, toks)
        if self.state_hook:
            self.state_hook(self, slots)
        return slots

    def loop(self, seqs, poss, cs, deps):
        slots = self.slots(seqs, poss)
        o = oracle.loop_step(self.om, self.op, self.oh, self.oe, slots, seqs, poss, cs, deps)
        if self.state_hook:
            self.state_hook(self, slots)
        return o

    def coda(self, seqs, poss):
        return oracle.coda(self.om, self.op, self.oh, self.slots(seqs, poss), seqs, poss)


def run_schedule(stage, prompts: List[np.ndarray], n_decode: List[int], depths: List[np.ndarray], R: int,
                 max_batch: int, on_loop=None):
    """Drive `stage` (methods prelude(seqs, poss, toks), loop(seqs, poss, cs,
    deps, replay) -> the oracle's step outputs, coda(seqs, poss) -> (logits,
    ids)) through whole decodes.  Returns the token ids (prompt + greedy)."""
    toks = [np.zeros(len(p) + n, np.int32) for p, n in zip(prompts, n_decode)]
    for q, p in enumerate(prompts):
        P = len(p)
        toks[q][:P] = p
        pos = np.arange(P, dtype=np.int32)
        seq = np.full(P, q, np.int32)
        for a in range(0, P, MAX_ROWS):
            stage.prelude(seq[a:a + MAX_ROWS], pos[a:a + MAX_ROWS], p[a:a + MAX_ROWS])
        for c in range(R):
            for a in range(0, P, MAX_ROWS):
                b = slice(a, a + MAX_ROWS)
                stage.loop(seq[b], pos[b], np.full(len(pos[b]), c, np.int32), np.full(len(pos[b]), R, np.int32),
                           replay=True)
        for a in range(0, P, MAX_ROWS):
            _, oid = stage.coda(seq[a:a + MAX_ROWS], pos[a:a + MAX_ROWS])
        if n_decode[q]:
            toks[q][P] = oid[-1]
    boundary = deque((q, len(prompts[q])) for q in range(len(prompts)) if n_decode[q])
    loopq = deque()
    n_loops = 0
    while boundary or loopq:
        if boundary:
            items = list(boundary)
            boundary.clear()
            seq = np.array([q for q, _ in items], np.int32)
            pos = np.array([t for _, t in items], np.int32)
            stage.prelude(seq, pos, np.array([toks[q][t] for q, t in items], np.int32))
            loopq.extend([q, t, 0] for q, t in items)
        batch = [loopq.popleft() for _ in range(min(max_batch, len(loopq)))]
        if not batch:
            continue
        seq = np.array([b[0] for b in batch], np.int32)
        pos = np.array([b[1] for b in batch], np.int32)
        cs = np.array([b[2] for b in batch], np.int32)
        deps = np.array([depths[b[0]][b[1]] for b in batch], np.int32)
        o = stage.loop(seq, pos, cs, deps, replay=False)
        n_loops += 1
        if on_loop:
            on_loop(n_loops)
        for i in o["cont"]:
            batch[i][2] += 1
            loopq.append(batch[i])
        ex = o["exited"]
        if len(ex):
            _, oid = stage.coda(seq[ex], pos[ex])
            for j, i in enumerate(ex):
                q, t = int(seq[i]), int(pos[i])
                if t + 1 < len(toks[q]):
                    toks[q][t + 1] = oid[j]
                    boundary.append((q, t + 1))
    return toks


def row_rel(got, want):
    """Largest relative error of a row, ||got_i - want_i||_2 / ||want_i||_2."""
    got, want = np.atleast_2d(np.asarray(got, np.float64)), np.atleast_2d(want)
    den = np.maximum(np.linalg.norm(want, axis=1), 1e-300)
    return float((np.linalg.norm(got - want, axis=1) / den).max()) if got.size else 0.0


# ---------------------------------------------------------------- free-running runs

def free_run_case(name: str):
    """Inputs of a free-running lockstep run (no resync): the model, its
    weights, prompts, per-token depths, decode lengths and batch size.
    ouro24: the Ouro-shaped model at full depth (24 core layers, r_max 4),
    2 sequences, prompt 16, decode 6, config 2's depth distribution.
    huginn4: the Huginn-shaped model whole (2 prelude, 4 recurrent layers with
    the injection adapter looped up to 32 times, 2 coda), 2 sequences, prompt
    3, decode 3, config 3's depth distribution."""
    if name == "huginn4":
        s = cdbgen.HUGINN
        P, N, n_seqs, stream = 3, 3, 2, 20
        depth_spec = cdbgen.WORKLOADS[3].depth
        w = cdbgen.model_weights(s)
        prompts = [cdbgen.prompt_ids(s.vocab, 1, P, stream=stream + q)[0] for q in range(n_seqs)]
        depths = [np.concatenate([np.full(P, s.r_max, np.int32),
                                  cdbgen.draw_depths(depth_spec, N, s.r_max, stream=stream + q)])
                  for q in range(n_seqs)]
        return s, w, prompts, depths, [N] * n_seqs, n_seqs
    if name == "ouro24":
        s = cdbgen.OURO
        P, N, n_seqs, stream = 16, 6, 2, 20
        depth_spec = cdbgen.OURO_DEPTHS
    elif name == "ouro2":
        s = cdbgen.shrink(cdbgen.OURO, n_core=2)
        P, N, n_seqs, stream = 16, 6, 2, 20
        depth_spec = cdbgen.OURO_DEPTHS
    else:
        raise KeyError(name)
    w = cdbgen.model_weights(cdbgen.OURO)
    if s.n_core != cdbgen.OURO.n_core:
        w = dict(w)
        w["layers"] = w["layers"][:s.n_core]
    prompts = [cdbgen.prompt_ids(s.vocab, 1, P, stream=stream + q)[0] for q in range(n_seqs)]
    depths = [np.concatenate([np.full(P, s.r_max, np.int32),
                              cdbgen.draw_depths(depth_spec, N, s.r_max, stream=stream + q)]) for q in range(n_seqs)]
    return s, w, prompts, depths, [N] * n_seqs, n_seqs


class DriftRun:
    """The fp64 oracle run alongside fp32-level realizations of its own
    arithmetic, each free-running on its own state and pools: the same source
    with fp32 accumulators, summing the projections in index order, in reverse
    and in blocks of 32; the fp64 steps with the state rounded to fp32 after
    every call (as a device keeps it); and the fp64 steps with fp32-sized
    relative noise (2^-24 N(0, 1)) on the state after every call, six draws.
    Every call records, per output, the largest distance of any realization
    from the fp64 run: how far an fp32 implementation of the same arithmetic
    can sit from the oracle after this many calls.  Decode calls hold one to a
    few rows, whose largest deviation a handful of realizations samples poorly;
    hence ten."""

    N_NOISE = 6

    def __init__(self, shape, weights, seq_lens, threads: int = 6):
        from concurrent.futures import ThreadPoolExecutor

        self.ref = OracleSide(shape, weights, seq_lens)
        rngs = [np.random.default_rng(7000 + k) for k in range(self.N_NOISE)]

        def to_fp32(side, slots):
            for a in (side.oh, side.oe):
                if a is not None:
                    a[slots] = a[slots].astype(np.float32)

        def noise(k):
            def hook(side, slots):
                for a in (side.oh, side.oe):
                    if a is not None:
                        a[slots] *= 1.0 + 2.0 ** -24 * rngs[k].standard_normal(a[slots].shape)
            return hook

        self.real = [OracleSide(shape, weights, seq_lens, acc32=True, sum_order=k) for k in (0, 1, 2)] + \
                    [OracleSide(shape, weights, seq_lens, state_hook=to_fp32)] + \
                    [OracleSide(shape, weights, seq_lens, state_hook=noise(k)) for k in range(self.N_NOISE)]
        self.pool = ThreadPoolExecutor(max_workers=threads)  # the oracle's ctypes calls release the GIL
        self.calls = []

    def _all(self, fn):
        futs = [self.pool.submit(fn, side) for side in [self.ref] + self.real]
        return [f.result() for f in futs]

    def _states(self, slots, outs):
        want = self.ref.oh[slots]
        d = [np.abs(side.oh[slots] - want) for side in self.real]
        each = [float(x.max()) for x in d]
        return {"h_max": max(each), "h_mean": max(float(x.mean()) for x in d),
                "h_rel": max(row_rel(side.oh[slots], want) for side in self.real), "h_max_each": each}

    def prelude(self, seqs, poss, toks):
        self._all(lambda side: side.prelude(seqs, poss, toks))
        rec = {"stage": "prelude", "rows": len(seqs)}
        rec.update(self._states(self.ref.slots(seqs, poss), None))
        self.calls.append(rec)

    def loop(self, seqs, poss, cs, deps, replay=False):
        outs = self._all(lambda side: side.loop(seqs, poss, cs, deps))
        rec = {"stage": "loop", "rows": len(seqs)}
        rec.update(self._states(self.ref.slots(seqs, poss), outs))
        rec["score_max_each"] = [float(np.abs(o["score"] - outs[0]["score"]).max()) for o in outs[1:]]
        rec["score_max"] = max(rec["score_max_each"])
        for o in outs[1:]:
            assert o["exit_mask"].tolist() == outs[0]["exit_mask"].tolist()
        self.calls.append(rec)
        return outs[0]

    def coda(self, seqs, poss):
        outs = self._all(lambda side: side.coda(seqs, poss))
        ol = outs[0][0]
        d = [np.abs(o[0] - ol) for o in outs[1:]]
        self.calls.append({"stage": "coda", "rows": len(seqs), "logit_max": max(float(x.max()) for x in d),
                           "logit_max_each": [float(x.max()) for x in d],
                           "logit_mean": max(float(x.mean()) for x in d),
                           "logit_rel": max(row_rel(o[0], ol) for o in outs[1:])})
        return outs[0]
