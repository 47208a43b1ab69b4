"""The oracle's batched CDB executor (test infrastructure only).

A plain refill scheduler (paper Section 4.1) over the oracle's stage operators
(orc_prelude / orc_loop_step / orc_coda), with its own page allocator and paged
fp64 pools.  It exists to check, on the CPU, that running tokens of many
sequences together in mixed-depth loop steps gives exactly what each sequence
gives alone (the paper's point that CDB carries out an exit rule without
changing the model's predictions, Section 3).

Prompt tokens run at depth r_max; decode tokens use their depth-table entry.
Pages: lowest free id first, every page of a sequence and every plane mapped
at admission, in (sequence, page index, plane) order.  The shared core
layouts (Section 4.2; App. C.1) are page-table aliasing: under the single
shared slot every core plane of a token page maps one page; under
first-then-shared plane 1 has its own page and planes 2..r_max share another.
"""
from __future__ import annotations

from collections import deque
from typing import Dict, List, Optional

import numpy as np

from . import KV_FIRST_THEN_SHARED, KV_FULL, KV_SHARED, Model, Paged, coda, loop_step, prelude

PAGE = 16


class Allocator:
    def __init__(self, n_pages: int):
        self.free = list(range(n_pages))

    def take(self) -> int:
        if not self.free:
            raise MemoryError("page pool exhausted")
        self.free.sort()
        return self.free.pop(0)


def core_pages_per_page(r_max: int, kv_layout: int) -> int:
    """Distinct core pages behind one 16-token page of a sequence."""
    if kv_layout == KV_SHARED:
        return 1
    if kv_layout == KV_FIRST_THEN_SHARED:
        return min(2, r_max)
    return r_max


def run(model: Model, prompts: List[np.ndarray], n_decode: List[int], depths: List[np.ndarray],
        forced: Optional[List[np.ndarray]] = None, max_batch: int = 4,
        kv_layout: int = KV_FULL) -> List[Dict[str, np.ndarray]]:
    """Decode every sequence with the refill policy.

    prompts[i]: prompt ids; n_decode[i]: decode inputs; depths[i]: exit depth per
    position (length len(prompt) + n_decode; prompt entries must be r_max);
    forced[i] (optional): the decode input ids (teacher forcing), else greedy.
    Returns per sequence: tokens, logits [T][V], h at exit [T][d], scores [T][r_max].
    """
    s = model.shape
    R = s.r_max
    n_seq = len(prompts)
    T = [len(p) + n for p, n in zip(prompts, n_decode)]
    max_pages = max((t + PAGE - 1) // PAGE for t in T)
    tot_pages = sum((t + PAGE - 1) // PAGE for t in T)
    n_core_pages = tot_pages * core_pages_per_page(R, kv_layout)
    paged = Paged(s, n_seq, max_pages, tot_pages if s.n_prelude else 0, n_core_pages,
                  tot_pages if s.n_coda else 0)
    a_pre, a_core, a_coda = Allocator(tot_pages), Allocator(n_core_pages), Allocator(tot_pages)
    for q in range(n_seq):
        for pg in range((T[q] + PAGE - 1) // PAGE):
            shared = -1
            for plane in range(R + 2):
                if plane == 0:
                    if s.n_prelude:
                        paged.page_table[q, plane, pg] = a_pre.take()
                elif plane == R + 1:
                    if s.n_coda:
                        paged.page_table[q, plane, pg] = a_coda.take()
                elif kv_layout == KV_SHARED or (kv_layout == KV_FIRST_THEN_SHARED and plane >= 2):
                    if shared < 0:
                        shared = a_core.take()
                    paged.page_table[q, plane, pg] = shared
                else:
                    paged.page_table[q, plane, pg] = a_core.take()

    base = np.cumsum([0] + T)  # state slot of (seq q, pos t) = base[q] + t
    n_slots = int(base[-1])
    state_h = np.zeros((max(n_slots, 1), s.d))
    state_e = np.zeros((max(n_slots, 1), s.d)) if s.injection else None
    out = [{"tokens": np.zeros(T[q], dtype=np.int32), "logits": np.zeros((T[q], s.vocab)),
            "h": np.zeros((T[q], s.d)), "scores": np.full((T[q], R), np.nan)} for q in range(n_seq)]
    for q in range(n_seq):
        assert np.all(depths[q][: len(prompts[q])] == R)
        out[q]["tokens"][: len(prompts[q])] = prompts[q]

    # ---- prefill: every prompt token, full depth, sequences one after another
    for q in range(n_seq):
        P = len(prompts[q])
        pos = np.arange(P, dtype=np.int32)
        slot = (base[q] + pos).astype(np.int32)
        seq = np.full(P, q, dtype=np.int32)
        prelude(model, paged, state_h, state_e, slot, seq, pos, prompts[q])
        for c in range(R):
            r = loop_step(model, paged, state_h, state_e, slot, seq, pos, np.full(P, c, np.int32),
                          np.full(P, R, np.int32))
            out[q]["scores"][pos, c] = r["score"]
        out[q]["h"][pos] = state_h[slot]
        logits, ids = coda(model, paged, state_h, slot, seq, pos)
        out[q]["logits"][pos] = logits
        if n_decode[q] > 0:
            nxt = forced[q][0] if forced is not None else ids[-1]
            out[q]["tokens"][P] = nxt

    # ---- decode: two queues -- tokens waiting for the boundary stages, and
    # loop work items; exits refill the batch on the next tick
    boundary = deque()  # (seq, pos) awaiting the prelude
    loopq = deque()  # [seq, pos, c]
    for q in range(n_seq):
        if n_decode[q] > 0:
            boundary.append((q, len(prompts[q])))
    while boundary or loopq:
        if boundary:
            items = list(boundary)
            boundary.clear()
            seq = np.array([q for q, _ in items], dtype=np.int32)
            pos = np.array([t for _, t in items], dtype=np.int32)
            slot = (base[seq] + pos).astype(np.int32)
            toks = np.array([out[q]["tokens"][t] for q, t in items], dtype=np.int32)
            prelude(model, paged, state_h, state_e, slot, seq, pos, toks)
            for q, t in items:
                loopq.append([q, t, 0])
        batch = [loopq.popleft() for _ in range(min(max_batch, len(loopq)))]
        if not batch:
            continue
        seq = np.array([b[0] for b in batch], dtype=np.int32)
        pos = np.array([b[1] for b in batch], dtype=np.int32)
        c = np.array([b[2] for b in batch], dtype=np.int32)
        dep = np.array([depths[b[0]][b[1]] for b in batch], dtype=np.int32)
        slot = (base[seq] + pos).astype(np.int32)
        r = loop_step(model, paged, state_h, state_e, slot, seq, pos, c, dep)
        for i, b in enumerate(batch):
            out[b[0]]["scores"][b[1], b[2]] = r["score"][i]
        for i in r["cont"]:
            batch[i][2] += 1
            loopq.append(batch[i])
        ex = r["exited"]
        if len(ex):
            eseq, epos, eslot = seq[ex], pos[ex], slot[ex]
            logits, ids = coda(model, paged, state_h, eslot, eseq, epos)
            for j, (q, t) in enumerate(zip(eseq, epos)):
                out[q]["logits"][t] = logits[j]
                out[q]["h"][t] = state_h[eslot[j]]
                if t + 1 < T[q]:
                    k = t + 1 - len(prompts[q])
                    out[q]["tokens"][t + 1] = forced[q][k] if forced is not None else ids[j]
                    boundary.append((int(q), int(t + 1)))
    return out
