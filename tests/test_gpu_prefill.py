"""GPU: chunked prefill (cdb_prefill) against the oracle's stage operators run on
the same prompt as one block (prelude, r_max loop steps at full depth, coda).
Under the full KV layout a prompt split into chunks reads exactly what the
single block reads, so chunks and block must agree.  Logits within the
tolerance, greedy ids where the top-2 gap is clear, K/V of every plane within
one bf16 step.  For real widths the bounds widen to 1.25 times the distance
between the oracle and its fp32-accumulator build on the same prompt, as in
the loop-step parity tests (deep random-init cores amplify rounding)."""
import sys

import numpy as np
import pytest
import torch

import cdbgen
import oracle
import paper_2608_09444_amd as cdb

pytestmark = pytest.mark.gpu

TOL_MAX, TOL_MEAN = 2e-2, 2e-3
DRIFT_FACTOR = 1.25  # bound: this times the fp32-accumulator oracle's distance from the fp64 oracle

# 18 q/k/v stripes, 6 output stripes, 5 vocabulary stripes: tiles that do not
# divide the 128-column workgroup tile; adapter and convergence score
ODD = cdbgen.ModelShape(name="odd-1-2-1-inj", d=192, n_heads=3, head_dim=64, d_ff=96, vocab=160, n_prelude=1,
                        n_core=2, n_coda=1, r_max=3, injection=1, exit_kind=1)


# head_dim 96 with 5 heads: 15 stripes per q/k/v part, an odd count, so one
# wave's stripe pair in the tile kernel straddles the q/k boundary (the
# Huginn-shaped 55 x 96 heads have 165 per part)
HD96 = cdbgen.ModelShape(name="hd96-1-2-1-inj", d=480, n_heads=5, head_dim=96, d_ff=256, vocab=320, n_prelude=1,
                         n_core=2, n_coda=1, r_max=2, injection=1, exit_kind=1)


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _core_prefix(shape, w, n_core, **kw):
    s = cdbgen.shrink(shape, n_core=n_core, **kw)
    L = shape.n_prelude
    layers = w["layers"][:L + n_core] + w["layers"][L + shape.n_core:]
    return s, dict(w, layers=layers)


def oracle_block(shape, w, prompt, acc32=False):
    """The prompt as one block through the oracle's paged stage operators."""
    R = shape.r_max
    P = len(prompt)
    pages = cdbgen.pages_for(P)
    om = oracle.Model(shape, w, bf16_storage=True, acc32=acc32)
    op = oracle.Paged(shape, 1, pages, pages if shape.n_prelude else 0, pages * R, pages if shape.n_coda else 0)
    nxt = {0: 0, 1: 0, 2: 0}
    for pg in range(pages):
        for plane in range(R + 2):
            stg = 0 if plane == 0 else (2 if plane == R + 1 else 1)
            if stg == 0 and not shape.n_prelude or stg == 2 and not shape.n_coda:
                continue
            op.page_table[0, plane, pg] = nxt[stg]
            nxt[stg] += 1
    pos = np.arange(P, dtype=np.int32)
    seq = np.zeros(P, np.int32)
    oh = np.zeros((P, shape.d))
    oe = np.zeros((P, shape.d)) if shape.injection else None
    oracle.prelude(om, op, oh, oe, pos, seq, pos, prompt)
    for c in range(R):
        oracle.loop_step(om, op, oh, oe, pos, seq, pos, np.full(P, c, np.int32), np.full(P, R, np.int32))
    ologits, oids = oracle.coda(om, op, oh, pos, seq, pos)
    return op, ologits, oids


def run_prefill(shape, w, prompt, chunks, check_rows=None, sensitivity=False):
    R = shape.r_max
    P = len(prompt)
    assert sum(chunks) == P
    pages = cdbgen.pages_for(P)
    op, ologits, oids = oracle_block(shape, w, prompt)
    tol_max, tol_mean, kv_tol = TOL_MAX, TOL_MEAN, TOL_MAX
    if sensitivity:
        op32, ol32, _ = oracle_block(shape, w, prompt, acc32=True)
        dl = np.abs(ol32 - ologits)
        tol_max = max(TOL_MAX, DRIFT_FACTOR * float(dl.max()))
        tol_mean = max(TOL_MEAN, DRIFT_FACTOR * float(dl.mean()))
        kv_tol = max(TOL_MAX, DRIFT_FACTOR * max(float(np.abs(a - b).max()) for a, b in
                                        ((op32.pre, op.pre), (op32.core, op.core), (op32.coda, op.coda))))
    gkv = cdb.PagedKV(shape, 1, pages, pages, pages * R, pages)
    gkv.page_table.copy_(torch.from_numpy(op.page_table))
    # device: the chunks in order
    gm = cdb.DeviceModel(shape, w)
    ws = cdb.Workspace(gm.desc, max(chunks))
    glogits = np.zeros((P, shape.vocab), np.float32)
    gids = np.zeros(P, np.int32)
    p0 = 0
    for n in chunks:
        tok = torch.as_tensor(prompt[p0:p0 + n], dtype=torch.int32, device="cuda")
        lg = torch.empty((n, shape.vocab), dtype=torch.float32, device="cuda")
        ids = torch.empty(n, dtype=torch.int32, device="cuda")
        cdb.cdb_prefill(gm.model, gkv.c, 0, p0, tok, lg, ids, ws.buf)
        torch.cuda.synchronize()
        glogits[p0:p0 + n] = lg.cpu().numpy()
        gids[p0:p0 + n] = ids.cpu().numpy()
        p0 += n
    assert cdb.cdb_read_device_error(ws.buf) == 0
    rows = np.arange(P) if check_rows is None else np.asarray(check_rows)
    d = np.abs(glogits[rows] - ologits[rows])
    err = {"logit_max": float(d.max()), "logit_mean": float(d.mean()), "bound": (tol_max, tol_mean)}
    assert err["logit_max"] <= tol_max and err["logit_mean"] <= tol_mean, err
    checked = 0
    for i in rows:
        top2 = np.sort(ologits[i])[-2:]
        if top2[1] - top2[0] > 2 * tol_max:
            assert gids[i] == oids[i], f"row {i}"
            checked += 1
        else:
            assert ologits[i][gids[i]] >= top2[1] - 2 * tol_max
    # K/V of every plane at the checked positions
    kv_max = 0.0
    for plane in range(R + 2):
        if plane == 0:
            gp, opool = gkv.pre, op.pre
        elif plane == R + 1:
            gp, opool = gkv.coda, op.coda
        else:
            gp, opool = gkv.core, op.core
        if opool.shape[1] == 0 or int(op.page_table[0, plane, 0]) < 0:
            continue
        for t in rows:
            pid = int(op.page_table[0, plane, t // 16])
            g = gp[:, pid, :, :, t % 16, :].float().cpu().numpy()
            o = opool[pid, :, :, :, t % 16, :]
            dd = np.abs(g - o)
            kv_max = max(kv_max, float(dd.max()))
            assert not (dd > np.maximum(kv_tol, np.abs(o) * 2.0 ** -7 * 1.001)).any(), (plane, t)
    err["kv_max"] = kv_max
    err["ids_checked"] = checked
    return err


def test_prefill_tiny_tile_and_skinny_chunks():
    s = cdbgen.TINY
    w = cdbgen.model_weights(s)
    prompt = cdbgen.prompt_ids(s.vocab, 1, 340, seed=80)[0]
    _say(f"[gpu] prefill {s.name}: chunks 300 (tile GEMMs) + 40")
    err = run_prefill(s, w, prompt, [300, 40])
    _say(f"[gpu]   {err}")
    assert err["ids_checked"] > 100


def test_prefill_ragged_tiles_with_injection():
    s = ODD
    w = cdbgen.model_weights(s)
    prompt = cdbgen.prompt_ids(s.vocab, 1, 290, seed=81)[0]
    _say(f"[gpu] prefill {s.name}: one chunk of 290")
    err = run_prefill(s, w, prompt, [290])
    _say(f"[gpu]   {err}")


def test_prefill_ouro_width_two_core_layers():
    s, w = _core_prefix(cdbgen.OURO, cdbgen.model_weights(cdbgen.OURO), 2)
    prompt = cdbgen.prompt_ids(s.vocab, 1, 320, seed=82)[0]
    _say(f"[gpu] prefill Ouro widths, 2 core layers: one chunk of 320")
    err = run_prefill(s, w, prompt, [320], check_rows=[0, 1, 15, 16, 127, 128, 200, 255, 256, 300, 319],
                      sensitivity=True)
    _say(f"[gpu]   {err}")


def test_prefill_huginn_width_head_dim_96():
    s, w = _core_prefix(cdbgen.HUGINN, cdbgen.model_weights(cdbgen.HUGINN), 1, r_max=2)
    prompt = cdbgen.prompt_ids(s.vocab, 1, 40, seed=83)[0]
    _say(f"[gpu] prefill Huginn widths (2-1-2, r_max 2): chunks 24 + 16")
    err = run_prefill(s, w, prompt, [24, 16], sensitivity=True)
    _say(f"[gpu]   {err}")


def test_prefill_ouro_width_second_chunk_over_earlier_context():
    # the second chunk's rows attend to 320 earlier positions and to each
    # other: key blocks stream from two chunks' pages, every wave takes several
    s, w = _core_prefix(cdbgen.OURO, cdbgen.model_weights(cdbgen.OURO), 2)
    prompt = cdbgen.prompt_ids(s.vocab, 1, 620, seed=84)[0]
    _say(f"[gpu] prefill Ouro widths, 2 core layers: chunks 320 + 300")
    err = run_prefill(s, w, prompt, [320, 300], check_rows=[0, 319, 320, 321, 400, 511, 512, 600, 619],
                      sensitivity=True)
    _say(f"[gpu]   {err}")


def test_prefill_ouro_width_full_chunk_then_short_chunk():
    # the largest chunk (128-row q/k/v tiles), then a skinny chunk over its 512 positions
    s, w = _core_prefix(cdbgen.OURO, cdbgen.model_weights(cdbgen.OURO), 2)
    prompt = cdbgen.prompt_ids(s.vocab, 1, 552, seed=85)[0]
    _say(f"[gpu] prefill Ouro widths, 2 core layers: chunks 512 + 40")
    err = run_prefill(s, w, prompt, [512, 40], check_rows=[0, 1, 127, 128, 255, 256, 383, 384, 500, 511, 512, 530, 551],
                      sensitivity=True)
    _say(f"[gpu]   {err}")


def test_prefill_head_dim_96_odd_stripes_per_part():
    s = HD96
    w = cdbgen.model_weights(s)
    prompt = cdbgen.prompt_ids(s.vocab, 1, 300, seed=86)[0]
    _say(f"[gpu] prefill {s.name}: chunks 264 (tile GEMMs) + 36")
    err = run_prefill(s, w, prompt, [264, 36])
    _say(f"[gpu]   {err}")
