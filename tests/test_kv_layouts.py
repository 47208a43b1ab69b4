"""Pins of the oracle's shared core KV layouts (Section 4.2; App. C.1, Table 1):
the single shared slot and first-then-shared, against brute force (read by
definition, no slot sharing), against the cases where a layout reduces to the
full depth-indexed cache, and against a PyTorch token-by-token decoder.  CPU
only."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import cdbgen
import oracle
from oracle import KV_FIRST_THEN_SHARED, KV_FULL, KV_SHARED, executor

SMALL = cdbgen.shrink(cdbgen.TINY, name="small-1-2-1", d=64, n_heads=2, head_dim=32, d_ff=96, vocab=61, r_max=3)
SMALL_INJ = cdbgen.shrink(SMALL, name="small-inj-2-2-1", n_prelude=2, injection=1, exit_kind=1, r_max=4)
LAYOUTS = [KV_FULL, KV_SHARED, KV_FIRST_THEN_SHARED]
NAMES = {KV_FULL: "full", KV_SHARED: "shared", KV_FIRST_THEN_SHARED: "first-then-shared"}


def run_ref(shape, layout, tokens, depth, bf16=False, w=None, n_prefill=0):
    """Reference run with every token after the first n_prefill decoded one at a time."""
    m = oracle.Model(shape, w if w is not None else cdbgen.model_weights(shape, seed=0), bf16_storage=bf16,
                     kv_layout=layout)
    return m.ref_sequence(tokens, depth, n_prefill=n_prefill)


@pytest.mark.parametrize("n_prefill", [0, 4, 9])
@pytest.mark.parametrize("bf16", [False, True])
@pytest.mark.parametrize("layout", LAYOUTS, ids=NAMES.get)
@pytest.mark.parametrize("shape", [SMALL, SMALL_INJ], ids=lambda s: s.name)
def test_cached_layout_equals_brute_force(shape, layout, bf16, n_prefill):
    w = cdbgen.model_weights(shape, seed=0)
    m = oracle.Model(shape, w, bf16_storage=bf16, kv_layout=layout)
    T = 9
    tokens = cdbgen.prompt_ids(shape.vocab, 1, T, seed=21)[0]
    depth = cdbgen.draw_depths(("uniform", 1, shape.r_max), T, shape.r_max, seed=22)
    assert len(set(depth.tolist())) > 1
    ref = m.ref_sequence(tokens, depth, n_prefill=n_prefill)
    bru = m.brute_force(tokens, depth, n_prefill=n_prefill)
    assert np.abs(ref["logits"] - bru["logits"]).max() <= 1e-12
    assert np.abs(ref["h"] - bru["h"]).max() <= 1e-12
    assert np.allclose(ref["scores"], bru["scores"], rtol=0, atol=1e-12, equal_nan=True)


def test_single_loop_makes_every_layout_the_plain_transformer():
    shape = cdbgen.shrink(SMALL, r_max=1)
    tokens = cdbgen.prompt_ids(shape.vocab, 1, 8, seed=23)[0]
    depth = np.ones(8, np.int32)
    full = run_ref(shape, KV_FULL, tokens, depth)["logits"]
    for layout in (KV_SHARED, KV_FIRST_THEN_SHARED):
        assert np.array_equal(run_ref(shape, layout, tokens, depth)["logits"], full)


def test_first_then_shared_equals_full_at_two_loops():
    # with r_max = 2 the shared second slot only ever holds loop 2 or, after an
    # exit at loop 1, the copied loop-1 state: exactly the full cache
    shape = cdbgen.shrink(SMALL, r_max=2)
    tokens = cdbgen.prompt_ids(shape.vocab, 1, 10, seed=24)[0]
    depth = cdbgen.draw_depths(("uniform", 1, 2), 10, 2, seed=25)
    assert set(depth.tolist()) == {1, 2}
    a = run_ref(shape, KV_FULL, tokens, depth)
    b = run_ref(shape, KV_FIRST_THEN_SHARED, tokens, depth)
    assert np.array_equal(a["logits"], b["logits"])
    c = run_ref(shape, KV_SHARED, tokens, depth)
    assert np.abs(c["logits"] - a["logits"]).max() > 1e-6  # loop 1 reads loop-2 states under one slot


def test_all_exits_after_one_loop_make_shared_equal_full():
    tokens = cdbgen.prompt_ids(SMALL.vocab, 1, 8, seed=26)[0]
    depth = np.ones(8, np.int32)
    full = run_ref(SMALL, KV_FULL, tokens, depth)["logits"]
    for layout in (KV_SHARED, KV_FIRST_THEN_SHARED):
        assert np.array_equal(run_ref(SMALL, layout, tokens, depth)["logits"], full)


def test_layouts_change_the_result_at_three_loops():
    tokens = cdbgen.prompt_ids(SMALL.vocab, 1, 8, seed=27)[0]
    fixed = np.full(8, 3, np.int32)
    outs = {l: run_ref(SMALL, l, tokens, fixed)["logits"] for l in LAYOUTS}
    for a in LAYOUTS:
        for b in LAYOUTS:
            if a < b:
                assert np.abs(outs[a][1:] - outs[b][1:]).max() > 1e-6, (NAMES[a], NAMES[b])
            # position 0 sees only itself: no layout can change it
            assert np.array_equal(outs[a][0], outs[b][0])


def test_prefill_block_reads_the_loop_being_run_under_every_layout():
    # one block run loop by loop: no slot is overwritten before it is read, so
    # the shared layouts read exactly what the full cache holds
    tokens = cdbgen.prompt_ids(SMALL.vocab, 1, 8, seed=32)[0]
    depth = cdbgen.draw_depths(("uniform", 1, 3), 8, 3, seed=33)
    full = run_ref(SMALL, KV_FULL, tokens, depth, n_prefill=8)["logits"]
    assert np.array_equal(full, run_ref(SMALL, KV_FULL, tokens, depth, n_prefill=0)["logits"])
    for layout in (KV_SHARED, KV_FIRST_THEN_SHARED):
        assert np.array_equal(run_ref(SMALL, layout, tokens, depth, n_prefill=8)["logits"], full)


def decoder_reference(shape, w, tokens, depth, read_loop):
    """Token-by-token PyTorch decoder that keeps the K/V of every (token, loop,
    core layer) it computed and, at loop r, gives an earlier token s the loop
    read_loop(r, d_s); library attention, complex-number RoPE.  No prefill block."""
    s = shape
    d, H, hd, half = s.d, s.n_heads, s.head_dim, s.head_dim // 2
    theta = s.rope_base ** (-2.0 * torch.arange(half, dtype=torch.float64) / hd)

    def f64(bits):
        return torch.from_numpy(cdbgen.bf16_to_f32(bits).astype(np.float64))

    def rope(x, t):  # [H, hd]
        z = torch.complex(x[:, :half], x[:, half:]) * torch.polar(torch.ones(half, dtype=torch.float64), t * theta)
        return torch.cat([z.real, z.imag], dim=-1)

    def rms(x):
        return F.rms_norm(x, (x.shape[-1],), eps=s.rms_eps)

    lw = [{k: f64(v) for k, v in L.items()} for L in w["layers"]]
    kv = {}  # (stage, layer, loop, t) -> (k [H, hd], v [H, hd])

    def layer(x, L, key, t, ctx):
        n = rms(x)
        q = rope((n @ lw[L]["q"].T).view(H, hd), t)
        k = rope((n @ lw[L]["k"].T).view(H, hd), t)
        v = (n @ lw[L]["v"].T).view(H, hd)
        kv[key + (t,)] = (k, v)
        K = torch.stack([kv[c][0] for c in ctx] + [k], dim=1)  # [H, t+1, hd]
        V = torch.stack([kv[c][1] for c in ctx] + [v], dim=1)
        o = F.scaled_dot_product_attention(q[:, None, :], K, V).reshape(d)
        x = x + o @ lw[L]["o"].T
        n = rms(x)
        return x + (F.silu(n @ lw[L]["gate"].T) * (n @ lw[L]["up"].T)) @ lw[L]["down"].T

    logits = []
    for t, tok in enumerate(tokens):
        x = f64(w["embed"])[int(tok)]
        for L in range(s.n_prelude):
            x = layer(x, L, ("p", L, 0), t, [("p", L, 0, u) for u in range(t)])
        e = x
        for r in range(1, int(depth[t]) + 1):
            x = x if not s.injection else torch.cat([x, e]) @ f64(w["adapter"]).T
            for l in range(s.n_core):
                ctx = [("c", l, read_loop(r, int(depth[u])), u) for u in range(t)]
                x = layer(x, s.n_prelude + l, ("c", l, r), t, ctx)
        for l in range(s.n_coda):
            L = s.n_prelude + s.n_core + l
            x = layer(x, L, ("o", l, 0), t, [("o", l, 0, u) for u in range(t)])
        logits.append((rms(x) @ f64(w["lm_head"]).T).numpy())
    return np.stack(logits)


READ = {KV_FULL: lambda r, ds: min(r, ds), KV_SHARED: lambda r, ds: ds,
        KV_FIRST_THEN_SHARED: lambda r, ds: 1 if r == 1 else ds}


@pytest.mark.parametrize("layout", LAYOUTS, ids=NAMES.get)
@pytest.mark.parametrize("shape", [SMALL, SMALL_INJ], ids=lambda s: s.name)
def test_layout_matches_pytorch_decoder(shape, layout):
    w = cdbgen.model_weights(shape, seed=0)
    T = 7
    tokens = cdbgen.prompt_ids(shape.vocab, 1, T, seed=28)[0]
    depth = cdbgen.draw_depths(("uniform", 1, shape.r_max), T, shape.r_max, seed=29)
    got = run_ref(shape, layout, tokens, depth, w=w)["logits"]
    want = decoder_reference(shape, w, tokens, depth, READ[layout])
    assert np.abs(got - want).max() < 1e-10


@pytest.mark.parametrize("layout", [KV_SHARED, KV_FIRST_THEN_SHARED], ids=NAMES.get)
def test_aliased_page_tables_give_each_sequence_alone(layout):
    # the batched executor only aliases page-table planes; copy-on-exit and the
    # kernels' reads are unchanged
    shape = SMALL_INJ
    w = cdbgen.model_weights(shape, seed=0)
    m = oracle.Model(shape, w, bf16_storage=True, kv_layout=layout)
    plens, ndec = [5, 18], [6, 4]
    prompts = [cdbgen.prompt_ids(shape.vocab, 1, p, seed=30, stream=i)[0] for i, p in enumerate(plens)]
    depths = []
    for i, (p, n) in enumerate(zip(plens, ndec)):
        dd = cdbgen.draw_depths(("uniform", 1, shape.r_max), n, shape.r_max, seed=31, stream=i)
        depths.append(np.concatenate([np.full(p, shape.r_max, np.int32), dd]))
    got = executor.run(m, prompts, ndec, depths, max_batch=2, kv_layout=layout)
    for q in range(2):
        alone = m.ref_sequence(np.concatenate([prompts[q], np.zeros(ndec[q], np.int32)]), depths[q],
                               n_given=plens[q])
        assert np.array_equal(got[q]["tokens"], alone["tokens"])
        assert np.array_equal(got[q]["logits"], alone["logits"])
