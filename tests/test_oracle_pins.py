"""Pins of the CPU oracle against facts that do not come from the oracle itself:
closed forms, library routines, a textbook unrolled transformer, brute force,
and the paper's worked examples.  CPU only."""
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import cdbgen
import oracle
from oracle import executor

GOLD = os.path.join(os.path.dirname(__file__), "golden")

# small shapes that keep every code path (prelude, core, coda, injection)
SMALL = cdbgen.shrink(cdbgen.TINY, name="small-1-2-1", d=64, n_heads=2, head_dim=32, d_ff=96, vocab=61, r_max=3)
SMALL_INJ = cdbgen.shrink(SMALL, name="small-inj-2-2-1", n_prelude=2, injection=1, exit_kind=1, r_max=4)


def weights(shape, seed=0):
    return cdbgen.model_weights(shape, seed=seed)


def f64(bits):
    return torch.from_numpy(cdbgen.bf16_to_f32(bits).astype(np.float64))


# ---------------------------------------------------------------- closed forms

def test_bf16_rounding_known_values():
    assert oracle.to_bf16(1.0) == 1.0
    assert oracle.to_bf16(1.0 + 2 ** -8) == 1.0  # tie, rounds to even
    assert oracle.to_bf16(1.0 + 3 * 2 ** -8) == 1.0 + 2 ** -6  # tie, rounds up to even
    assert oracle.to_bf16(1.0 + 3 * 2 ** -9) == 1.0 + 2 ** -7
    assert oracle.to_bf16(-2.5) == -2.5
    x = 0.1234567
    assert abs(oracle.to_bf16(x) - x) <= x * 2 ** -9


def test_rmsnorm_closed_form():
    for c in (3.0, -0.5, 1e-3):
        y = oracle.rmsnorm(np.full(16, c), 1e-6)
        assert np.allclose(y, c / math.sqrt(c * c + 1e-6), rtol=1e-15, atol=0)
    x = np.random.default_rng(0).standard_normal(100)
    y = oracle.rmsnorm(x, 0.0)
    assert math.isclose(np.mean(y * y), 1.0, rel_tol=1e-12)
    assert np.allclose(y, F.rms_norm(torch.from_numpy(x), (100,), eps=0.0).numpy(), rtol=1e-13)


def test_rope_is_a_rotation_by_pos_times_frequency():
    # head_dim 2: a single pair rotated by exactly `pos` radians (base^0 = 1)
    for pos in (0, 1, 7, 513):
        v = oracle.rope(np.array([0.3, -1.2]), 1, 2, pos, 10000.0)
        c, s = math.cos(pos), math.sin(pos)
        assert np.allclose(v, [0.3 * c + 1.2 * s, -1.2 * c + 0.3 * s], rtol=0, atol=1e-14)
    # norm preserved per pair, and q(m).k(n) depends on m - n only
    g = np.random.default_rng(1)
    q, k = g.standard_normal(128), g.standard_normal(128)
    for m, n in ((5, 2), (103, 100), (700, 697)):
        a = oracle.rope(q, 1, 128, m, 10000.0) @ oracle.rope(k, 1, 128, n, 10000.0)
        b = oracle.rope(q, 1, 128, 3, 10000.0) @ oracle.rope(k, 1, 128, 0, 10000.0)
        assert math.isclose(a, b, rel_tol=1e-9, abs_tol=1e-9)
    r = oracle.rope(q, 2, 64, 37, 10000.0)
    for h in range(2):
        x, y = q[64 * h:64 * h + 64], r[64 * h:64 * h + 64]
        assert np.allclose(x[:32] ** 2 + x[32:] ** 2, y[:32] ** 2 + y[32:] ** 2, rtol=1e-12)


def test_attention_special_cases_and_library():
    g = np.random.default_rng(2)
    q = g.standard_normal(32)
    v = g.standard_normal((1, 32))
    assert np.allclose(oracle.attend(q, g.standard_normal((1, 32)), v), v[0], rtol=1e-15)
    k_same = np.tile(g.standard_normal(32), (5, 1))
    vs = g.standard_normal((5, 32))
    assert np.allclose(oracle.attend(q, k_same, vs), vs.mean(0), rtol=1e-12)
    K, V = g.standard_normal((40, 32)), g.standard_normal((40, 32))
    ref = F.scaled_dot_product_attention(torch.from_numpy(q)[None, None, None], torch.from_numpy(K)[None, None],
                                         torch.from_numpy(V)[None, None])[0, 0, 0].numpy()
    assert np.allclose(oracle.attend(q, K, V), ref, rtol=1e-12, atol=1e-13)


def test_silu_identities():
    assert oracle.silu(0.0) == 0.0
    for x in (-3.0, -0.2, 0.7, 5.0):
        assert math.isclose(oracle.silu(x) - oracle.silu(-x), x, rel_tol=1e-13)
        assert math.isclose(oracle.silu(x), F.silu(torch.tensor(x, dtype=torch.float64)).item(), rel_tol=1e-14)
    assert math.isclose(oracle.silu(40.0), 40.0, rel_tol=1e-15)


# ------------------------------------------------ textbook unrolled transformer

def unrolled_reference(shape, w, tokens, bf16=False):
    """Fixed depth r_max as a plain weight-tied transformer over the whole
    sequence at once: layers [prelude, (adapter,) core x r_max, coda], causal
    library attention, complex-number RoPE.  Returns logits, per-loop states.

    bf16: round to bf16 (torch's own conversion, through fp32 as a device that
    computes in fp32 does) exactly where the model keeps values in bf16: the
    normalised input of every projection (q/k/v, gate/up, LM head), K and V
    after RoPE, the attention output, the SwiGLU product and the adapter input
    [h; e].  Everything else stays fp64."""
    s = shape

    def st(x):
        return x.to(torch.float32).to(torch.bfloat16).to(torch.float64) if bf16 else x
    T = len(tokens)
    d, H, hd = s.d, s.n_heads, s.head_dim
    pos = torch.arange(T, dtype=torch.float64)
    half = hd // 2
    theta = s.rope_base ** (-2.0 * torch.arange(half, dtype=torch.float64) / hd)
    rot = torch.polar(torch.ones(T, half, dtype=torch.float64), pos[:, None] * theta[None, :])

    def rope(x):  # [T, H, hd]
        z = torch.complex(x[..., :half], x[..., half:]) * rot[:, None, :]
        return torch.cat([z.real, z.imag], dim=-1)

    def rms(x):
        return F.rms_norm(x, (x.shape[-1],), eps=s.rms_eps)

    def layer(x, L):
        lw = {k: f64(v) for k, v in w["layers"][L].items()}
        n = st(rms(x))
        q = rope((n @ lw["q"].T).view(T, H, hd)).transpose(0, 1)
        k = st(rope((n @ lw["k"].T).view(T, H, hd))).transpose(0, 1)
        v = st((n @ lw["v"].T).view(T, H, hd)).transpose(0, 1)
        o = st(F.scaled_dot_product_attention(q, k, v, is_causal=True).transpose(0, 1).reshape(T, d))
        x = x + o @ lw["o"].T
        n = st(rms(x))
        return x + st(F.silu(n @ lw["gate"].T) * (n @ lw["up"].T)) @ lw["down"].T

    x = f64(w["embed"])[torch.as_tensor(tokens, dtype=torch.long)]
    for L in range(s.n_prelude):
        x = layer(x, L)
    e = x
    states = [x]
    for _ in range(s.r_max):
        u = x if not s.injection else st(torch.cat([x, e], dim=-1)) @ f64(w["adapter"]).T
        for l in range(s.n_core):
            u = layer(u, s.n_prelude + l)
        x = u
        states.append(x)
    for l in range(s.n_coda):
        x = layer(x, s.n_prelude + s.n_core + l)
    logits = st(rms(x)) @ f64(w["lm_head"]).T
    return logits.numpy(), [t.numpy() for t in states]


@pytest.mark.parametrize("shape", [SMALL, SMALL_INJ], ids=lambda s: s.name)
def test_fixed_depth_equals_unrolled_weight_tied_transformer(shape):
    w = weights(shape)
    m = oracle.Model(shape, w, bf16_storage=False)
    T = 11
    tokens = cdbgen.prompt_ids(shape.vocab, 1, T, seed=5)[0]
    depth = np.full(T, shape.r_max, dtype=np.int32)
    got = m.ref_sequence(tokens, depth)
    logits, states = unrolled_reference(shape, w, tokens)
    assert np.abs(got["logits"] - logits).max() < 1e-10
    assert np.abs(got["h"] - states[-1]).max() < 1e-10
    # exit scores after every loop (sigmoid gate or L2 convergence distance)
    for r in range(1, shape.r_max + 1):
        if shape.exit_kind == 1:
            want = np.linalg.norm(states[r] - states[r - 1], axis=1)
        else:
            n = F.rms_norm(torch.from_numpy(states[r]), (shape.d,), eps=shape.rms_eps).numpy()
            want = 1.0 / (1.0 + np.exp(-(n @ cdbgen.bf16_to_f32(w["w_exit"]).astype(np.float64))))
        assert np.allclose(got["scores"][:, r - 1], want, rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("shape", [SMALL, SMALL_INJ], ids=lambda s: s.name)
def test_bf16_storage_rounds_where_the_unrolled_transformer_does(shape):
    """The oracle's bf16-storage mode (the mode the device is graded against)
    equals the unrolled transformer with torch's bf16 conversion applied at the
    model's storage points, and differs from the unrounded model: a rounding
    point dropped from or added to the oracle moves its logits by ~1e-3."""
    w = weights(shape)
    T = 11
    tokens = cdbgen.prompt_ids(shape.vocab, 1, T, seed=5)[0]
    depth = np.full(T, shape.r_max, dtype=np.int32)
    got = oracle.Model(shape, w, bf16_storage=True).ref_sequence(tokens, depth)
    logits, states = unrolled_reference(shape, w, tokens, bf16=True)
    assert np.abs(got["logits"] - logits).max() <= 1e-10
    assert np.abs(got["h"] - states[-1]).max() <= 1e-10
    exact, _ = unrolled_reference(shape, w, tokens, bf16=False)
    assert np.abs(got["logits"] - exact).max() > 1e-4


def test_argmax_takes_the_lowest_index_on_ties():
    """Greedy ties: copying the winning LM-head row to a lower and a higher
    index makes an exact three-way tie; the oracle's greedy id is the lowest
    of them, as numpy's argmax (first occurrence) gives."""
    shape = SMALL
    w = weights(shape)
    T = 6
    tokens = cdbgen.prompt_ids(shape.vocab, 1, T, seed=14)[0]
    depth = np.full(T, shape.r_max, dtype=np.int32)
    ids = oracle.Model(shape, w, bf16_storage=True).ref_sequence(tokens, depth)["logits"].argmax(axis=1)
    for t in range(T - 1):
        win = int(ids[t])
        lo, hi = (win - 1 - t) % shape.vocab, (win + 1 + t) % shape.vocab
        lm = w["lm_head"].copy()
        lm[lo] = lm[win]
        lm[hi] = lm[win]
        ww = dict(w, lm_head=lm)
        # positions <= t given, so the states are those of the first run; id t + 1 is greedy
        res = oracle.Model(shape, ww, bf16_storage=True).ref_sequence(tokens, depth, n_given=t + 1)
        row = res["logits"][t]
        tied = np.flatnonzero(row == row.max()).tolist()
        assert tied == sorted({lo, win, hi})
        assert res["tokens"][t + 1] == tied[0] == int(np.argmax(row))


def test_fixed_depth_bf16_storage_stays_near_exact():
    w = weights(SMALL)
    T = 9
    tokens = cdbgen.prompt_ids(SMALL.vocab, 1, T, seed=6)[0]
    depth = np.full(T, SMALL.r_max, dtype=np.int32)
    a = oracle.Model(SMALL, w, bf16_storage=False).ref_sequence(tokens, depth)
    b = oracle.Model(SMALL, w, bf16_storage=True).ref_sequence(tokens, depth)
    diff = np.abs(a["logits"] - b["logits"])
    assert 0 < diff.max() < 5e-2  # rounding happens, and stays at bf16 scale


@pytest.mark.parametrize("shape", [SMALL, SMALL_INJ], ids=lambda s: s.name)
def test_fp32_realizations_are_distinct_fp32_implementations(shape):
    """The fp32-accumulator builds that size tolerances (projection sums in
    index order, in reverse, in blocks of 32) each stay within fp32 rounding of
    the fp64 oracle and differ from one another: three distinct fp32
    implementations of the same arithmetic.  The fp64 oracle exists in one
    summation order only."""
    w = weights(shape)
    T = 9
    tokens = cdbgen.prompt_ids(shape.vocab, 1, T, seed=7)[0]
    depth = np.full(T, shape.r_max, dtype=np.int32)
    ref = oracle.Model(shape, w, bf16_storage=False).ref_sequence(tokens, depth)["logits"]
    scale = float(np.abs(ref).max())
    outs = [oracle.Model(shape, w, bf16_storage=False, acc32=True, sum_order=k).ref_sequence(tokens, depth)["logits"]
            for k in (0, 1, 2)]
    for o in outs:
        d = float(np.abs(o - ref).max())
        assert 0 < d < 1e-4 * scale
    for a in range(3):
        for b in range(a + 1, 3):
            assert not np.array_equal(outs[a], outs[b])
    with pytest.raises(ValueError):
        oracle.Model(shape, w, sum_order=1)


# ----------------------------------------------------- brute force (no cache)

@pytest.mark.parametrize("bf16", [False, True])
@pytest.mark.parametrize("shape", [SMALL, SMALL_INJ], ids=lambda s: s.name)
def test_cached_reference_equals_brute_force(shape, bf16):
    w = weights(shape)
    m = oracle.Model(shape, w, bf16_storage=bf16)
    T = 9
    tokens = cdbgen.prompt_ids(shape.vocab, 1, T, seed=7)[0]
    depth = cdbgen.draw_depths(("uniform", 1, shape.r_max), T, shape.r_max, seed=8)
    assert len(set(depth.tolist())) > 1
    ref = m.ref_sequence(tokens, depth)
    bru = m.brute_force(tokens, depth)
    assert np.abs(ref["logits"] - bru["logits"]).max() <= 1e-12
    assert np.abs(ref["h"] - bru["h"]).max() <= 1e-12
    assert np.allclose(ref["scores"], bru["scores"], rtol=0, atol=1e-12, equal_nan=True)


def test_depths_change_the_result():
    # a plausible mistake -- ignoring the depth table -- would make these equal
    w = weights(SMALL)
    m = oracle.Model(SMALL, w, bf16_storage=False)
    tokens = cdbgen.prompt_ids(SMALL.vocab, 1, 6, seed=9)[0]
    a = m.ref_sequence(tokens, np.array([3, 3, 1, 3, 3, 3], np.int32))
    b = m.ref_sequence(tokens, np.array([3, 3, 3, 3, 3, 3], np.int32))
    assert np.abs(a["logits"][:2] - b["logits"][:2]).max() == 0  # causal: earlier positions untouched
    assert np.abs(a["logits"][2:] - b["logits"][2:]).max() > 1e-6


# ---------------------------------------------------------- Fig. 2 worked example

def test_fig2_last_exited_cache_contents():
    gold = json.load(open(os.path.join(GOLD, "fig2_last_exited.json")))
    shape = cdbgen.shrink(SMALL, r_max=gold["r_max"])
    m = oracle.Model(shape, weights(shape), bf16_storage=False)
    depth = np.array(gold["exit_depths"], dtype=np.int32)
    tokens = cdbgen.prompt_ids(shape.vocab, 1, len(depth), seed=10)[0]
    kv = m.ref_sequence(tokens, depth, want_kv=True)["core_kv"]  # [T][plane][layer][2][d]
    R = shape.r_max
    stored = np.zeros((R, len(depth)), dtype=int)
    for s in range(len(depth)):
        for p in range(R):
            same = [L for L in range(p + 1) if np.array_equal(kv[s, p], kv[s, L])]
            stored[p, s] = same[0] + 1
        # planes up to the exit hold distinct computed states
        for a in range(depth[s]):
            for b in range(a):
                assert not np.array_equal(kv[s, a], kv[s, b])
    assert stored.tolist() == gold["last_exited_rows_are_depth_slots_1_to_3_cols_are_tokens"]


# ---------------------------------------------- batched executor invariances

@pytest.mark.parametrize("bf16", [False, True])
@pytest.mark.parametrize("shape", [SMALL, SMALL_INJ], ids=lambda s: s.name)
def test_mixed_depth_batch_equals_each_sequence_alone(shape, bf16):
    w = weights(shape)
    m = oracle.Model(shape, w, bf16_storage=bf16)
    plens, ndec = [5, 3, 7], [6, 4, 5]
    prompts = [cdbgen.prompt_ids(shape.vocab, 1, p, seed=11, stream=i)[0] for i, p in enumerate(plens)]
    depths = []
    for i, (p, n) in enumerate(zip(plens, ndec)):
        dd = cdbgen.draw_depths(("uniform", 1, shape.r_max), n, shape.r_max, seed=12, stream=i)
        depths.append(np.concatenate([np.full(p, shape.r_max, np.int32), dd]))
    got = executor.run(m, prompts, ndec, depths, max_batch=2)
    for q in range(3):
        alone = m.ref_sequence(np.concatenate([prompts[q], np.zeros(ndec[q], np.int32)]), depths[q],
                               n_given=plens[q])
        assert np.array_equal(got[q]["tokens"], alone["tokens"])
        assert np.array_equal(got[q]["logits"], alone["logits"])
        assert np.array_equal(got[q]["h"], alone["h"])
        assert np.array_equal(np.isnan(got[q]["scores"]), np.isnan(alone["scores"]))
        ok = ~np.isnan(alone["scores"])
        assert np.array_equal(got[q]["scores"][ok], alone["scores"][ok])


def test_zero_exits_equals_fixed_depth_unrolled():
    shape = SMALL
    w = weights(shape)
    m = oracle.Model(shape, w, bf16_storage=False)
    plens, ndec = [4, 6], [3, 2]
    prompts = [cdbgen.prompt_ids(shape.vocab, 1, p, seed=13, stream=i)[0] for i, p in enumerate(plens)]
    depths = [np.full(p + n, shape.r_max, np.int32) for p, n in zip(plens, ndec)]
    got = executor.run(m, prompts, ndec, depths, max_batch=3)
    for q in range(2):
        logits, _ = unrolled_reference(shape, w, got[q]["tokens"])
        assert np.abs(got[q]["logits"] - logits).max() < 1e-10


# ------------------------------------------------------ exit mask / compaction

def test_exit_compaction_is_a_stable_partition():
    g = np.random.default_rng(3)
    for n in (0, 1, 5, 64, 300):
        depth = g.integers(1, 5, n).astype(np.int32)
        c = np.floor(g.random(n) * depth).astype(np.int32)
        r = oracle.exit_compact(c, depth, 4)
        ex = [i for i in range(n) if c[i] + 1 == depth[i]]
        assert r["exited"].tolist() == ex
        assert r["cont"].tolist() == [i for i in range(n) if i not in ex]
        assert r["exit_mask"].tolist() == [int(i in ex) for i in range(n)]
        assert r["counts"].tolist() == [n - len(ex), len(ex)]


def test_exit_compaction_rejects_invalid_rows():
    with pytest.raises(ValueError):
        oracle.exit_compact([2], [2], 4)  # c == depth: the row already exited
    with pytest.raises(ValueError):
        oracle.exit_compact([0], [5], 4)  # depth > r_max
    with pytest.raises(ValueError):
        oracle.exit_compact([0], [0], 4)  # depth < 1


def test_loop_step_reports_unmapped_pages():
    shape = SMALL
    m = oracle.Model(shape, weights(shape), bf16_storage=True)
    paged = oracle.Paged(shape, 1, 1, 1, 1, 1)
    h = np.zeros((1, shape.d))
    with pytest.raises(ValueError):
        oracle.loop_step(m, paged, h, None, [0], [0], [0], [0], [2])
