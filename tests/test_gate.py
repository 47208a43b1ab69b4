"""Threshold exits and the lookahead gate (Section 4.3; App. C.2): the oracle's
rule against cases with a known answer and against its own scores, and the
host driver's gated scheduling against a simulated device.  CPU only."""
import numpy as np
import pytest

import cdbgen
import oracle
from paper_2608_09444_amd.driver import TICK_LOOP, Driver

SMALL = cdbgen.shrink(cdbgen.TINY, name="small-1-2-1", d=64, n_heads=2, head_dim=32, d_ff=96, vocab=61, r_max=4)
SMALL_L2 = cdbgen.shrink(SMALL, name="small-l2-2-2-1", n_prelude=2, injection=1, exit_kind=1, r_max=5)
P, N = 5, 6  # prompt tokens, decode tokens


def model(shape):
    return oracle.Model(shape, cdbgen.model_weights(shape, seed=0), bf16_storage=False)


def tokens(shape, seed=60):
    return cdbgen.prompt_ids(shape.vocab, 1, P + N, seed=seed)[0]


def fixed_table(shape, decode_depth):
    return np.concatenate([np.full(P, shape.r_max, np.int32), np.full(N, decode_depth, np.int32)])


def never(shape):
    return 2.0 if shape.exit_kind == 0 else 0.0   # sigmoid < 2; a distance is never < 0


def always(shape):
    return -1.0 if shape.exit_kind == 0 else 1e30


@pytest.mark.parametrize("lookahead", [False, True])
@pytest.mark.parametrize("shape", [SMALL, SMALL_L2], ids=lambda s: s.name)
def test_never_met_threshold_runs_full_depth(shape, lookahead):
    m = model(shape)
    g = m.ref_sequence_gated(tokens(shape), n_given=P + N, threshold=never(shape), lookahead=lookahead,
                             n_prefill=P)
    assert (g["depth"] == shape.r_max).all()
    ref = m.ref_sequence(tokens(shape), fixed_table(shape, shape.r_max), n_prefill=P)
    assert np.array_equal(g["logits"], ref["logits"])


@pytest.mark.parametrize("lookahead", [False, True])
@pytest.mark.parametrize("shape", [SMALL, SMALL_L2], ids=lambda s: s.name)
def test_always_met_threshold_gives_the_minimum_depth(shape, lookahead):
    # gate: depth 1, or 2 with lookahead; convergence (decisions from loop 2): 2, or 3
    m = model(shape)
    g = m.ref_sequence_gated(tokens(shape), n_given=P + N, threshold=always(shape), lookahead=lookahead,
                             n_prefill=P)
    want = (1 if shape.exit_kind == 0 else 2) + (1 if lookahead else 0)
    assert (g["depth"][:P] == shape.r_max).all() and (g["depth"][P:] == want).all()
    ref = m.ref_sequence(tokens(shape), fixed_table(shape, want), n_prefill=P)
    assert np.array_equal(g["logits"], ref["logits"])


@pytest.mark.parametrize("lookahead", [False, True])
@pytest.mark.parametrize("shape", [SMALL, SMALL_L2], ids=lambda s: s.name)
def test_chosen_depths_follow_the_rule_on_their_own_scores(shape, lookahead):
    m = model(shape)
    R = shape.r_max
    tok = tokens(shape, seed=61)
    full = m.ref_sequence(tok, fixed_table(shape, R), n_prefill=P)
    first = 1 if shape.exit_kind == 0 else 2
    thr = float(np.median(full["scores"][P:, first - 1]))  # about half the tokens meet it at the first chance
    g = m.ref_sequence_gated(tok, n_given=P + N, threshold=thr, lookahead=lookahead, n_prefill=P)
    dep = g["depth"]
    assert len(set(dep[P:].tolist())) > 1

    def meets(r, s):
        return r >= first and (s < thr if shape.exit_kind == 1 else s >= thr)

    for t in range(P, P + N):
        d, sc = int(dep[t]), g["scores"][t]
        assert np.isnan(sc[d:]).all() and not np.isnan(sc[:d]).any()
        want = R
        for r in range(1, d + 1):  # the first loop whose score meets the criterion ends the token
            if meets(r, sc[r - 1]):
                want = min(r + (1 if lookahead else 0), R)
                break
        assert d == want, (t, d, want, sc)
    # the gated run is the plain run with the depths it chose
    ref = m.ref_sequence(tok, dep, n_prefill=P)
    assert np.array_equal(g["logits"], ref["logits"])


def test_single_loop_models_always_exit_after_it():
    shape = cdbgen.shrink(SMALL, r_max=1)
    m = model(shape)
    for la in (False, True):
        g = m.ref_sequence_gated(tokens(shape), n_given=P + N, threshold=never(shape), lookahead=la, n_prefill=P)
        assert (g["depth"] == 1).all()


@pytest.mark.parametrize("lookahead", [False, True])
def test_step_rule_matches_the_reference(lookahead):
    # the per-step decisions the batched path uses, fed one token's score
    # sequence, end the token where the dense reference ends it
    shape = SMALL
    m = model(shape)
    tok = tokens(shape, seed=62)
    full = m.ref_sequence(tok, fixed_table(shape, shape.r_max), n_prefill=P)
    thr = float(np.median(full["scores"][P:]))
    g = m.ref_sequence_gated(tok, n_given=P + N, threshold=thr, lookahead=lookahead, n_prefill=P)
    for t in range(P, P + N):
        pend = np.zeros(1, np.uint8)
        for c in range(shape.r_max):
            mask, nxt = m.gate_decide([c], [g["scores"][t, c]], thr, lookahead, pend)
            if mask[0]:
                assert c + 1 == g["depth"][t]
                break
            # known one loop ahead: with lookahead every exit, without it only r_max
            want_next = g["depth"][t] == c + 2 if lookahead else c + 2 == shape.r_max
            assert nxt[0] == int(want_next)


# ------------------------------------------------------ driver, gated mode

def simulate(d, shape, score_of, thr, lookahead):
    """Steps a gated driver with a simulated device that applies the oracle's
    step rule to scores score_of(seq, token, loop).  Returns per-(seq, token)
    loops run."""
    m = model(shape)
    pending = {}
    loops = {}
    prev = None
    while True:
        t = d.next()
        if t is None:
            return loops
        if t.stage == 0:
            d.set_time(t.wait_until)
            continue
        if t.stage == TICK_LOOP:
            n = t.n_rows
            c = np.array([t.c[i] for i in range(n)], np.int32)
            keys = [(t.seq[i], t.decode_index[i]) for i in range(n)]
            sc = np.array([score_of(q, k, int(ci)) for (q, k), ci in zip(keys, c)])
            pend = np.array([pending.get(k, 0) for k in keys], np.uint8)
            mask, nxt = m.gate_decide(c, sc, thr, lookahead, pend)
            for k, p, ci in zip(keys, pend, c):
                pending[k] = int(p)
                loops[k] = max(loops.get(k, 0), int(ci) + 1)
            if lookahead:
                if prev is not None:
                    assert d.loop_result(*prev) == 0
                prev = (t, mask, nxt)
            else:
                assert d.loop_result(t, mask, nxt) == 0
        assert d.complete(t) == 0


@pytest.mark.parametrize("refill", [True, False])
@pytest.mark.parametrize("lookahead", [False, True])
def test_gated_driver_runs_each_token_to_the_rule_depth(lookahead, refill):
    shape = SMALL
    R = shape.r_max
    rng = np.random.default_rng(3)
    n_seq, n_dec = 7, [5, 3, 6, 2, 4, 6, 1]
    table = rng.random((n_seq, 8, R))
    thr = 0.7
    d = Driver(max_batch=4, max_active=5, r_max=R, max_seqs=n_seq, max_pages=2, core_pages=5 * 2 * R,
               refill=refill, gated=True, lookahead=lookahead, threshold=thr)
    for q in range(n_seq):
        d.add_sequence(10, None, n_decode=n_dec[q])
    loops = simulate(d, shape, lambda q, k, c: table[q, k, c], thr, lookahead)
    for q in range(n_seq):
        for k in range(n_dec[q]):
            sc = table[q, k]
            met = [r for r in range(1, R + 1) if sc[r - 1] >= thr]
            want = R
            if met:
                want = min(R, met[0] + (1 if lookahead else 0))
            assert loops[(q, k)] == want, (q, k, sc, loops[(q, k)])
    st = d.stats()
    assert st["tokens"] == sum(n_dec) and st["loop_rows"] == sum(loops.values())


def test_lookahead_completion_needs_the_previous_result():
    d = Driver(max_batch=2, max_active=2, r_max=4, max_seqs=2, max_pages=1, core_pages=8, gated=True,
               lookahead=True, threshold=0.5)
    d.add_sequence(3, None, n_decode=2)
    t = d.next()
    assert d.complete(t) == 0           # prelude
    t1 = d.next()
    assert t1.stage == TICK_LOOP and d.complete(t1) == 0
    t2 = d.next()
    assert t2.stage == TICK_LOOP
    assert d.complete(t2) == -1         # the first loop's result has not been given
    # a result that contradicts the exits applied is refused
    assert d.loop_result(t1, np.ones(t1.n_rows, np.uint8), np.zeros(t1.n_rows, np.uint8)) == -1
