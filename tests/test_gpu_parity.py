"""GPU parity: the HIP stage calls against the CPU oracle, element by element,
on identical seeded inputs.  Integer outputs (exit masks, compaction lists,
counts) must match exactly.  Hidden states, exit scores and logits must lie
within max-abs 2e-2 / mean-abs 2e-3, or, where larger, within 1.25 times the
largest distance of fp32-level realizations of the oracle from the fp64 oracle
on the same inputs (a random-init core turns rounding-level differences into
bf16 rounding flips that cascade from layer to layer; an fp32 implementation
cannot be expected to sit closer than that).  Every test prints its errors,
relative errors ||dh||/||h|| and the ratio of each error to its bound.  K/V
entries must agree within one bf16 step or that bound."""
import sys

import numpy as np
import pytest

import cdbgen

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _workload_inputs(shape, n_seqs, prompt, n_dec, depth_spec, seed_stream=0):
    prompts = [cdbgen.prompt_ids(shape.vocab, 1, prompt, stream=seed_stream + q)[0] for q in range(n_seqs)]
    depths = []
    for q in range(n_seqs):
        dd = cdbgen.draw_depths(depth_spec, n_dec, shape.r_max, stream=seed_stream + q)
        depths.append(np.concatenate([np.full(prompt, shape.r_max, np.int32), dd]))
    return prompts, depths


def test_config1_tiny_end_to_end():
    from lockstep import Lockstep
    wl = cdbgen.WORKLOADS[1]
    s = wl.shape
    _say(f"[gpu] config 1 {s.name}: {wl.n_seqs} seqs, prompt {wl.prompt}, decode {wl.decode}")
    w = cdbgen.model_weights(s)
    prompts, depths = _workload_inputs(s, wl.n_seqs, wl.prompt, wl.decode, wl.depth)
    ls = Lockstep(s, w, [wl.prompt + wl.decode] * wl.n_seqs, wl.max_batch)
    ls.run(prompts, [wl.decode] * wl.n_seqs, depths)
    _say(f"[gpu] config 1 errors {ls.errors} calls {ls.calls} argmax checked {ls.argmax_checked}")
    assert ls.device_error() == 0
    assert ls.calls["loop"] > wl.decode


def _sample_rows(rows_np, r_max, k=16):
    from lockstep import sample_rows
    return sample_rows(rows_np, r_max, k=k)


def _core_prefix(shape, w, n_core):
    """The same model with only its first n_core core layers (same widths,
    kernels and launch shapes; a shallower core keeps rounding-level
    differences from being amplified layer after layer)."""
    s = cdbgen.shrink(shape, n_core=n_core)
    ww = dict(w)
    ww["layers"] = w["layers"][:shape.n_prelude + n_core] + w["layers"][shape.n_prelude + shape.n_core:]
    return s, ww


@pytest.mark.parametrize("n_core", [2, 24])
def test_config2_loop_step_full_batch_sampled_rows(n_core):
    """The benchmark's launch: 64 mixed-depth rows of the Ouro-shaped model at
    decode positions 512..767; 16 rows checked against the oracle (both rows of
    four attention pairs, every loop index, exiting and continuing rows)."""
    from lockstep import injected_loop_step
    s, w = _core_prefix(cdbgen.OURO, cdbgen.model_weights(cdbgen.OURO), n_core)
    rows = cdbgen.decode_snapshot(64, cdbgen.OURO_DEPTHS, s.r_max, 512, 767, stream=7)
    sample = _sample_rows(rows, s.r_max)
    _say(f"[gpu] config 2 full batch, {n_core} core layers, sampled rows {sample}: c {rows['c'][sample]} "
         f"depth {rows['depth'][sample]}")
    err = injected_loop_step(s, w, rows, sample, sensitivity=True)
    _say(f"[gpu] config 2 ({n_core} core layers) errors {err}")


@pytest.mark.parametrize("n_core", [1, 4])
def test_config3_huginn_loop_step_full_batch_sampled_rows(n_core):
    """128 rows of the Huginn-shaped model (adapter, 55 heads x 96, r_max 32) at
    decode positions 256..767; 16 rows checked against the oracle."""
    from lockstep import injected_loop_step
    s, w = _core_prefix(cdbgen.HUGINN, cdbgen.model_weights(cdbgen.HUGINN), n_core)
    wl = cdbgen.WORKLOADS[3]
    rows = cdbgen.decode_snapshot(128, wl.depth, s.r_max, 256, 767, stream=9)
    sample = _sample_rows(rows, s.r_max)
    _say(f"[gpu] config 3 full batch, {n_core} core layers, sampled rows {sample}: c {rows['c'][sample]} "
         f"depth {rows['depth'][sample]}")
    err = injected_loop_step(s, w, rows, sample, sensitivity=True)
    _say(f"[gpu] config 3 ({n_core} core layers) errors {err}")


def test_config4_long_context_256_rows_sampled():
    """256 rows (the config's batch), 50/50 exits at loop 1 and 4; sampled rows
    sit at long contexts 2048..4223, the others at short ones to bound memory.
    Full 24-layer core."""
    from lockstep import injected_loop_step
    s = cdbgen.OURO
    wl = cdbgen.WORKLOADS[4]
    rows = cdbgen.decode_snapshot(256, wl.depth, s.r_max, 16, 200, stream=11)
    g = np.random.default_rng(3)
    sample = _sample_rows(rows, s.r_max, k=16)
    for i in sample:
        rows["pos"][i] = int(g.integers(2048, 4224))
    _say(f"[gpu] config 4, 256 rows, sampled rows {sample}: pos {rows['pos'][sample]} c {rows['c'][sample]}")
    err = injected_loop_step(s, cdbgen.model_weights(s), rows, sample, sensitivity=True)
    _say(f"[gpu] config 4 errors {err}")


def test_config4_loop_step_as_benched_sampled_rows():
    """The long-context loop step exactly as the benchmark times it: 256 rows,
    every one at a position drawn from [2048, 4223] (prompt U[2048, 4096] +
    decode 128), each row on its own pages (≈ 155 GB of K/V); 16 rows checked
    against the oracle, integer outputs for the whole batch."""
    import torch
    from lockstep import injected_loop_step
    s = cdbgen.OURO
    wl = cdbgen.WORKLOADS[4]
    rows = cdbgen.decode_snapshot(wl.max_batch, wl.depth, s.r_max, wl.prompt[0], wl.prompt[1] + wl.decode - 1,
                                  stream=40)
    sample = _sample_rows(rows, s.r_max, k=16)
    _say(f"[gpu] config 4 as benched, 256 rows at mean context {rows['pos'].mean() + 1:.0f}, sampled rows "
         f"{sample}: pos {rows['pos'][sample]} c {rows['c'][sample]}")
    err = injected_loop_step(s, cdbgen.model_weights(s), rows, sample, sensitivity=True)
    torch.cuda.empty_cache()
    _say(f"[gpu] config 4 as benched errors {err}")


def test_config2_reduced_length_end_to_end():
    """Ouro widths with a 2-layer core, 2 sequences, prompt 16, decode 6, batch
    2; every call checked from the oracle's states (resync)."""
    from lockstep import Lockstep
    s, w = _core_prefix(cdbgen.OURO, cdbgen.model_weights(cdbgen.OURO), 2)
    prompts, depths = _workload_inputs(s, 2, 16, 6, cdbgen.OURO_DEPTHS, seed_stream=20)
    _say(f"[gpu] config 2 reduced end to end, depths {[d[16:].tolist() for d in depths]}")
    ls = Lockstep(s, w, [22, 22], max_batch=2, resync=True, sensitivity=True)
    ls.run(prompts, [6, 6], depths)
    _say(f"[gpu] config 2 reduced errors {ls.errors} oracle self {ls.self_diff} calls {ls.calls}")
    assert ls.device_error() == 0


def test_config3_reduced_depth_end_to_end():
    """Huginn widths (2 prelude + 2 coda layers, adapter, 55 x 96 heads) with a
    1-layer core and r_max 3: 2 sequences, prompt 3, decode 3, batch 2; every call
    checked from the oracle's states (resync)."""
    from lockstep import Lockstep
    s, w = _core_prefix(cdbgen.HUGINN, cdbgen.model_weights(cdbgen.HUGINN), 1)
    s = cdbgen.shrink(s, r_max=3)
    prompts, depths = _workload_inputs(s, 2, 3, 3, ("uniform", 1, 3), seed_stream=30)
    _say(f"[gpu] config 3 reduced-depth end to end, depths {[d[3:].tolist() for d in depths]}")
    ls = Lockstep(s, w, [6, 6], max_batch=2, resync=True, sensitivity=True)
    ls.run(prompts, [3, 3], depths)
    _say(f"[gpu] config 3 reduced errors {ls.errors} oracle self {ls.self_diff} calls {ls.calls}")
    assert ls.device_error() == 0


@pytest.mark.parametrize("case", ["ouro2", "ouro24"])
def test_config2_free_running_decode_at_full_depth(case):
    """Whole decodes at Ouro widths with no resync: 2 sequences, prompt 16,
    decode 6, config 2's depth distribution, states from the embedding of real
    token ids (teacher-forced with the oracle's greedy ids).  ouro24 is the full
    24-layer core at r_max 4.  Each call is bounded by the stored envelope of
    the oracle's own fp32-level realizations run free over the same decode
    (tests/golden/drift_<case>.json, written by make_drift_envelope.py from the
    oracle alone)."""
    _free_run(case)


def test_config3_free_running_decode_at_full_depth():
    """The Huginn-shaped model whole (2 prelude layers, 4 recurrent layers with
    the injection adapter looped up to 32 times, 2 coda layers, vocab 65536)
    decoding with no resync: 2 sequences, prompt 3 (32 loops each), decode 3
    at config 3's lognormal depths, rows of both sequences sharing loop steps
    at different loop indices.  Bounded call by call by the stored envelope of
    the oracle's own fp32-level realizations (tests/golden/drift_huginn4.json)."""
    _free_run("huginn4")


def _free_run(case):
    import json
    import os
    from lockstep import Lockstep
    from oracle_side import free_run_case
    s, w, prompts, depths, n_dec, max_batch = free_run_case(case)
    env = json.load(open(os.path.join(os.path.dirname(__file__), "golden", f"drift_{case}.json")))
    assert env["depths"] == [d.tolist() for d in depths]
    n_prompt = len(prompts[0])
    _say(f"[gpu] free-running {case}: {s.n_core} core layers, depths {[d[n_prompt:].tolist() for d in depths]}")
    ls = Lockstep(s, w, [len(p) + n for p, n in zip(prompts, n_dec)], max_batch=max_batch, envelope=env)
    toks = ls.run(prompts, n_dec, depths)
    assert [t.tolist() for t in toks] == env["tokens"]
    _say(f"[gpu] free-running {case} errors {ls.errors} ratio to bound {ls.ratio} calls {ls.calls} "
         f"one-row calls {ls.single_row} realizations' own spread {env.get('spread')} "
         f"argmax checked {ls.argmax_checked}; oracle fp32 realizations: h {env['run_h_max']:.4g} / "
         f"{env['run_h_mean']:.4g} rel {env['run_h_rel']:.4g}, logits {env['run_logit_max']:.4g} / "
         f"{env['run_logit_mean']:.4g}")
    assert ls.device_error() == 0
