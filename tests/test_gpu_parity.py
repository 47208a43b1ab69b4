"""GPU parity: the HIP stage calls against the CPU oracle, element by element,
on identical seeded inputs.  Integer outputs (exit masks, compaction lists,
counts) must match exactly; hidden states, exit scores and logits within
max-abs 2e-2 / mean-abs 2e-3; K/V entries within one bf16 step."""
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
