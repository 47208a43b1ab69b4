"""Writes the drift envelopes of the free-running lockstep runs
(tests/golden/drift_<case>.json): per call, how far fp32-level realizations of
the oracle's own arithmetic sit from the fp64 oracle (oracle_side.DriftRun).
Calls only the oracle.  Usage: python tests/golden/make_drift_envelope.py ouro24"""
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path[:0] = [os.path.dirname(HERE), os.path.dirname(os.path.dirname(HERE))]

from oracle_side import DriftRun, free_run_case, run_schedule  # noqa: E402


def spread(calls, key):
    """How far one realization exceeds the largest of the others (leave-one-out),
    at most over the run, among the realizations that have drifted at that call
    (at least a tenth of the call's largest distance; a call with fewer than two
    such is skipped): the device, one more fp32 implementation, may exceed the
    realizations' largest distance by as much."""
    worst = 1.0
    for c in calls:
        each = c.get(key + "_each")
        if not each:
            continue
        top = max(each)
        drifted = [v for v in each if top > 0 and v >= 0.1 * top]
        if len(drifted) < 2:
            continue
        for r, v in enumerate(drifted):
            others = max(drifted[:r] + drifted[r + 1:])
            worst = max(worst, v / others)
    return worst


def main(name):
    s, w, prompts, depths, n_dec, max_batch = free_run_case(name)
    t0 = time.time()
    dr = DriftRun(s, w, [len(p) + n for p, n in zip(prompts, n_dec)])
    toks = run_schedule(dr, prompts, n_dec, depths, s.r_max, max_batch,
                        on_loop=lambda k: print(f"loop call {k}, {time.time() - t0:.0f} s", flush=True))
    out = {"case": name, "model": s.name, "n_core": s.n_core, "r_max": s.r_max,
           "prompts": [p.tolist() for p in prompts], "depths": [d.tolist() for d in depths],
           "tokens": [t.tolist() for t in toks], "calls": dr.calls}
    for key in ("h_max", "h_mean", "h_rel", "logit_max", "logit_mean", "logit_rel", "score_max"):
        vals = [c[key] for c in dr.calls if key in c]
        out["run_" + key] = max(vals) if vals else 0.0
    out["spread"] = {key: spread(dr.calls, key) for key in ("h_max", "logit_max", "score_max")}
    path = os.path.join(HERE, f"drift_{name}.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(f"wrote {path}: " + ", ".join(f"{k} {v:.4g}" for k, v in out.items() if k.startswith("run_")))


if __name__ == "__main__":
    main(sys.argv[1] if len(sys.argv) > 1 else "ouro24")
