"""Seeded synthetic inputs for continuous depth batching.

This module is shared by the tests, the benchmark, the smoke check and the
oracle's tests.  It holds no arithmetic of the method itself: model shapes,
random weights (drawn in fp32 and stored as bf16 bit patterns), token ids,
per-token exit depths, arrival times, random KV contents and row batches.

Seeds (fixed): weights 0, prompts 1, depths 2, arrivals 3.  Every tensor has its
own stream, derived from (seed, tensor index), so any one tensor can be drawn
without drawing the others.

Shapes follow the paper's two model families (Section 6.1): Ouro 1.4B is fully
looped, 0-24-0 with r_max = 4; Huginn 3.5B is 2-4-2 with an input-injection
adapter and r_max = 32 (its trained maximum, App. C.1).  A tiny 1-2-1 model is
used for exhaustive checks.
"""
from __future__ import annotations

import dataclasses
import math
import os
from typing import Dict, List, Optional

import numpy as np

WEIGHT_SEED, PROMPT_SEED, DEPTH_SEED, ARRIVAL_SEED = 0, 1, 2, 3
PAGE_TOKENS = 16


@dataclasses.dataclass(frozen=True)
class ModelShape:
    name: str
    d: int
    n_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    n_prelude: int
    n_core: int
    n_coda: int
    r_max: int
    injection: int  # 0: none, 1: concat adapter [h; e] -> d
    exit_kind: int  # 0: sigmoid(w_exit . RMSNorm(h)), 1: ||h_new - h_old||_2
    rms_eps: float = 1e-6
    rope_base: float = 10000.0

    @property
    def n_layers(self) -> int:
        return self.n_prelude + self.n_core + self.n_coda


TINY = ModelShape("tiny-1-2-1", 256, 4, 64, 1024, 1024, 1, 2, 1, 4, 0, 0)
OURO = ModelShape("ouro-1.4b-shaped", 2048, 16, 128, 5632, 49152, 0, 24, 0, 4, 0, 0)
HUGINN = ModelShape("huginn-3.5b-shaped", 5280, 55, 96, 17920, 65536, 2, 4, 2, 32, 1, 1)
SHAPES = {s.name: s for s in (TINY, OURO, HUGINN)}


def shrink(shape: ModelShape, **kw) -> ModelShape:
    """A copy of a shape with some fields replaced (reduced test models)."""
    return dataclasses.replace(shape, **kw)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    shape: ModelShape
    n_seqs: int
    prompt: object  # int, or (lo, hi) uniform, or ("lognormal", median, sigma, lo, hi)
    decode: object  # int or ("lognormal", median, sigma, lo, hi)
    depth: tuple  # ("uniform", lo, hi) | ("categorical", {d: p}) | ("lognormal", median, sigma, lo, hi) | ("bimodal", a, b)
    max_batch: int
    arrivals_per_s: Optional[float] = None
    prefill_chunk: Optional[int] = None


OURO_DEPTHS = ("categorical", {1: 0.3, 2: 0.3, 3: 0.2, 4: 0.2})
WORKLOADS = {
    1: Workload("tiny parity: 8 seqs, prompt 32, decode 16", TINY, 8, 32, 16, ("uniform", 1, 4), 8),
    2: Workload("ouro-shaped decode: bs 64, prompt 512, decode 256", OURO, 64, 512, 256, OURO_DEPTHS, 64),
    3: Workload("huginn-shaped decode: bs 128, prompt 256, decode 512", HUGINN, 128, 256, 512,
                ("lognormal", 12.0, 0.5, 4, 32), 128),
    4: Workload("ouro-shaped long context: bs 256, prompt U[2048,4096], decode 128", OURO, 256, (2048, 4096), 128,
                ("bimodal", 1, 4), 256),
    5: Workload("ouro-shaped serving: 2000 requests, Poisson 20/s", OURO, 2000,
                ("lognormal", 300.0, 1.0, 16, 4096), ("lognormal", 400.0, 1.0, 16, 2048), OURO_DEPTHS, 64,
                arrivals_per_s=20.0, prefill_chunk=512),
}


# ------------------------------------------------------------------ helpers

def _rng(seed: int, *stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, *stream])))


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> fp32 values (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


_BLOCK = 1 << 20  # elements per independently seeded block
_POOL = None


def _pool():
    global _POOL
    if _POOL is None:
        from concurrent.futures import ThreadPoolExecutor
        _POOL = ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1))
    return _POOL


def normal_bf16_many(specs) -> List[np.ndarray]:
    """Several N(0, std) tensors, drawn in fp32 and stored as bf16 bits.  Each
    spec is (shape, std, seed, *stream).  A tensor's flat array is cut into
    blocks of 2^20 elements, block b drawn from stream (seed, *stream, b), so the
    values do not depend on how many threads draw them."""
    outs, tasks = [], []
    for spec in specs:
        shape, std, seed, stream = spec[0], spec[1], spec[2], tuple(spec[3:])
        n = int(np.prod(shape))
        out = np.empty(n, dtype=np.uint16)
        outs.append(out.reshape(shape))
        for b in range((n + _BLOCK - 1) // _BLOCK):
            tasks.append((out, n, b, std, seed, stream))

    def fill(t):
        out, n, b, std, seed, stream = t
        lo, hi = b * _BLOCK, min(n, (b + 1) * _BLOCK)
        x = _rng(seed, *stream, b).standard_normal(size=hi - lo, dtype=np.float32)
        x *= np.float32(std)
        out[lo:hi] = bf16_bits(x)

    if len(tasks) <= 1:
        for t in tasks:
            fill(t)
    else:
        list(_pool().map(fill, tasks))
    return outs


def normal_bf16(shape, std: float, seed: int, *stream: int) -> np.ndarray:
    return normal_bf16_many([(shape, std, seed, *stream)])[0]


# ------------------------------------------------------------------ weights

LAYER_TENSORS = ("q", "k", "v", "o", "gate", "up", "down")


def layer_shapes(s: ModelShape) -> Dict[str, tuple]:
    d, F = s.d, s.d_ff
    return {"q": (d, d), "k": (d, d), "v": (d, d), "o": (d, d), "gate": (F, d), "up": (F, d), "down": (d, F)}


def layer_weights(s: ModelShape, layer: int, seed: int = WEIGHT_SEED, std: float = 0.02) -> Dict[str, np.ndarray]:
    """Weights of one transformer layer (index over prelude, core, coda), as
    row-major [out][in] bf16 bit arrays."""
    names = list(layer_shapes(s))
    arrs = normal_bf16_many([(shp, std, seed, 4 + 7 * layer + j) for j, shp in enumerate(layer_shapes(s).values())])
    return dict(zip(names, arrs))


def model_weights(s: ModelShape, seed: int = WEIGHT_SEED, std: float = 0.02) -> Dict[str, object]:
    """All weights of a model, N(0, std) drawn in fp32, stored as bf16 bits."""
    specs = [((s.vocab, s.d), std, seed, 0), ((s.vocab, s.d), std, seed, 1), ((s.d,), std, seed, 2)]
    if s.injection:
        specs.append(((s.d, 2 * s.d), std, seed, 3))
    names = list(layer_shapes(s))
    for L in range(s.n_layers):
        specs += [(shp, std, seed, 4 + 7 * L + j) for j, shp in enumerate(layer_shapes(s).values())]
    arrs = normal_bf16_many(specs)
    w: Dict[str, object] = {"embed": arrs[0], "lm_head": arrs[1], "w_exit": arrs[2],
                            "adapter": arrs[3] if s.injection else None}
    k = 4 if s.injection else 3
    w["layers"] = [dict(zip(names, arrs[k + 7 * L: k + 7 * L + 7])) for L in range(s.n_layers)]
    return w


def param_counts(s: ModelShape) -> Dict[str, int]:
    per_layer = sum(a * b for a, b in layer_shapes(s).values())
    core = s.n_core * per_layer + (2 * s.d * s.d if s.injection else 0)
    return {"per_layer": per_layer, "core": core, "boundary_layers": (s.n_prelude + s.n_coda) * per_layer,
            "embed": s.vocab * s.d, "lm_head": s.vocab * s.d}


# ------------------------------------------------------------------ token ids / depths / arrivals

def prompt_ids(vocab: int, n: int, length: int, seed: int = PROMPT_SEED, stream: int = 0) -> np.ndarray:
    return _rng(seed, stream).integers(0, vocab, size=(n, length), dtype=np.int64).astype(np.int32)


def draw_depths(spec: tuple, size, r_max: int, seed: int = DEPTH_SEED, stream: int = 0) -> np.ndarray:
    """Per-token exit depths in [1, r_max] from a depth spec."""
    g = _rng(seed, stream)
    kind = spec[0]
    if kind == "uniform":
        out = g.integers(spec[1], spec[2] + 1, size=size)
    elif kind == "categorical":
        vals = np.array(sorted(spec[1]), dtype=np.int64)
        p = np.array([spec[1][v] for v in vals], dtype=np.float64)
        out = vals[g.choice(len(vals), size=size, p=p / p.sum())]
    elif kind == "lognormal":
        med, sig, lo, hi = spec[1:]
        x = np.exp(np.log(med) + sig * g.standard_normal(size=size))
        out = np.clip(np.floor(x + 0.5), lo, hi)
    elif kind == "bimodal":
        out = np.where(g.random(size=size) < 0.5, spec[1], spec[2])
    else:
        raise ValueError(kind)
    out = np.asarray(out, dtype=np.int32)
    if out.size and (out.min() < 1 or out.max() > r_max):
        raise ValueError("depth outside [1, r_max]")
    return out


def mean_depth(spec: tuple, r_max: int) -> float:
    """Expected exit depth of a depth spec (exact where closed form, else by a large draw)."""
    if spec[0] == "uniform":
        return (spec[1] + spec[2]) / 2.0
    if spec[0] == "categorical":
        p = spec[1]
        return sum(k * v for k, v in p.items()) / sum(p.values())
    if spec[0] == "bimodal":
        return (spec[1] + spec[2]) / 2.0
    return float(draw_depths(spec, 2_000_000, r_max, seed=12345).mean())


def lengths(spec, n: int, seed: int, stream: int) -> np.ndarray:
    if isinstance(spec, int):
        return np.full(n, spec, dtype=np.int32)
    g = _rng(seed, stream)
    if spec[0] == "lognormal":
        med, sig, lo, hi = spec[1:]
        x = np.exp(np.log(med) + sig * g.standard_normal(size=n))
        return np.clip(np.floor(x + 0.5), lo, hi).astype(np.int32)
    lo, hi = spec
    return g.integers(lo, hi + 1, size=n).astype(np.int32)


def poisson_arrivals(n: int, rate: float, seed: int = ARRIVAL_SEED) -> np.ndarray:
    return np.cumsum(_rng(seed, 0).exponential(1.0 / rate, size=n))


# ------------------------------------------------------------------ KV contents / row batches

def random_kv_bf16(shape, seed: int, stream: int = 0, std: float = 1.0) -> np.ndarray:
    return normal_bf16(shape, std, seed, 1000 + stream)


def random_state(n: int, d: int, seed: int, stream: int = 0, std: float = 1.0) -> np.ndarray:
    return (_rng(seed, 2000 + stream).standard_normal(size=(n, d), dtype=np.float32) * np.float32(std))


def decode_snapshot(n_rows: int, spec: tuple, r_max: int, pos_lo: int, pos_hi: int, seed: int = DEPTH_SEED,
                    stream: int = 7) -> Dict[str, np.ndarray]:
    """One mixed-depth loop-step batch as it stands mid-decode in refill mode:
    row i belongs to sequence i (slot i) at a position drawn from [pos_lo, pos_hi];
    a work item of a token with depth d is d times as frequent as the token, so
    depths are drawn size-biased and the loop index uniformly below the depth."""
    g = _rng(seed, stream)
    base = draw_depths(spec, 200_000, r_max, seed, stream + 1).astype(np.int64)
    counts = np.bincount(base, minlength=r_max + 1).astype(np.float64)
    wts = counts * np.arange(r_max + 1)
    wts /= wts.sum()
    depth = g.choice(r_max + 1, size=n_rows, p=wts).astype(np.int32)
    c = np.floor(g.random(n_rows) * depth).astype(np.int32)
    pos = g.integers(pos_lo, pos_hi + 1, size=n_rows).astype(np.int32)
    idx = np.arange(n_rows, dtype=np.int32)
    return {"slot": idx.copy(), "seq": idx.copy(), "pos": pos, "c": c, "depth": depth}


def pages_for(tokens: int) -> int:
    return (tokens + PAGE_TOKENS - 1) // PAGE_TOKENS
