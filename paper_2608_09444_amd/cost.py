"""Decode FLOP accounting and the FLOP bound on the early-exit speed-up
(Section 5, Eq. 2), used to report measured end-to-end speed-ups next to the
most they could be.

F_r is one core application for one token (2 FLOPs per core weight, the
input-injection adapter included); F_0 is the loop-independent part (prelude
and coda layers, and the LM head; the embedding is a lookup).  With ctx > 0
the attention products over ctx keys (4 * d * ctx per layer) are added.
"""
from __future__ import annotations


def layer_params(shape) -> int:
    d, f = shape.d, shape.d_ff
    return 4 * d * d + 3 * d * f


def core_flops(shape, ctx: int = 0) -> float:
    """F_r: one pass through the core for one token."""
    adapter = 2 * shape.d * shape.d if shape.injection else 0
    return 2.0 * (shape.n_core * layer_params(shape) + adapter) + 4.0 * shape.n_core * shape.d * ctx


def boundary_flops(shape, ctx: int = 0) -> float:
    """F_0: prelude, coda and LM head for one token."""
    nl = shape.n_prelude + shape.n_coda
    return 2.0 * (nl * layer_params(shape) + shape.d * shape.vocab) + 4.0 * nl * shape.d * ctx


def flop_bound(shape, mean_depth: float, ctx: int = 0) -> float:
    """(F_0 + r_max F_r) / (F_0 + d_bar F_r): the largest speed-up adaptive
    depth can give over fixed depth r_max at mean exit depth d_bar."""
    f0, fr = boundary_flops(shape, ctx), core_flops(shape, ctx)
    return (f0 + shape.r_max * fr) / (f0 + mean_depth * fr)
