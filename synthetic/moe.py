"""Seeded synthetic router outputs for one GRPO prompt group (test data only).

A token-local Top-k MoE router gives every token u a probability row
p[u, :] over E experts and its k selected experts r[u, :].  Under prefix
reuse the P shared prefix tokens exist once physically and stand for N
logical copies; the suffix tokens of the N trajectories exist once each.

Draw order, from one ``numpy.random.default_rng(seed)`` (PCG64) stream:
[ragged groups: the suffix lengths, uniform integers, drawn first], then
router logits for the prefix tokens, then for the packed suffix tokens, all
``standard_normal(dtype=float32)``.  The probability rows are the float64
softmax of the logits rounded once to float32, and r holds the indices of
the k largest logits of each row, largest first (the draws are continuous,
so ties do not occur).  This module holds none of the accounting arithmetic;
the router itself is upstream of the method.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, Optional, Sequence, Tuple

import numpy as np

__all__ = ["RouterShape", "make_router_group", "ROUTER_SHAPES"]


@dataclass(frozen=True)
class RouterShape:
    num_experts: int
    top_k: int
    prefix_len: int
    suffix_lens: Tuple[int, ...]

    @property
    def n(self) -> int:
        return len(self.suffix_lens)


def _router_rows(rng: np.random.Generator, n_tokens: int, e: int, k: int):
    logits = rng.standard_normal(size=(n_tokens, e), dtype=np.float32)
    z = logits.astype(np.float64)
    z = np.exp(z - z.max(axis=1, keepdims=True)) if n_tokens else z
    p = (z / z.sum(axis=1, keepdims=True)).astype(np.float32) if n_tokens else z.astype(np.float32)
    order = np.argsort(-logits, axis=1, kind="stable")[:, :k] if n_tokens else np.zeros((0, k), np.int64)
    return p, order.astype(np.int32)


def make_router_group(shape: RouterShape, seed: int = 0,
                      ragged: Optional[Tuple[int, int]] = None) -> Dict[str, np.ndarray]:
    """Router outputs of one prompt group.

    Returns p_p [P, E] float32, r_p [P, k] int32 for the prefix tokens (one
    physical copy), p_s [T, E], r_s [T, k] for the packed suffix tokens,
    cu_seqlens [N+1] int32, suffix_lens [N] int32 and the shape (with the
    drawn lengths when ragged).
    """
    rng = np.random.default_rng(seed)
    lens = tuple(shape.suffix_lens)
    if ragged is not None:
        lo, hi = ragged
        lens = tuple(int(v) for v in rng.integers(lo, hi + 1, size=len(lens)))
    shp = RouterShape(shape.num_experts, shape.top_k, shape.prefix_len, lens)
    e, k = shp.num_experts, shp.top_k
    p_p, r_p = _router_rows(rng, shp.prefix_len, e, k)
    p_s, r_s = _router_rows(rng, int(sum(lens)), e, k)
    cu = np.zeros(len(lens) + 1, dtype=np.int32)
    cu[1:] = np.cumsum(lens)
    return {"p_p": p_p, "r_p": r_p, "p_s": p_s, "r_s": r_s, "cu_seqlens": cu,
            "suffix_lens": np.asarray(lens, dtype=np.int32), "shape": shp}


# Qwen3-MoE-30B-A3B router: 128 experts, top-8; the group of its attention
# workload (P = 8192, N = 16 suffixes of 128..2048 tokens).
ROUTER_SHAPES: Dict[str, RouterShape] = {
    "qwen3_moe_router_p8192_n16_ragged": RouterShape(128, 8, 8192, (0,) * 16),
    "tiny_router": RouterShape(8, 2, 24, (5, 9, 3)),
}
