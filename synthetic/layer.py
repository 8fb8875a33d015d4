"""Seeded synthetic decoder-layer groups (test data only).

One Llama3-style decoder layer and one GRPO prompt group [P||S(1)]...[P||S(N)]
of layer inputs.  Draw order from one ``numpy.random.default_rng(seed)``
(PCG64) stream, all float32 then rounded to bf16 (ties to even) for bf16
groups: [ragged groups: the suffix lengths], the weights
W_q [hidden, Hq*d], W_k [hidden, Hkv*d], W_v [hidden, Hkv*d],
W_o [Hq*d, hidden], W_gate [hidden, I], W_up [hidden, I], W_down [I, hidden]
(each N(0, std^2)), then the prefix input X_P [P, hidden], then for each
suffix i: X_S(i) [S_i, hidden], dY_S(i) [S_i, hidden], dY_P(i) [P, hidden]
(each N(0, 1)).  Norm gains are one and there are no biases.  The module
holds none of the layer arithmetic.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, Optional, Tuple

import numpy as np

from . import round_to_bf16

__all__ = ["LayerShape", "make_layer_group", "make_stack_group", "LAYER_SHAPES"]


@dataclass(frozen=True)
class LayerShape:
    hidden: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    intermediate: int
    prefix_len: int
    suffix_lens: Tuple[int, ...]
    dtype: str = "bf16"
    rope_theta: float = 500000.0
    norm_eps: float = 1e-5
    weight_std: float = 0.02

    @property
    def n(self) -> int:
        return len(self.suffix_lens)


def make_layer_group(shape: LayerShape, seed: int = 0,
                     ragged: Optional[Tuple[int, int]] = None) -> Dict:
    rng = np.random.default_rng(seed)
    lens = tuple(shape.suffix_lens)
    if ragged is not None:
        lo, hi = ragged
        lens = tuple(int(v) for v in rng.integers(lo, hi + 1, size=len(lens)))
    shp = LayerShape(shape.hidden, shape.num_q_heads, shape.num_kv_heads, shape.head_dim,
                     shape.intermediate, shape.prefix_len, lens, shape.dtype, shape.rope_theta,
                     shape.norm_eps, shape.weight_std)

    def draw(shp_, std=1.0):
        x = rng.standard_normal(size=shp_, dtype=np.float32)
        if std != 1.0:
            x = (x * np.float32(std)).astype(np.float32)
        return round_to_bf16(x) if shp.dtype == "bf16" else x

    h, hq, hkv, d, I = shp.hidden, shp.num_q_heads, shp.num_kv_heads, shp.head_dim, shp.intermediate
    sd = shp.weight_std
    w = {"wq": draw((h, hq * d), sd), "wk": draw((h, hkv * d), sd), "wv": draw((h, hkv * d), sd),
         "wo": draw((hq * d, h), sd), "wg": draw((h, I), sd), "wu": draw((h, I), sd),
         "wd": draw((I, h), sd)}
    x_p = draw((shp.prefix_len, h))
    x_s, dy_s, dy_p = [], [], []
    for s in lens:
        x_s.append(draw((s, h)))
        dy_s.append(draw((s, h)))
        dy_p.append(draw((shp.prefix_len, h)))
    return {"shape": shp, "weights": w, "x_p": x_p, "x_s": x_s, "dy_s": dy_s, "dy_p": dy_p}


def make_stack_group(shape: LayerShape, layers: int, seed: int = 0,
                     ragged: Optional[Tuple[int, int]] = None) -> Dict:
    """A stack of ``layers`` decoder layers of one shape, each with its own
    weights, and one prompt group of inputs to the bottom layer and upstream
    adjoints at the top.  Draw order: [ragged groups: the suffix lengths],
    then for each layer its seven weights in the single-layer order, then
    X_P, then for each suffix X_S(i), dY_S(i), dY_P(i).  Returns the
    single-layer dict with ``weights`` a list (bottom layer first)."""
    rng = np.random.default_rng(seed)
    lens = tuple(shape.suffix_lens)
    if ragged is not None:
        lo, hi = ragged
        lens = tuple(int(v) for v in rng.integers(lo, hi + 1, size=len(lens)))
    shp = LayerShape(shape.hidden, shape.num_q_heads, shape.num_kv_heads, shape.head_dim,
                     shape.intermediate, shape.prefix_len, lens, shape.dtype, shape.rope_theta,
                     shape.norm_eps, shape.weight_std)

    def draw(shp_, std=1.0):
        x = rng.standard_normal(size=shp_, dtype=np.float32)
        if std != 1.0:
            x = (x * np.float32(std)).astype(np.float32)
        return round_to_bf16(x) if shp.dtype == "bf16" else x

    h, hq, hkv, d, I = shp.hidden, shp.num_q_heads, shp.num_kv_heads, shp.head_dim, shp.intermediate
    sd = shp.weight_std
    ws = []
    for _ in range(layers):
        ws.append({"wq": draw((h, hq * d), sd), "wk": draw((h, hkv * d), sd), "wv": draw((h, hkv * d), sd),
                   "wo": draw((hq * d, h), sd), "wg": draw((h, I), sd), "wu": draw((h, I), sd),
                   "wd": draw((I, h), sd)})
    x_p = draw((shp.prefix_len, h))
    x_s, dy_s, dy_p = [], [], []
    for s in lens:
        x_s.append(draw((s, h)))
        dy_s.append(draw((s, h)))
        dy_p.append(draw((shp.prefix_len, h)))
    return {"shape": shp, "layers": layers, "weights": ws, "x_p": x_p, "x_s": x_s, "dy_s": dy_s,
            "dy_p": dy_p}


LAYER_SHAPES: Dict[str, LayerShape] = {
    # Llama3-8B decoder layer, long context: P = 28672, N = 8 x 128
    "llama3_8b_layer_p28672_n8_s128": LayerShape(4096, 32, 8, 128, 14336, 28672, (128,) * 8),
    # the same layer at a prefix the fp64 oracle finishes quickly
    "llama3_8b_layer_p512_n3": LayerShape(4096, 32, 8, 128, 14336, 512, (128, 64, 97)),
    # a small layer for parity across several tiles
    "small_layer": LayerShape(256, 4, 2, 64, 512, 200, (70, 33, 129)),
}
