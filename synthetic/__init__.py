"""Seeded synthetic inputs for one GRPO prompt group [P||S(1)] ... [P||S(N)].

This module is test data only: it draws random tensors and rounds them to the
storage dtype.  It holds none of the attention arithmetic, so both the fp64
CPU oracle and the GPU path can take their inputs from it without sharing any
code of the method itself.

Workload shape (paper Sec. 2.1, "GRPO Training Anatomy"): a prompt group is N
sequences that share one token-identical prefix of length P; sequence i has
its own suffix of length S_i.  Attention inputs are given directly (no
projections): prefix Q/K/V, per-suffix Q/K/V, and upstream adjoints dO for
every row of every trajectory.

Draw order, from one ``numpy.random.default_rng(seed)`` (PCG64) stream, all
``standard_normal(dtype=float32)``:
  [ragged groups: the suffix lengths, uniform integers, drawn first]
  Q_P, K_P, V_P, then for i = 1..N: Q_S(i), K_S(i), V_S(i), dO_S(i), dO_P(i).
bf16 storage rounds each float32 draw to nearest-even once.

The upstream adjoint of the shared prefix rows seen by the three-phase
schedule is G_Y = sum_i dO_P(i) (paper App. A.4/A.5: the accumulated direct
prefix adjoint).  The synthetic group supplies it as an input, summed exactly
in float64 and rounded once to the storage dtype; the dense baseline consumes
the per-trajectory dO_P(i) instead.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "GroupShape",
    "ragged_suffix_lengths",
    "round_to_bf16",
    "bf16_bits",
    "make_group",
    "NAMED_SHAPES",
]


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even).

    Returns float32 values that are exactly representable in bfloat16.
    Inputs are finite N(0,1) draws, so no NaN/Inf handling is needed.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """uint16 bit patterns of float32 values already representable in bf16."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return (u >> np.uint32(16)).astype(np.uint16)


@dataclass(frozen=True)
class GroupShape:
    """Shape of one prompt group's attention layer.

    num_q_heads / num_kv_heads: GQA heads (q head h reads kv head h // G,
    G = num_q_heads // num_kv_heads); head_dim: d; prefix_len: P;
    suffix_lens: (S_1, ..., S_N); dtype: "f32" or "bf16" storage.
    """

    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    prefix_len: int
    suffix_lens: Tuple[int, ...]
    dtype: str = "bf16"

    @property
    def n(self) -> int:
        return len(self.suffix_lens)

    @property
    def total_suffix(self) -> int:
        return int(sum(self.suffix_lens))

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    def cu_seqlens(self) -> np.ndarray:
        cu = np.zeros(self.n + 1, dtype=np.int32)
        cu[1:] = np.cumsum(np.asarray(self.suffix_lens, dtype=np.int64))
        return cu


def ragged_suffix_lengths(n: int, lo: int, hi: int, seed: int) -> Tuple[int, ...]:
    """N suffix lengths uniform on the integers [lo, hi] (both ends included),
    drawn first from the group's generator stream."""
    rng = np.random.default_rng(seed)
    return tuple(int(v) for v in rng.integers(lo, hi + 1, size=n))


def _draw(rng: np.random.Generator, shape, dtype: str) -> np.ndarray:
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if dtype == "bf16":
        x = round_to_bf16(x)
    elif dtype != "f32":
        raise ValueError(f"unknown dtype {dtype!r}")
    return x


def make_group(
    shape: GroupShape,
    seed: int = 0,
    ragged: Optional[Tuple[int, int]] = None,
    with_prefix_adjoint: bool = True,
) -> Dict[str, np.ndarray]:
    """Draw one prompt group's inputs.

    ragged=(lo, hi): draw the suffix lengths from the same stream first
    (shape.suffix_lens then only fixes N).  Returns float32 arrays holding
    values representable in ``shape.dtype``:
      q_p [P,Hq,d], k_p/v_p [P,Hkv,d];
      q_s/do_s [T,Hq,d], k_s/v_s [T,Hkv,d] packed over suffixes (T = sum S_i);
      do_p [N,P,Hq,d] per-trajectory prefix-row adjoints;
      g_y [P,Hq,d] = dtype-rounding of the float64 sum over i of do_p[i];
      cu_seqlens [N+1] int32; suffix_lens [N] int32.
    """
    rng = np.random.default_rng(seed)
    lens = tuple(shape.suffix_lens)
    if ragged is not None:
        lo, hi = ragged
        lens = tuple(int(v) for v in rng.integers(lo, hi + 1, size=len(lens)))
    shp = GroupShape(shape.num_q_heads, shape.num_kv_heads, shape.head_dim,
                     shape.prefix_len, lens, shape.dtype)
    hq, hkv, d, p = shp.num_q_heads, shp.num_kv_heads, shp.head_dim, shp.prefix_len
    dt = shp.dtype
    q_p = _draw(rng, (p, hq, d), dt)
    k_p = _draw(rng, (p, hkv, d), dt)
    v_p = _draw(rng, (p, hkv, d), dt)
    q_s, k_s, v_s, do_s, do_p = [], [], [], [], []
    for s in lens:
        q_s.append(_draw(rng, (s, hq, d), dt))
        k_s.append(_draw(rng, (s, hkv, d), dt))
        v_s.append(_draw(rng, (s, hkv, d), dt))
        do_s.append(_draw(rng, (s, hq, d), dt))
        if with_prefix_adjoint:
            do_p.append(_draw(rng, (p, hq, d), dt))
        else:
            do_p.append(np.zeros((p, hq, d), dtype=np.float32))
    out = {
        "q_p": q_p, "k_p": k_p, "v_p": v_p,
        "q_s": np.concatenate(q_s, axis=0) if lens else np.zeros((0, hq, d), np.float32),
        "k_s": np.concatenate(k_s, axis=0) if lens else np.zeros((0, hkv, d), np.float32),
        "v_s": np.concatenate(v_s, axis=0) if lens else np.zeros((0, hkv, d), np.float32),
        "do_s": np.concatenate(do_s, axis=0) if lens else np.zeros((0, hq, d), np.float32),
        "do_p": np.stack(do_p, axis=0) if lens else np.zeros((0, p, hq, d), np.float32),
        "cu_seqlens": shp.cu_seqlens(),
        "suffix_lens": np.asarray(lens, dtype=np.int32),
    }
    gy = out["do_p"].astype(np.float64).sum(axis=0).astype(np.float32)
    out["g_y"] = round_to_bf16(gy) if dt == "bf16" else gy
    out["shape"] = shp
    return out


# Workloads, named by what they are.  The paper's own workloads are real GRPO
# batches (RAG, multimodal); these stand in with the paper's model shapes and
# prefix/suffix regimes and N(0,1) data.
NAMED_SHAPES: Dict[str, GroupShape] = {
    # tiny fp32 group: 2 q / 2 kv heads, d=64, P=128, N=4 suffixes of 32
    "tiny_f32": GroupShape(2, 2, 64, 128, (32,) * 4, "f32"),
    # Llama3-8B-shaped attention: GQA 32/8, d=128, P=4096, N=8 x 512
    "llama3_8b_p4096_n8_s512": GroupShape(32, 8, 128, 4096, (512,) * 8, "bf16"),
    # Qwen3-MoE-30B-A3B attention: GQA 32/4, d=128, P=8192, N=16 ragged [128,2048]
    "qwen3_moe_p8192_n16_ragged": GroupShape(32, 4, 128, 8192, (0,) * 16, "bf16"),
    # long-context Llama3-8B layer attention: P=28672, N=8 x 128
    "llama3_8b_p28672_n8_s128": GroupShape(32, 8, 128, 28672, (128,) * 8, "bf16"),
}


def qwen3_sweep_shape(prefix_len: int, n: int) -> GroupShape:
    """Qwen3-8B-shaped attention: GQA 32/8, d=128, suffixes of 1024 tokens."""
    return GroupShape(32, 8, 128, prefix_len, (1024,) * n, "bf16")
