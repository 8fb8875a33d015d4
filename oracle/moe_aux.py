"""fp64 CPU oracle of the MoE router auxiliary-loss accounting under prefix
reuse (paper Sec. 3.5, Sec. 4.6 and App. B).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The reuse schedule holds each shared prefix token once; for the router's
auxiliary loss it carries a logical multiplicity m_u (N for a prefix token
shared by N trajectories of the reduction scope, 1 for a suffix token).
App. B defines, for a Top-k router with probabilities p[u, e] and selected
experts r[u, j]:

    C_e = sum_u m_u sum_j 1[r[u, j] = e]      (hard count, no gradient)
    R_e = sum_u m_u p[u, e]
    M   = sum_u m_u
    f_e = C_e / (k M),  P_e = R_e / M,  L_aux = lambda E sum_e f_e P_e

and states that these equal the statistics of the materialized batch with N
explicit prefix copies.  With C_e held constant the gradient follows from
the chain rule: dL_aux / dp[u, e] = lambda E f_e m_u / M.
"""
from __future__ import annotations

from typing import Dict

import numpy as np


def logical_stats(p: np.ndarray, r: np.ndarray, m: np.ndarray, n_experts: int):
    """(C, R, M) of App. B over physical tokens with multiplicities m."""
    p = np.asarray(p, dtype=np.float64)
    r = np.asarray(r, dtype=np.int64)
    m = np.asarray(m, dtype=np.int64)
    counts = np.zeros(n_experts, dtype=np.int64)
    # each selected expert of token u adds m_u
    np.add.at(counts, r.reshape(-1), np.repeat(m, r.shape[1]))
    mass = (m.astype(np.float64)[:, None] * p).sum(axis=0) if len(m) else np.zeros(n_experts)
    return counts, mass, int(m.sum())


def aux_loss(counts, mass, total, top_k: int, lam: float):
    """f_e, P_e and L_aux = lambda E sum_e f_e P_e (App. B)."""
    n_experts = len(counts)
    f = np.asarray(counts, dtype=np.float64) / (top_k * total)
    pe = np.asarray(mass, dtype=np.float64) / total
    return f, pe, lam * n_experts * float(np.dot(f, pe))


def aux_grad(f, total, m, lam: float):
    """dL_aux/dp[u, e] = lambda E f_e m_u / M for the tokens with multiplicities m
    (C_e treated as a constant, App. B)."""
    n_experts = len(f)
    return lam * n_experts * np.outer(np.asarray(m, dtype=np.float64), np.asarray(f)) / total


def _multiplicities(inp: Dict, n_copies: int):
    shp = inp["shape"]
    m_p = np.full(shp.prefix_len, n_copies, dtype=np.int64)
    m_s = np.ones(int(inp["suffix_lens"].sum()), dtype=np.int64)
    return m_p, m_s


def reuse_reference(inp: Dict, lam: float, n_copies: int = -1) -> Dict[str, np.ndarray]:
    """The reuse schedule's accounting: prefix tokens once with m = N (or
    n_copies), suffix tokens with m = 1; gradients per physical token."""
    shp = inp["shape"]
    n = shp.n if n_copies < 0 else n_copies
    m_p, m_s = _multiplicities(inp, n)
    p = np.concatenate([inp["p_p"], inp["p_s"]], axis=0)
    r = np.concatenate([inp["r_p"], inp["r_s"]], axis=0)
    counts, mass, total = logical_stats(p, r, np.concatenate([m_p, m_s]), shp.num_experts)
    f, pe, loss = aux_loss(counts, mass, total, shp.top_k, lam)
    return {"C": counts, "R": mass, "M": total, "f": f, "P": pe, "L": loss,
            "dp_p": aux_grad(f, total, m_p, lam), "dp_s": aux_grad(f, total, m_s, lam)}


def materialized_reference(inp: Dict, lam: float, n_copies: int = -1) -> Dict[str, np.ndarray]:
    """The dense baseline's accounting: every trajectory holds its own copy
    of the prefix tokens (all multiplicities 1).  The prefix gradient is the
    sum over the copies, which is what reaches the shared prefix."""
    shp = inp["shape"]
    n = shp.n if n_copies < 0 else n_copies
    parts_p, parts_r = [], []
    for _ in range(n):
        parts_p.append(inp["p_p"])
        parts_r.append(inp["r_p"])
    parts_p.append(inp["p_s"])
    parts_r.append(inp["r_s"])
    p = np.concatenate(parts_p, axis=0)
    r = np.concatenate(parts_r, axis=0)
    ones = np.ones(p.shape[0], dtype=np.int64)
    counts, mass, total = logical_stats(p, r, ones, shp.num_experts)
    f, pe, loss = aux_loss(counts, mass, total, shp.top_k, lam)
    g = aux_grad(f, total, ones, lam)
    pl = shp.prefix_len
    dp_p = sum(g[c * pl:(c + 1) * pl] for c in range(n)) if n else np.zeros((pl, shp.num_experts))
    return {"C": counts, "R": mass, "M": total, "f": f, "P": pe, "L": loss,
            "dp_p": dp_p, "dp_s": g[n * pl:]}
