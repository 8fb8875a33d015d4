"""fp64 CPU oracle for prefix-shared causal attention of one GRPO prompt group.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
benchmark's CPU-baseline leg may import or run this module; the product path
never does.  It shares no code with the GPU library.

What it computes (paper Sec. 2.1 and App. A.1): a prompt group is N sequences
X(i) = [X_1; X_2(i)] that share one prefix.  Attention of sequence i is
ordinary causal softmax attention over its own L_i = P + S_i tokens,
inclusive of the diagonal, with score scale 1/sqrt(d_h) (Sec. 3.1).  Prefix
rows never see suffix keys; suffix rows see the whole prefix and their own
causal history, never another suffix (Sec. 3.2 Phase B, Sec. 4.2).

Two independent fp64 implementations live here:

* ``dense_group_reference`` -- the plain definition: recompute attention and
  its backward over every full sequence [P||S(i)] independently, exactly as a
  dense trainer does (Sec. 2.1), and sum the gradients of the shared prefix
  inputs over i (a shared input's gradient is the sum over its uses).
* ``three_phase_reference`` -- the paper's reordered schedule (Sec. 3.2,
  App. A.2-A.5): Phase A prefix forward once; Phase B per (packed) suffix
  microbatch with the joint prefix/suffix softmax, emitting
  gV_1 = P_21^T dH_2 and gK_1 = dS_21^T Q_2 / sqrt(d_h) into a gradient cache;
  Phase C one prefix backward that injects the cache:
  dV_1 = P_11^T G_Y + G_V, dK_1 = dS_11^T Q_1 / sqrt(d_h) + G_K,
  dQ_1 = dS_11 K_1 / sqrt(d_h).

Proposition 1 (Sec. 3.1, App. A.4) says the two agree over the reals.

GQA (not discussed in the paper; required by the workloads): q head h reads
kv head h // G with G = Hq / Hkv; gradients of a kv head sum over its G q heads.
LSE is the natural log of the row sum of exp of the scaled scores.

Layouts follow the GPU boundary: token-major [T, H, d]; LSE [H, T].
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np

__all__ = [
    "causal_attention",
    "dense_group_reference",
    "three_phase_reference",
    "group_loss",
]

_CHUNK = 1024  # query rows per block of materialised scores (memory only)


def _f64(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


def _softmax_rows(s: np.ndarray):
    """Row softmax of a score block whose masked entries are -inf.

    Returns (probabilities, natural-log row LSE)."""
    m = np.max(s, axis=1, keepdims=True)
    e = np.exp(s - m)
    l = np.sum(e, axis=1, keepdims=True)
    return e / l, (m + np.log(l))[:, 0]


def _softmax_backward(p: np.ndarray, dp: np.ndarray) -> np.ndarray:
    """SoftmaxBackward (App. A.4): dS = P * (dP - rowsum(dP * P))."""
    return p * (dp - np.sum(dp * p, axis=1, keepdims=True))


def causal_attention(q, k, v, do, scale, *, first_query_pos=0):
    """Causal attention of one sequence with its backward, all in fp64.

    q, do: [Lq, Hq, d] are the query rows at positions first_query_pos ...
    first_query_pos + Lq - 1 of a sequence whose keys/values k, v:
    [Lk, Hkv, d] sit at positions 0 .. Lk-1.  Key j is visible to the query
    at position r iff j <= r.  Returns o, lse [Hq, Lq], dq, dk, dv.
    """
    q, k, v, do = _f64(q), _f64(k), _f64(v), _f64(do)
    lq, hq, d = q.shape
    lk, hkv, _ = k.shape
    g = hq // hkv
    o = np.zeros_like(q)
    lse = np.zeros((hq, lq))
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    key_pos = np.arange(lk)
    for h in range(hq):
        kh, vh = k[:, h // g, :], v[:, h // g, :]
        for r0 in range(0, lq, _CHUNK):
            r1 = min(lq, r0 + _CHUNK)
            pos = first_query_pos + np.arange(r0, r1)
            s = scale * (q[r0:r1, h, :] @ kh.T)
            s[key_pos[None, :] > pos[:, None]] = -np.inf
            p, lse[h, r0:r1] = _softmax_rows(s)
            o[r0:r1, h, :] = p @ vh
            dph = do[r0:r1, h, :] @ vh.T
            ds = _softmax_backward(p, dph)
            dq[r0:r1, h, :] = scale * (ds @ kh)
            dk[:, h // g, :] += scale * (ds.T @ q[r0:r1, h, :])
            dv[:, h // g, :] += p.T @ do[r0:r1, h, :]
    return o, lse, dq, dk, dv


def sampled_rows_reference(inp: Dict[str, np.ndarray], prefix_rows, suffix_rows,
                           scale: Optional[float] = None) -> Dict[str, Dict]:
    """O, LSE and dQ of a few query rows of a group, each from its own
    sequence's definition (Sec. 2.1: trajectory i is [P||S(i)], causal).

    prefix_rows: prefix positions r; a prefix row sees prefix keys 0..r in
    every trajectory, so O and LSE are the same for all i and the group's
    dQ is the sum over the trajectories of each one's dQ with dO_P(i).
    suffix_rows: pairs (i, t), row t of suffix i, seeing all prefix keys and
    keys 0..t of its own suffix.  For groups too large for the full oracle:
    each row costs one row of attention."""
    shp = inp["shape"]
    sc = _default_scale(shp.head_dim, scale)
    P, cu = shp.prefix_len, inp["cu_seqlens"]
    out = {"prefix": {}, "suffix": {}}
    for r in prefix_rows:
        kk, vv = inp["k_p"][:r + 1], inp["v_p"][:r + 1]
        dq = 0.0
        for i in range(shp.n):
            o, lse, dqi, _, _ = causal_attention(inp["q_p"][r:r + 1], kk, vv, inp["do_p"][i][r:r + 1], sc,
                                                 first_query_pos=r)
            dq = dq + dqi
        out["prefix"][r] = {"o": o[0], "lse": lse[:, 0], "dq": dq[0]}
    for i, t in suffix_rows:
        a = int(cu[i])
        kk = np.concatenate([inp["k_p"], inp["k_s"][a:a + t + 1]], axis=0)
        vv = np.concatenate([inp["v_p"], inp["v_s"][a:a + t + 1]], axis=0)
        o, lse, dq, _, _ = causal_attention(inp["q_s"][a + t:a + t + 1], kk, vv, inp["do_s"][a + t:a + t + 1], sc,
                                            first_query_pos=P + t)
        out["suffix"][(i, t)] = {"o": o[0], "lse": lse[:, 0], "dq": dq[0]}
    return out


def causal_forward_rows(q, k, v, scale, *, first_query_pos=0):
    """The forward half of ``causal_attention``: O and the row LSE of query
    rows at positions first_query_pos .. first_query_pos + Lq - 1 of one
    sequence whose keys/values sit at positions 0 .. Lk - 1 (key j visible
    to position r iff j <= r).  Rows are taken in chunks and each chunk only
    against the keys its last row sees (memory only).  Returns o [Lq, Hq, d]
    and lse [Hq, Lq]."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    lq, hq, d = q.shape
    g = hq // k.shape[1]
    o = np.zeros_like(q)
    lse = np.zeros((hq, lq))
    for r0 in range(0, lq, _CHUNK):
        r1 = min(lq, r0 + _CHUNK)
        pos = first_query_pos + np.arange(r0, r1)
        nk = min(k.shape[0], int(pos[-1]) + 1)
        hidden = np.arange(nk)[None, :] > pos[:, None]
        for h in range(hq):
            s = scale * (q[r0:r1, h, :] @ k[:nk, h // g, :].T)
            s[hidden] = -np.inf
            p, lse[h, r0:r1] = _softmax_rows(s)
            o[r0:r1, h, :] = p @ v[:nk, h // g, :]
    return o, lse


def sampled_keys_reference(inp: Dict[str, np.ndarray], prefix_keys, suffix_keys,
                           scale: Optional[float] = None) -> Dict[str, Dict]:
    """dK and dV of a few keys of a group, and for prefix keys the cache
    values gK, gV, each from its own sequences' definition (Sec. 2.1).

    prefix_keys: prefix positions j.  Key j is seen by the prefix rows
    r >= j of every trajectory (with that trajectory's dO_P(i)) and by every
    suffix row of every trajectory; its gradient is the sum over all those
    uses.  gK(j) and gV(j) are the suffix rows' part of it (App. A.3: the
    suffix-row x prefix-key block, summed over i).
    suffix_keys: pairs (i, t), key t of suffix i, seen by the rows u >= t of
    suffix i only.
    Every row's probabilities come from its own LSE and O (computed by
    ``causal_forward_rows`` over the row's visible keys), then per key
    P = exp(s - LSE), dP = dO . v, D = dO . O, dS = P (dP - D),
    dK = scale sum dS q, dV = sum P dO, summed over the G query heads of
    the key's kv head.  For groups too large for the full oracle: the cost
    is one forward over the rows that see a sampled key, plus one column of
    scores per sampled key."""
    shp = inp["shape"]
    sc = _default_scale(shp.head_dim, scale)
    P, n, cu = shp.prefix_len, shp.n, np.asarray(inp["cu_seqlens"], np.int64)
    hq, hkv = shp.num_q_heads, shp.num_kv_heads
    g = hq // hkv
    q_p, k_p, v_p = _f64(inp["q_p"]), _f64(inp["k_p"]), _f64(inp["v_p"])
    out = {"prefix": {}, "suffix": {}}
    prefix_keys = sorted(set(int(j) for j in prefix_keys))
    need_sfx = set(i for i, _ in suffix_keys) | (set(range(n)) if prefix_keys else set())
    # forward statistics of every row that sees a sampled key
    sfx = {}
    for i in sorted(need_sfx):
        a, b = int(cu[i]), int(cu[i + 1])
        kk = np.concatenate([k_p, _f64(inp["k_s"][a:b])], axis=0)
        vv = np.concatenate([v_p, _f64(inp["v_s"][a:b])], axis=0)
        q_i, do_i = _f64(inp["q_s"][a:b]), _f64(inp["do_s"][a:b])
        o_i, lse_i = causal_forward_rows(q_i, kk, vv, sc, first_query_pos=P)
        sfx[i] = (q_i, do_i, lse_i, np.einsum("thd,thd->ht", do_i, o_i))
    if prefix_keys:
        r_min = prefix_keys[0]
        o_p, lse_p = causal_forward_rows(q_p[r_min:], k_p, v_p, sc, first_query_pos=r_min)
        do_p = _f64(inp["do_p"][:, r_min:])                      # [N, P - r_min, Hq, d]
        d_p = np.einsum("nrhd,rhd->nhr", do_p, o_p)             # D of each trajectory's prefix rows
        qp = q_p[r_min:]
    for j in prefix_keys:
        dk, dv = np.zeros((hkv, shp.head_dim)), np.zeros((hkv, shp.head_dim))
        gk, gv = np.zeros_like(dk), np.zeros_like(dv)
        for h in range(hq):
            kv = h // g
            kj, vj = k_p[j, kv], v_p[j, kv]
            # prefix rows r >= j, the same probabilities in every trajectory
            rows = slice(j - r_min, P - r_min)
            p = np.exp(sc * (qp[rows, h] @ kj) - lse_p[h, rows])
            for i in range(n):
                doi = do_p[i, rows, h]
                ds = p * (doi @ vj - d_p[i, h, rows])
                dk[kv] += sc * (ds @ qp[rows, h])
                dv[kv] += p @ doi
            # every suffix row of every trajectory
            for i in range(n):
                q_i, do_i, lse_i, d_i = sfx[i]
                p = np.exp(sc * (q_i[:, h] @ kj) - lse_i[h])
                ds = p * (do_i[:, h] @ vj - d_i[h])
                gk[kv] += sc * (ds @ q_i[:, h])
                gv[kv] += p @ do_i[:, h]
        out["prefix"][j] = {"dk": dk + gk, "dv": dv + gv, "g_k": gk, "g_v": gv}
    for i, t in suffix_keys:
        a = int(cu[i])
        q_i, do_i, lse_i, d_i = sfx[i]
        dk, dv = np.zeros((hkv, shp.head_dim)), np.zeros((hkv, shp.head_dim))
        for h in range(hq):
            kv = h // g
            kj, vj = _f64(inp["k_s"][a + t, kv]), _f64(inp["v_s"][a + t, kv])
            p = np.exp(sc * (q_i[t:, h] @ kj) - lse_i[h, t:])
            ds = p * (do_i[t:, h] @ vj - d_i[h, t:])
            dk[kv] += sc * (ds @ q_i[t:, h])
            dv[kv] += p @ do_i[t:, h]
        out["suffix"][(i, t)] = {"dk": dk, "dv": dv}
    return out


def _default_scale(d: int, scale: Optional[float]) -> float:
    return 1.0 / np.sqrt(d) if not scale else float(scale)


def dense_group_reference(inp: Dict[str, np.ndarray], scale: Optional[float] = None,
                          do_p: Optional[np.ndarray] = None) -> Dict[str, np.ndarray]:
    """The plain definition: every trajectory [P||S(i)] recomputed on its own.

    ``inp`` holds q_p, k_p, v_p, q_s, k_s, v_s, do_s and cu_seqlens (packed
    suffix rows, see the synthetic generator); ``do_p`` [N, P, Hq, d] are the
    per-trajectory prefix-row adjoints (default: inp["do_p"]).

    Rows >= P of sequence i are suffix i's outputs and gradients.  The prefix
    forward results must be identical for every i (prefix rows never see
    suffix keys); prefix gradients are summed over i.  The gradient-KV cache
    check values G_K, G_V are the suffix-row x prefix-key blocks of the
    dense backward, gK(i) = dS[P:, :P]^T Q[P:] / sqrt(d_h) and
    gV(i) = P[P:, :P]^T dO[P:] (Sec. 3.1 Insight 2, App. A.3), summed over i.
    """
    q_p, k_p, v_p = _f64(inp["q_p"]), _f64(inp["k_p"]), _f64(inp["v_p"])
    q_s, k_s, v_s, do_s = _f64(inp["q_s"]), _f64(inp["k_s"]), _f64(inp["v_s"]), _f64(inp["do_s"])
    cu = np.asarray(inp["cu_seqlens"], dtype=np.int64)
    do_p = _f64(inp["do_p"] if do_p is None else do_p)
    p_len, hq, d = q_p.shape
    hkv = k_p.shape[1]
    g = hq // hkv
    sc = _default_scale(d, scale)
    n = len(cu) - 1
    t = int(cu[-1])

    out = {
        "o_p": None, "lse_p": None,
        "o_s": np.zeros((t, hq, d)), "lse_s": np.zeros((hq, t)),
        "dq_p": np.zeros((p_len, hq, d)), "dk_p": np.zeros((p_len, hkv, d)),
        "dv_p": np.zeros((p_len, hkv, d)),
        "dq_s": np.zeros((t, hq, d)), "dk_s": np.zeros((t, hkv, d)),
        "dv_s": np.zeros((t, hkv, d)),
        "g_k": np.zeros((p_len, hkv, d)), "g_v": np.zeros((p_len, hkv, d)),
        "prefix_forward_spread": 0.0,
    }
    for i in range(n):
        a, b = int(cu[i]), int(cu[i + 1])
        q = np.concatenate([q_p, q_s[a:b]], axis=0)
        k = np.concatenate([k_p, k_s[a:b]], axis=0)
        v = np.concatenate([v_p, v_s[a:b]], axis=0)
        do = np.concatenate([do_p[i], do_s[a:b]], axis=0)
        o, lse, dq, dk, dv = causal_attention(q, k, v, do, sc)
        if out["o_p"] is None:
            out["o_p"], out["lse_p"] = o[:p_len].copy(), lse[:, :p_len].copy()
        else:
            out["prefix_forward_spread"] = max(
                out["prefix_forward_spread"],
                float(np.max(np.abs(o[:p_len] - out["o_p"]), initial=0.0)),
                float(np.max(np.abs(lse[:, :p_len] - out["lse_p"]), initial=0.0)))
        out["o_s"][a:b], out["lse_s"][:, a:b] = o[p_len:], lse[:, p_len:]
        out["dq_p"] += dq[:p_len]
        out["dk_p"] += dk[:p_len]
        out["dv_p"] += dv[:p_len]
        out["dq_s"][a:b], out["dk_s"][a:b], out["dv_s"][a:b] = dq[p_len:], dk[p_len:], dv[p_len:]
        # cache check values: suffix rows against prefix keys only
        if b > a and p_len > 0:
            gk, gv = _suffix_rows_vs_prefix(q, k, v, do, o, lse, sc, p_len, g)
            out["g_k"] += gk
            out["g_v"] += gv
    if out["o_p"] is None:  # N == 0 cannot happen for a group; keep shapes sane
        out["o_p"], out["lse_p"] = np.zeros((p_len, hq, d)), np.zeros((hq, p_len))
    return out


def _suffix_rows_vs_prefix(q, k, v, do, o, lse, sc, p_len, g):
    """The suffix-row x prefix-key blocks of one dense sequence's backward:
    gK = dS[P:, :P]^T Q[P:] * scale and gV = P[P:, :P]^T dO[P:], from the
    full-row probabilities (rows normalised over prefix and suffix keys)."""
    hq = q.shape[1]
    hkv = k.shape[1]
    d = q.shape[2]
    gk = np.zeros((p_len, hkv, d))
    gv = np.zeros((p_len, hkv, d))
    lk = k.shape[0]
    key_pos = np.arange(lk)
    for h in range(hq):
        kh, vh = k[:, h // g, :], v[:, h // g, :]
        pos = np.arange(p_len, q.shape[0])
        s = sc * (q[p_len:, h, :] @ kh.T)
        s[key_pos[None, :] > pos[:, None]] = -np.inf
        p = np.exp(s - lse[h, p_len:][:, None])
        dph = do[p_len:, h, :] @ vh.T
        drow = np.sum(do[p_len:, h, :] * o[p_len:, h, :], axis=1, keepdims=True)
        ds = p * (dph - drow)
        gk[:, h // g, :] += sc * (ds[:, :p_len].T @ q[p_len:, h, :])
        gv[:, h // g, :] += p[:, :p_len].T @ do[p_len:, h, :]
    return gk, gv


# ---------------------------------------------------------------------------
# The reordered three-phase schedule (Sec. 3.2, App. A.2-A.5), written
# independently of the dense definition above.
# ---------------------------------------------------------------------------

def _phase_a_prefix_forward(q_p, k_p, v_p, sc, g):
    """Phase A: H_1 = P_11 V_1 with P_11 the causal prefix softmax (App. A.1).
    Returns O_P [P,Hq,d] and LSE_P [Hq,P]."""
    p_len, hq, d = q_p.shape
    o = np.zeros((p_len, hq, d))
    lse = np.zeros((hq, p_len))
    if p_len == 0:
        return o, lse
    causal = np.triu(np.ones((p_len, p_len), dtype=bool), k=1)
    for h in range(hq):
        s11 = sc * (q_p[:, h, :] @ k_p[:, h // g, :].T)
        s11[causal] = -np.inf
        p11, lse[h] = _softmax_rows(s11)
        o[:, h, :] = p11 @ v_p[:, h // g, :]
    return o, lse


def _phase_b_microbatch(q_mb, k_mb, v_mb, do_mb, seg, k_p, v_p, sc, g):
    """Phase B for one packed suffix microbatch (Sec. 4.2 packed layout).

    Rows are the concatenated suffixes of the microbatch; ``seg`` gives each
    row's suffix id and ``loc`` its local position.  Keys are the read-only
    prefix block (visible to every suffix row) followed by the packed suffix
    keys, visible only within the same suffix and causally (block-diagonal
    causal).  One joint softmax per row over [S_21, S_22] (App. A.2).
    Returns O, LSE and dQ_2, dK_2, dV_2 and this microbatch's gK_1, gV_1.
    """
    t, hq, d = q_mb.shape
    p_len = k_p.shape[0]
    hkv = k_p.shape[1]
    loc = np.zeros(t, dtype=np.int64)
    for sid in np.unique(seg):
        idx = np.nonzero(seg == sid)[0]
        loc[idx] = np.arange(len(idx))
    visible22 = (seg[:, None] == seg[None, :]) & (loc[None, :] <= loc[:, None])
    o = np.zeros((t, hq, d))
    lse = np.zeros((hq, t))
    dq2 = np.zeros((t, hq, d))
    dk2 = np.zeros((t, hkv, d))
    dv2 = np.zeros((t, hkv, d))
    gk1 = np.zeros((p_len, hkv, d))
    gv1 = np.zeros((p_len, hkv, d))
    for h in range(hq):
        kv = h // g
        s21 = sc * (q_mb[:, h, :] @ k_p[:, kv, :].T)           # [t, P]
        s22 = sc * (q_mb[:, h, :] @ k_mb[:, kv, :].T)          # [t, t]
        s22 = np.where(visible22, s22, -np.inf)
        p_joint, lse[h] = _softmax_rows(np.concatenate([s21, s22], axis=1))
        p21, p22 = p_joint[:, :p_len], p_joint[:, p_len:]
        o[:, h, :] = p21 @ v_p[:, kv, :] + p22 @ v_mb[:, kv, :]  # H_2 = P_21 V_1 + P_22 V_2
        dh2 = do_mb[:, h, :]
        gv1[:, kv, :] += p21.T @ dh2                            # gV_1 = P_21^T dH_2
        dv2[:, kv, :] += p22.T @ dh2                            # dV_2 = P_22^T dH_2
        dp21 = dh2 @ v_p[:, kv, :].T                             # dP_21 = dH_2 V_1^T
        dp22 = dh2 @ v_mb[:, kv, :].T                            # dP_22 = dH_2 V_2^T
        ds_joint = _softmax_backward(p_joint, np.concatenate([dp21, dp22], axis=1))
        ds21, ds22 = ds_joint[:, :p_len], ds_joint[:, p_len:]
        dq2[:, h, :] = sc * (ds21 @ k_p[:, kv, :] + ds22 @ k_mb[:, kv, :])
        dk2[:, kv, :] += sc * (ds22.T @ q_mb[:, h, :])          # dK_2 = dS_22^T Q_2 / sqrt(d_h)
        gk1[:, kv, :] += sc * (ds21.T @ q_mb[:, h, :])          # gK_1 = dS_21^T Q_2 / sqrt(d_h)
    return o, lse, dq2, dk2, dv2, gk1, gv1


def _phase_c_prefix_backward(q_p, k_p, v_p, o_p, g_y, g_k, g_v, sc, g):
    """Phase C: one prefix backward with the injected cache (App. A.3-A.5):
    dP_11 = G_Y V_1^T, dS_11 = SoftmaxBackward(P_11, dP_11),
    dQ_1 = dS_11 K_1 / sqrt(d_h), dK_1 = dS_11^T Q_1 / sqrt(d_h) + G_K,
    dV_1 = P_11^T G_Y + G_V."""
    p_len, hq, d = q_p.shape
    hkv = k_p.shape[1]
    dq = np.zeros((p_len, hq, d))
    dk = g_k.copy()
    dv = g_v.copy()
    if p_len == 0:
        return dq, dk, dv
    causal = np.triu(np.ones((p_len, p_len), dtype=bool), k=1)
    for h in range(hq):
        kv = h // g
        s11 = sc * (q_p[:, h, :] @ k_p[:, kv, :].T)
        s11[causal] = -np.inf
        p11, _ = _softmax_rows(s11)
        dp11 = g_y[:, h, :] @ v_p[:, kv, :].T
        ds11 = _softmax_backward(p11, dp11)
        dq[:, h, :] = sc * (ds11 @ k_p[:, kv, :])
        dk[:, kv, :] += sc * (ds11.T @ q_p[:, h, :])
        dv[:, kv, :] += p11.T @ g_y[:, h, :]
    return dq, dk, dv


def three_phase_reference(inp: Dict[str, np.ndarray], scale: Optional[float] = None,
                          microbatches: Optional[Sequence[Sequence[int]]] = None,
                          g_y: Optional[np.ndarray] = None) -> Dict[str, np.ndarray]:
    """The paper's three-phase schedule in fp64 (Sec. 3.2).

    microbatches: suffix ids per Phase-B microbatch, in execution order
    (default: one suffix per microbatch, in order).  Any split and any order
    is allowed; every suffix must appear exactly once.
    g_y: the accumulated prefix-row adjoint G_Y = sum_i dO_P(i)
    (default: inp["g_y"], the synthetic group's value).
    Returns the same keys as ``dense_group_reference``.
    """
    q_p, k_p, v_p = _f64(inp["q_p"]), _f64(inp["k_p"]), _f64(inp["v_p"])
    q_s, k_s, v_s, do_s = _f64(inp["q_s"]), _f64(inp["k_s"]), _f64(inp["v_s"]), _f64(inp["do_s"])
    cu = np.asarray(inp["cu_seqlens"], dtype=np.int64)
    gy = _f64(inp["g_y"] if g_y is None else g_y)
    p_len, hq, d = q_p.shape
    hkv = k_p.shape[1]
    g = hq // hkv
    sc = _default_scale(d, scale)
    n = len(cu) - 1
    t = int(cu[-1])
    if microbatches is None:
        microbatches = [[i] for i in range(n)]
    seen = sorted(i for mb in microbatches for i in mb)
    if seen != list(range(n)):
        raise ValueError("every suffix must appear in exactly one microbatch")

    # Phase A: prefix forward once; K_1, V_1 stay as the forward cache.
    o_p, lse_p = _phase_a_prefix_forward(q_p, k_p, v_p, sc, g)

    # Phase B: suffix microbatches read K_1/V_1 and accumulate gK/gV.
    g_k = np.zeros((p_len, hkv, d))
    g_v = np.zeros((p_len, hkv, d))
    o_s = np.zeros((t, hq, d)); lse_s = np.zeros((hq, t))
    dq_s = np.zeros((t, hq, d)); dk_s = np.zeros((t, hkv, d)); dv_s = np.zeros((t, hkv, d))
    for mb in microbatches:
        rows = np.concatenate([np.arange(cu[i], cu[i + 1]) for i in mb]).astype(np.int64)
        seg = np.concatenate([np.full(cu[i + 1] - cu[i], i) for i in mb]).astype(np.int64)
        if len(rows) == 0:
            continue
        o, lse, dq2, dk2, dv2, gk1, gv1 = _phase_b_microbatch(
            q_s[rows], k_s[rows], v_s[rows], do_s[rows], seg, k_p, v_p, sc, g)
        o_s[rows], lse_s[:, rows] = o, lse
        dq_s[rows], dk_s[rows], dv_s[rows] = dq2, dk2, dv2
        g_k += gk1
        g_v += gv1

    # Phase C: inject the cache, prefix backward once.
    dq_p, dk_p, dv_p = _phase_c_prefix_backward(q_p, k_p, v_p, o_p, gy, g_k, g_v, sc, g)
    return {
        "o_p": o_p, "lse_p": lse_p, "o_s": o_s, "lse_s": lse_s,
        "dq_p": dq_p, "dk_p": dk_p, "dv_p": dv_p,
        "dq_s": dq_s, "dk_s": dk_s, "dv_s": dv_s,
        "g_k": g_k, "g_v": g_v,
    }


def group_loss(inp: Dict[str, np.ndarray], scale: Optional[float] = None,
               do_p: Optional[np.ndarray] = None) -> float:
    """The scalar whose gradients the references return:
    L = sum_i [ <dO_P(i), O_P> + <dO_S(i), O_S(i)> ] (forward only, fp64).
    Used for finite-difference checks of both references."""
    q_p, k_p, v_p = _f64(inp["q_p"]), _f64(inp["k_p"]), _f64(inp["v_p"])
    q_s, k_s, v_s, do_s = _f64(inp["q_s"]), _f64(inp["k_s"]), _f64(inp["v_s"]), _f64(inp["do_s"])
    cu = np.asarray(inp["cu_seqlens"], dtype=np.int64)
    dop = _f64(inp["do_p"] if do_p is None else do_p)
    p_len, hq, d = q_p.shape
    g = hq // k_p.shape[1]
    sc = _default_scale(d, scale)
    total = 0.0
    for i in range(len(cu) - 1):
        a, b = int(cu[i]), int(cu[i + 1])
        q = np.concatenate([q_p, q_s[a:b]], axis=0)
        k = np.concatenate([k_p, k_s[a:b]], axis=0)
        v = np.concatenate([v_p, v_s[a:b]], axis=0)
        do = np.concatenate([dop[i], do_s[a:b]], axis=0)
        L = q.shape[0]
        mask = np.triu(np.ones((L, L), dtype=bool), k=1)
        for h in range(hq):
            s = sc * (q[:, h, :] @ k[:, h // g, :].T)
            s[mask] = -np.inf
            s = s - s.max(axis=1, keepdims=True)
            pm = np.exp(s)
            pm /= pm.sum(axis=1, keepdims=True)
            total += float(np.sum(do[:, h, :] * (pm @ v[:, h // g, :])))
    return total
