"""fp64 CPU oracle of one Llama3-style decoder layer over a GRPO prompt
group, dense and reordered (paper Sec. 3.1-3.2; App. A.6 parameter-gradient
accounting; App. A.7 extension across layers).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Layer (pre-norm, no biases, norm gains one):
    h = x + Attn(RoPE(rms(x) W_q), RoPE(rms(x) W_k), rms(x) W_v) W_o
    y = h + (silu(rms(h) W_gate) * (rms(h) W_up)) W_down
rms(x) = x / sqrt(mean(x^2) + eps); RoPE pairs dimension j with j + d/2
(rotate-half) at angle pos * theta^(-2j/d); attention is causal with GQA
(q head h reads kv head h // G) and scale 1/sqrt(d).  Positions are 0..P-1
for the prefix and P..P+S_i-1 for suffix i, as in the sequence [P||S(i)].

``dense_layer_reference`` runs every trajectory [P||S(i)] through the layer
with upstream [dY_P(i); dY_S(i)] and sums the shared prefix's and the
weights' gradients.  ``reordered_layer_reference`` is the schedule: Phase A
prefix forward once; Phase B per suffix, forward and backward with the
prefix K/V as leaves whose gradients accumulate (the gK/gV cache); Phase C
one prefix backward with G_Y = sum_i dY_P(i) and the accumulated cache
injected into the prefix K/V.  Both use torch autograd in float64.

``dense_stack_reference`` and ``reordered_stack_reference`` do the same
for a stack of layers, each with its own weights, the output of layer l
being the input of layer l + 1 (App. A.7): the reordered stack runs the
prefix through every layer once (Phase A), each suffix forward through
every layer against that layer's cached prefix K/V and backward from the
top (Phase B, one cache per layer), then the prefix backward from the top
layer down (Phase C), layer l's injected cache and upstream adjoint giving
the prefix hidden-state adjoint that layer l - 1 receives as its G_Y.
"""
from __future__ import annotations

from typing import Dict, List

import numpy as np
import torch

W_KEYS = ("wq", "wk", "wv", "wo", "wg", "wu", "wd")


def _t(x, grad=False):
    return torch.tensor(np.asarray(x, dtype=np.float64), dtype=torch.float64, requires_grad=grad)


def rms(x, eps):
    return x / torch.sqrt((x * x).mean(dim=-1, keepdim=True) + eps)


def rope(x, pos, theta):
    """x [T, H, d] at positions pos [T]: rotate-half pairing (j, j + d/2)."""
    d = x.shape[-1]
    half = d // 2
    inv = theta ** (-torch.arange(0, half, dtype=torch.float64) * 2.0 / d)
    ang = pos.to(torch.float64)[:, None] * inv[None, :]
    cos = torch.cat([torch.cos(ang), torch.cos(ang)], dim=-1)[:, None, :]
    sin = torch.cat([torch.sin(ang), torch.sin(ang)], dim=-1)[:, None, :]
    rot = torch.cat([-x[..., half:], x[..., :half]], dim=-1)
    return x * cos + rot * sin


def attention(q, k, v, visible):
    """q [Tq, Hq, d], k/v [Tk, Hkv, d], visible [Tq, Tk] bool."""
    hq, hkv, d = q.shape[1], k.shape[1], q.shape[2]
    g = hq // hkv
    outs = []
    for h in range(hq):
        s = (q[:, h] @ k[:, h // g].T) / np.sqrt(d)
        s = s.masked_fill(~visible, float("-inf"))
        p = torch.softmax(s, dim=-1)
        outs.append(p @ v[:, h // g])
    return torch.stack(outs, dim=1)


def _qkv(x, W, shp, pos):
    t = x.shape[0]
    h1 = rms(x, shp.norm_eps)
    q = rope((h1 @ W["wq"]).view(t, shp.num_q_heads, shp.head_dim), pos, shp.rope_theta)
    k = rope((h1 @ W["wk"]).view(t, shp.num_kv_heads, shp.head_dim), pos, shp.rope_theta)
    v = (h1 @ W["wv"]).view(t, shp.num_kv_heads, shp.head_dim)
    return q, k, v


def _tail(x, o, W, shp):
    h = x + o.reshape(x.shape[0], -1) @ W["wo"]
    h2 = rms(h, shp.norm_eps)
    return h + (torch.nn.functional.silu(h2 @ W["wg"]) * (h2 @ W["wu"])) @ W["wd"]


def _weights(inp):
    return {k: _t(inp["weights"][k], grad=True) for k in W_KEYS}


def dense_layer_reference(inp: Dict) -> Dict:
    shp = inp["shape"]
    P = shp.prefix_len
    W = _weights(inp)
    y_s, dx_s = [], []
    dx_p = torch.zeros(P, shp.hidden, dtype=torch.float64)
    y_p = None
    for i in range(shp.n):
        x = _t(np.concatenate([inp["x_p"], inp["x_s"][i]], axis=0), grad=True)
        L = x.shape[0]
        pos = torch.arange(L)
        q, k, v = _qkv(x, W, shp, pos)
        vis = torch.tril(torch.ones(L, L, dtype=torch.bool))
        y = _tail(x, attention(q, k, v, vis), W, shp)
        dy = _t(np.concatenate([inp["dy_p"][i], inp["dy_s"][i]], axis=0))
        y.backward(dy)
        dx_p += x.grad[:P]
        dx_s.append(x.grad[P:].numpy())
        y_s.append(y[P:].detach().numpy())
        if y_p is None:
            y_p = y[:P].detach().numpy()
    return {"y_p": y_p, "y_s": y_s, "dx_p": dx_p.numpy(), "dx_s": dx_s,
            "dw": {k: W[k].grad.numpy() for k in W_KEYS}}


def reordered_layer_reference(inp: Dict) -> Dict:
    shp = inp["shape"]
    P = shp.prefix_len
    W = _weights(inp)
    # Phase A: the prefix forward once; its graph is kept for Phase C
    x_p = _t(inp["x_p"], grad=True)
    q_p, k_p, v_p = _qkv(x_p, W, shp, torch.arange(P))
    y_p = _tail(x_p, attention(q_p, k_p, v_p, torch.tril(torch.ones(P, P, dtype=torch.bool))), W, shp)
    # the cache: prefix K/V (after RoPE) as leaves whose gradients accumulate
    k_c = k_p.detach().requires_grad_(True)
    v_c = v_p.detach().requires_grad_(True)
    # Phase B: each suffix forward and backward against the cached prefix K/V
    y_s, dx_s = [], []
    for i in range(shp.n):
        x_s = _t(inp["x_s"][i], grad=True)
        s = x_s.shape[0]
        q_s, k_s, v_s = _qkv(x_s, W, shp, torch.arange(P, P + s))
        vis = torch.cat([torch.ones(s, P, dtype=torch.bool), torch.tril(torch.ones(s, s, dtype=torch.bool))], dim=1)
        o = attention(q_s, torch.cat([k_c, k_s]), torch.cat([v_c, v_s]), vis)
        y = _tail(x_s, o, W, shp)
        y.backward(_t(inp["dy_s"][i]))
        y_s.append(y.detach().numpy())
        dx_s.append(x_s.grad.numpy())
    # Phase C: one prefix backward with G_Y and the injected cache
    g_y = _t(np.sum(np.asarray(inp["dy_p"], dtype=np.float64), axis=0))
    grads = [g_y]
    outs = [y_p]
    for t, leaf in ((k_p, k_c), (v_p, v_c)):
        if leaf.grad is not None:
            outs.append(t)
            grads.append(leaf.grad)
    torch.autograd.backward(outs, grads)
    return {"y_p": y_p.detach().numpy(), "y_s": y_s, "dx_p": x_p.grad.numpy(), "dx_s": dx_s,
            "dw": {k: W[k].grad.numpy() for k in W_KEYS}}


def group_loss(inp: Dict) -> float:
    """L = sum_i <Y(i), dY(i)> over the dense trajectories (for finite differences)."""
    shp = inp["shape"]
    W = {k: _t(inp["weights"][k]) for k in W_KEYS}
    total = 0.0
    with torch.no_grad():
        for i in range(shp.n):
            x = _t(np.concatenate([inp["x_p"], inp["x_s"][i]], axis=0))
            L = x.shape[0]
            q, k, v = _qkv(x, W, shp, torch.arange(L))
            y = _tail(x, attention(q, k, v, torch.tril(torch.ones(L, L, dtype=torch.bool))), W, shp)
            dy = _t(np.concatenate([inp["dy_p"][i], inp["dy_s"][i]], axis=0))
            total += float((y * dy).sum())
    return total


# ---------------------------------------------------------------------------
# A stack of layers (App. A.7: the schedule extended across layers)
# ---------------------------------------------------------------------------

def _stack_weights(inp):
    return [{k: _t(w[k], grad=True) for k in W_KEYS} for w in inp["weights"]]


def _layer(x, W, shp, pos, visible, k_extra=None, v_extra=None):
    """One layer over rows x at positions pos; k_extra/v_extra: cached
    prefix K/V placed before the rows' own keys.  Returns y, k, v."""
    q, k, v = _qkv(x, W, shp, pos)
    kk = k if k_extra is None else torch.cat([k_extra, k])
    vv = v if v_extra is None else torch.cat([v_extra, v])
    return _tail(x, attention(q, kk, vv, visible), W, shp), k, v


def dense_stack_reference(inp: Dict) -> Dict:
    """Every trajectory [P||S(i)] through all layers, upstream
    [dY_P(i); dY_S(i)] at the top; the prefix's and every layer's weight
    gradients summed over the trajectories."""
    shp = inp["shape"]
    P = shp.prefix_len
    Ws = _stack_weights(inp)
    y_s, dx_s, y_p = [], [], None
    dx_p = torch.zeros(P, shp.hidden, dtype=torch.float64)
    for i in range(shp.n):
        x0 = _t(np.concatenate([inp["x_p"], inp["x_s"][i]], axis=0), grad=True)
        L = x0.shape[0]
        pos = torch.arange(L)
        vis = torch.tril(torch.ones(L, L, dtype=torch.bool))
        x = x0
        for W in Ws:
            x, _, _ = _layer(x, W, shp, pos, vis)
        x.backward(_t(np.concatenate([inp["dy_p"][i], inp["dy_s"][i]], axis=0)))
        dx_p += x0.grad[:P]
        dx_s.append(x0.grad[P:].numpy())
        y_s.append(x[P:].detach().numpy())
        if y_p is None:
            y_p = x[:P].detach().numpy()
    return {"y_p": y_p, "y_s": y_s, "dx_p": dx_p.numpy(), "dx_s": dx_s,
            "dw": [{k: W[k].grad.numpy() for k in W_KEYS} for W in Ws]}


def reordered_stack_reference(inp: Dict) -> Dict:
    """The three-phase schedule over the stack (see the module docstring)."""
    shp = inp["shape"]
    P = shp.prefix_len
    Ws = _stack_weights(inp)
    pos_p = torch.arange(P)
    vis_p = torch.tril(torch.ones(P, P, dtype=torch.bool))
    # Phase A: the prefix through every layer once; layer l's graph (input
    # leaf, output, K/V) is kept for its Phase C
    xs, ys, ks, vs = [], [], [], []
    x = _t(inp["x_p"])
    for W in Ws:
        x_in = x.detach().requires_grad_(True)
        y, k, v = _layer(x_in, W, shp, pos_p, vis_p)
        xs.append(x_in); ys.append(y); ks.append(k); vs.append(v)
        x = y
    # the caches: every layer's prefix K/V as leaves whose gradients accumulate
    k_c = [k.detach().requires_grad_(True) for k in ks]
    v_c = [v.detach().requires_grad_(True) for v in vs]
    # Phase B: each suffix forward through the layers against their cached
    # prefix K/V, then backward from the top
    y_s, dx_s = [], []
    for i in range(shp.n):
        x0 = _t(inp["x_s"][i], grad=True)
        s = x0.shape[0]
        pos = torch.arange(P, P + s)
        vis = torch.cat([torch.ones(s, P, dtype=torch.bool), torch.tril(torch.ones(s, s, dtype=torch.bool))], dim=1)
        x = x0
        for l, W in enumerate(Ws):
            x, _, _ = _layer(x, W, shp, pos, vis, k_c[l], v_c[l])
        x.backward(_t(inp["dy_s"][i]))
        y_s.append(x.detach().numpy())
        dx_s.append(x0.grad.numpy())
    # Phase C: from the top layer down, the upstream adjoint of layer l's
    # prefix output plus its injected cache give the adjoint of its input,
    # which is layer l - 1's upstream
    g = _t(np.sum(np.asarray(inp["dy_p"], dtype=np.float64), axis=0))
    for l in reversed(range(len(Ws))):
        outs, grads = [ys[l]], [g]
        for t, leaf in ((ks[l], k_c[l]), (vs[l], v_c[l])):
            if leaf.grad is not None:
                outs.append(t)
                grads.append(leaf.grad)
        torch.autograd.backward(outs, grads)
        g = xs[l].grad
    return {"y_p": ys[-1].detach().numpy(), "y_s": y_s, "dx_p": g.numpy(), "dx_s": dx_s,
            "dw": [{k: W[k].grad.numpy() for k in W_KEYS} for W in Ws]}


def stack_group_loss(inp: Dict) -> float:
    """L = sum_i <Y(i), dY(i)> over the dense trajectories through the stack."""
    shp = inp["shape"]
    Ws = [{k: _t(w[k]) for k in W_KEYS} for w in inp["weights"]]
    total = 0.0
    with torch.no_grad():
        for i in range(shp.n):
            x = _t(np.concatenate([inp["x_p"], inp["x_s"][i]], axis=0))
            L = x.shape[0]
            pos, vis = torch.arange(L), torch.tril(torch.ones(L, L, dtype=torch.bool))
            for W in Ws:
                x, _, _ = _layer(x, W, shp, pos, vis)
            dy = _t(np.concatenate([inp["dy_p"][i], inp["dy_s"][i]], axis=0))
            total += float((x * dy).sum())
    return total
