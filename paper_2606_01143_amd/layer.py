"""One Llama3-style decoder layer run through the three-phase schedule, and
the dense per-trajectory baseline, on one GPU.

Everything outside attention acts on each token on its own (paper
Sec. 3.1), so the layer splits at attention's K/V interface: Phase A runs
the prefix tokens through the layer once, keeping the prefix K/V (after
RoPE) resident; Phase B runs each suffix microbatch forward and backward,
its attention reading the prefix K/V and adding gK/gV into the fp32 cache;
Phase C runs the prefix backward once with G_Y = sum_i dY_P(i) and the
cache injected into attention's prefix K/V gradient.  Weight gradients
are the prefix part once plus every suffix part (App. A.6), accumulated in
fp32.

The token-wise operations (RMSNorm, RoPE, SwiGLU) are the library's
kernels, attention is the library's schedule calls, and the projections
are BLAS GEMMs (torch.matmul on the GPU, which ROCm serves with
hipBLASLt).  Forward and backward are written out by hand; nothing here
uses autograd.
"""
from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np
import torch

from . import binding as B

W_KEYS = ("wq", "wk", "wv", "wo", "wg", "wu", "wd")


class DecoderLayer:
    def __init__(self, inp: Dict, device="cuda:0"):
        shp = inp["shape"]
        dev = torch.device(device)
        up = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(device=dev, dtype=torch.bfloat16)
        self._setup(shp, {k: up(inp["weights"][k]) for k in W_KEYS}, dev, None)
        self.x_p = up(inp["x_p"])
        self.x_s = [up(x) for x in inp["x_s"]]
        self.dy_s = [up(x) for x in inp["dy_s"]]
        self.dy_p = [up(x) for x in inp["dy_p"]]
        # G_Y summed in fp32, rounded once
        self.g_y = torch.stack([x.float() for x in self.dy_p]).sum(0).to(torch.bfloat16) if shp.n else \
            torch.zeros_like(self.x_p)

    @classmethod
    def of_weights(cls, shape, weights: Dict[str, torch.Tensor], device, ws: Optional[torch.Tensor] = None):
        """A layer of a stack: its bf16 weights on the device, its own gK/gV
        cache; ``ws`` a workspace shared by the stack's layers."""
        layer = cls.__new__(cls)
        layer._setup(shape, weights, torch.device(device), ws)
        return layer

    def _setup(self, shp, weights, dev, ws):
        if shp.dtype != "bf16":
            raise ValueError("the layer path runs in bf16")
        self.shape = shp
        self.dev = dev
        self.w = weights
        hq, hkv, d, P = shp.num_q_heads, shp.num_kv_heads, shp.head_dim, shp.prefix_len
        self.dims = B.make_dims(hq, hkv, d, P, "bf16")
        self.gk = torch.zeros(P, hkv, d, dtype=torch.float32, device=self.dev)
        self.gv = torch.zeros_like(self.gk)
        if ws is None:
            ws = torch.empty(self.workspace_bytes(shp), dtype=torch.uint8, device=self.dev)
        self.ws = ws
        self._cu = {}
        self._dense_dims = {}

    @staticmethod
    def workspace_bytes(shp) -> int:
        dims = B.make_dims(shp.num_q_heads, shp.num_kv_heads, shp.head_dim, shp.prefix_len, "bf16")
        mx = max(shp.suffix_lens) if shp.n else 1
        return max(B.workspace_size(B.OP_PREFIX_BWD, dims), B.workspace_size(B.OP_SUFFIX_FWD, dims, 1, mx, mx),
                   B.workspace_size(B.OP_SUFFIX_BWD, dims, 1, mx, mx), 256)

    # ---------------------------------------------------------- token-wise
    def _forward(self, x: torch.Tensor, pos0: int, attend) -> Dict[str, torch.Tensor]:
        shp, w = self.shape, self.w
        T, hq, hkv, d = x.shape[0], shp.num_q_heads, shp.num_kv_heads, shp.head_dim
        e = lambda *s, dt=torch.bfloat16: torch.empty(*s, dtype=dt, device=self.dev)
        c = {"x": x, "n1": e(T, shp.hidden), "r1": e(T, dt=torch.float32)}
        B.rmsnorm_fwd(x, c["n1"], c["r1"], shp.norm_eps)
        q = (c["n1"] @ w["wq"]).view(T, hq, d)
        k = (c["n1"] @ w["wk"]).view(T, hkv, d)
        c["v"] = (c["n1"] @ w["wv"]).view(T, hkv, d)
        c["q"], c["k"] = e(T, hq, d), e(T, hkv, d)
        B.rope_fwd(q, c["q"], pos0, shp.rope_theta)
        B.rope_fwd(k, c["k"], pos0, shp.rope_theta)
        c["o"], c["lse"] = e(T, hq, d), e(T, hq, dt=torch.float32)
        attend(c)
        c["h"] = x + c["o"].view(T, -1) @ w["wo"]
        c["n2"], c["r2"] = e(T, shp.hidden), e(T, dt=torch.float32)
        B.rmsnorm_fwd(c["h"], c["n2"], c["r2"], shp.norm_eps)
        c["g"] = c["n2"] @ w["wg"]
        c["u"] = c["n2"] @ w["wu"]
        c["m"] = torch.empty_like(c["g"])
        B.swiglu_fwd(c["g"], c["u"], c["m"])
        c["y"] = c["h"] + c["m"] @ w["wd"]
        return c

    def _backward(self, c: Dict[str, torch.Tensor], dy: torch.Tensor, pos0: int, attend_bwd,
                  dw: Dict[str, torch.Tensor]) -> torch.Tensor:
        shp, w = self.shape, self.w
        T, hq, hkv, d = dy.shape[0], shp.num_q_heads, shp.num_kv_heads, shp.head_dim
        dm = dy @ w["wd"].t()
        dw["wd"] += (c["m"].t() @ dy).float()
        dg, du = torch.empty_like(c["g"]), torch.empty_like(c["u"])
        B.swiglu_bwd(c["g"], c["u"], dm, dg, du)
        dn2 = dg @ w["wg"].t() + du @ w["wu"].t()
        dw["wg"] += (c["n2"].t() @ dg).float()
        dw["wu"] += (c["n2"].t() @ du).float()
        dh = torch.empty_like(dy)
        B.rmsnorm_bwd(c["h"], c["r2"], dn2, dh, add=dy)
        do = (dh @ w["wo"].t()).view(T, hq, d).contiguous()
        dw["wo"] += (c["o"].view(T, -1).t() @ dh).float()
        dq_r = torch.empty_like(c["q"])
        dk_r, dv = torch.empty_like(c["k"]), torch.empty_like(c["v"])
        attend_bwd(c, do, dq_r, dk_r, dv)
        dq, dk = torch.empty_like(dq_r), torch.empty_like(dk_r)
        B.rope_bwd(dq_r, dq, pos0, shp.rope_theta)
        B.rope_bwd(dk_r, dk, pos0, shp.rope_theta)
        dq2, dk2, dv2 = dq.view(T, -1), dk.view(T, -1), dv.view(T, -1)
        dn1 = dq2 @ w["wq"].t() + dk2 @ w["wk"].t() + dv2 @ w["wv"].t()
        dw["wq"] += (c["n1"].t() @ dq2).float()
        dw["wk"] += (c["n1"].t() @ dk2).float()
        dw["wv"] += (c["n1"].t() @ dv2).float()
        dx = torch.empty_like(dy)
        B.rmsnorm_bwd(c["x"], c["r1"], dn1, dx, add=dh)
        return dx

    def _zero_dw(self):
        return {k: torch.zeros(v.shape, dtype=torch.float32, device=self.dev) for k, v in self.w.items()}

    def _cu_of(self, s: int) -> torch.Tensor:
        if s not in self._cu:
            self._cu[s] = torch.tensor([0, s], dtype=torch.int32, device=self.dev)
        return self._cu[s]

    # ------------------------------------------------------------ schedule
    def run_schedule(self) -> Dict:
        shp, dims, P = self.shape, self.dims, self.shape.prefix_len
        dw = self._zero_dw()
        B.gkv_cache_zero(dims, self.gk, self.gv)
        # Phase A: the prefix through the layer once
        def prefix_attn(c):
            B.prefix_fwd(dims, c["q"], c["k"], c["v"], c["o"], c["lse"])
        cp = self._forward(self.x_p, 0, prefix_attn)
        k_p, v_p = cp["k"], cp["v"]
        # Phase B: each suffix forward and backward against the prefix K/V
        y_s, dx_s = [], []
        for x_s, dy_s in zip(self.x_s, self.dy_s):
            s = x_s.shape[0]
            cu = self._cu_of(s)

            def suffix_attn(c, s=s, cu=cu):
                B.suffix_attn_fwd(dims, k_p, v_p, c["q"], c["k"], c["v"], cu, 1, s, s, c["o"], c["lse"], self.ws)

            def suffix_attn_bwd(c, do, dq, dk, dv, s=s, cu=cu):
                B.suffix_attn_bwd_accum(dims, k_p, v_p, c["q"], c["k"], c["v"], c["o"], c["lse"], do, cu, 1, s, s,
                                        dq, dk, dv, self.gk, self.gv, self.ws)

            cs = self._forward(x_s, P, suffix_attn)
            dx_s.append(self._backward(cs, dy_s, P, suffix_attn_bwd, dw))
            y_s.append(cs["y"])
            del cs
        # Phase C: the prefix backward once, G_Y upstream, the cache injected
        def prefix_attn_bwd(c, do, dq, dk, dv):
            B.prefix_bwd(dims, c["q"], c["k"], c["v"], c["o"], c["lse"], do, self.gk, self.gv, dq, dk, dv, self.ws)
        dx_p = self._backward(cp, self.g_y, 0, prefix_attn_bwd, dw)
        return {"y_p": cp["y"], "y_s": y_s, "dx_p": dx_p, "dx_s": dx_s, "dw": dw}

    # --------------------------------------------------------------- dense
    def _dims_for(self, L: int):
        if L not in self._dense_dims:
            shp = self.shape
            dims = B.make_dims(shp.num_q_heads, shp.num_kv_heads, shp.head_dim, L, "bf16")
            ws = torch.empty(max(B.workspace_size(B.OP_PREFIX_BWD, dims), 256), dtype=torch.uint8,
                             device=self.dev)
            # a zero cache (two buffers: the caches may not overlap)
            zero = tuple(torch.zeros(L, shp.num_kv_heads, shp.head_dim, dtype=torch.float32, device=self.dev)
                         for _ in range(2))
            self._dense_dims[L] = (dims, ws, zero)
        return self._dense_dims[L]

    def run_dense(self) -> Dict:
        """Every trajectory [P||S(i)] through the layer with causal attention
        over the whole sequence; the prefix's and the weights' gradients
        summed."""
        shp, P = self.shape, self.shape.prefix_len
        dw = self._zero_dw()
        y_s, dx_s, y_p = [], [], None
        dx_p = torch.zeros(P, shp.hidden, dtype=torch.float32, device=self.dev)
        for x_s, dy_s, dy_p in zip(self.x_s, self.dy_s, self.dy_p):
            x = torch.cat([self.x_p, x_s])
            L = x.shape[0]
            dims, ws, zero = self._dims_for(L)

            def attn(c, dims=dims):
                B.prefix_fwd(dims, c["q"], c["k"], c["v"], c["o"], c["lse"])

            def attn_bwd(c, do, dq, dk, dv, dims=dims, ws=ws, zero=zero):
                B.prefix_bwd(dims, c["q"], c["k"], c["v"], c["o"], c["lse"], do, zero[0], zero[1], dq, dk, dv, ws)

            c = self._forward(x, 0, attn)
            dx = self._backward(c, torch.cat([dy_p, dy_s]), 0, attn_bwd, dw)
            dx_p += dx[:P].float()
            dx_s.append(dx[P:])
            y_s.append(c["y"][P:])
            if y_p is None:
                y_p = c["y"][:P]
            del c
        return {"y_p": y_p, "y_s": y_s, "dx_p": dx_p.to(torch.bfloat16), "dx_s": dx_s, "dw": dw}
