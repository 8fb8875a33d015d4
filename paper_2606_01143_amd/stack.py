"""A stack of decoder layers run through the three-phase schedule, chained
across layers (paper App. A.7), with the prefix-state lifecycle of Sec. 3.3
and Sec. 4.3.

The layers are Llama3-style decoder layers (``layer.DecoderLayer``), each
with its own weights and gK/gV cache; the output of layer l is the input
of layer l + 1.  Phase A runs the prefix through every layer once.  Phase
B runs each suffix microbatch forward through every layer, its attention
reading that layer's prefix K/V, and backward from the top, each layer
adding its gK/gV into its own cache.  Phase C runs the prefix backward from
the top layer down: layer l gets the upstream adjoint of its prefix output
and its injected cache, and returns the adjoint of its prefix input, which
is the upstream adjoint of layer l - 1's prefix output.  Weight gradients
are every layer's prefix part plus its suffix parts (App. A.6).

Per layer the schedule keeps a *hot* set resident through Phase B: the
prefix K/V (after RoPE) that the suffixes attend to, and the cache.  The
rest of what Phase A saves for Phase C is *dormant* during Phase B: the
layer's input, both norms' outputs and statistics, the prefix queries,
attention output and LSE, the residual stream after attention and the MLP
activations.  With ``offload=True`` each layer's dormant set is packed to
pinned host memory right after its Phase A (asynchronously, on a copy
stream) and restored for its Phase C: prefetched one layer ahead when an
HBM budget check allows, demand-loaded otherwise.  That turns the dormant
set into Phase-B HBM headroom (the paper's Table 6).  Every launch is the
same with and without offload, so the results are bitwise identical.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch

from . import binding as B
from .layer import DecoderLayer, W_KEYS


# ---------------------------------------------------------------- host side
class PinnedPool:
    """A pinned host staging arena sized from the dormant footprint with
    headroom (Sec. 4.3: about 1.5x), handing out aligned slices; when it is
    exhausted, requests fall back to one pinned allocation each (correct,
    slower)."""

    def __init__(self, nbytes: int, alloc: Optional[Callable[[int], torch.Tensor]] = None,
                 align: int = 4096):
        self._alloc = alloc or (lambda n: torch.empty(n, dtype=torch.uint8, pin_memory=True))
        self.align = align
        self.capacity = max(int(nbytes), 0)
        self.arena = self._alloc(self.capacity) if self.capacity else None
        self.offset = 0
        self.fallbacks = 0

    def take(self, nbytes: int) -> torch.Tensor:
        start = (self.offset + self.align - 1) // self.align * self.align
        if self.arena is not None and start + nbytes <= self.capacity:
            self.offset = start + nbytes
            return self.arena[start:start + nbytes]
        self.fallbacks += 1
        return self._alloc(nbytes)

    def reset(self) -> None:
        self.offset = 0


@dataclass
class HbmBudget:
    """Prefetch guard (Sec. 4.3): a prefetch of `need` bytes (times `slack`)
    is issued only if the memory it could come from keeps `reserve` bytes
    spare: the driver-visible free memory plus the allocator's cached but
    unused blocks, capped by `limit` minus what the allocator has handed
    out."""
    reserve: int = 1 << 30
    slack: float = 1.1
    limit: Optional[int] = None  # cap on allocated bytes, None = device memory
    mem_get_info: Callable[[], Tuple[int, int]] = None
    allocated: Callable[[], int] = None
    reserved: Callable[[], int] = None

    def headroom(self) -> int:
        free, total = (self.mem_get_info or torch.cuda.mem_get_info)()
        held = (self.allocated or torch.cuda.memory_allocated)()
        cached = (self.reserved or torch.cuda.memory_reserved)() - held
        limit = self.limit if self.limit is not None else total
        return min(free + max(cached, 0), limit - held)

    def allows(self, need: int) -> bool:
        return self.headroom() - int(need * self.slack) >= self.reserve


# ---------------------------------------------------------------- the stack
# what Phase A of a layer saves for its Phase C besides the hot prefix K/V
# (the layer's prefix output is the next layer's input "x")
_DORMANT = ("x", "n1", "r1", "q", "o", "lse", "h", "n2", "r2", "g", "u", "m")


class DecoderStack:
    """``layers`` decoder layers over one prompt group on one GPU.

    Inputs come either from a synthetic stack group (``inp`` from
    ``synthetic.layer.make_stack_group``: weights per layer, the group's
    inputs to the bottom layer and upstream adjoints at the top), or, with
    ``inp=None``, are drawn on the device from (``shape``, ``layers``,
    ``seed``): weights N(0, std^2), inputs and adjoints N(0, 1), in bf16."""

    def __init__(self, inp: Optional[Dict] = None, *, shape=None, layers: Optional[int] = None,
                 seed: int = 0, device="cuda:0", offload: bool = False, pool_factor: float = 1.5,
                 budget: Optional[HbmBudget] = None):
        self.dev = torch.device(device)
        bf = torch.bfloat16
        if inp is not None:
            shape, layers = inp["shape"], len(inp["weights"])
            up = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(device=self.dev, dtype=bf)
            weights = [{k: up(w[k]) for k in W_KEYS} for w in inp["weights"]]
            self.x_p = up(inp["x_p"])
            self.x_s = [up(x) for x in inp["x_s"]]
            self.dy_s = [up(x) for x in inp["dy_s"]]
            dy_p = [up(x) for x in inp["dy_p"]]
        else:
            g = torch.Generator(device=self.dev)
            g.manual_seed(seed)
            rnd = lambda *sh, std=1.0: (torch.randn(*sh, generator=g, device=self.dev) * std).to(bf)
            h, hq, hkv, d, I = shape.hidden, shape.num_q_heads, shape.num_kv_heads, shape.head_dim, \
                shape.intermediate
            sd = shape.weight_std
            weights = [{"wq": rnd(h, hq * d, std=sd), "wk": rnd(h, hkv * d, std=sd),
                        "wv": rnd(h, hkv * d, std=sd), "wo": rnd(hq * d, h, std=sd), "wg": rnd(h, I, std=sd),
                        "wu": rnd(h, I, std=sd), "wd": rnd(I, h, std=sd)} for _ in range(layers)]
            self.x_p = rnd(shape.prefix_len, h)
            self.x_s = [rnd(s, h) for s in shape.suffix_lens]
            self.dy_s = [rnd(s, h) for s in shape.suffix_lens]
            dy_p = [rnd(shape.prefix_len, h) for _ in shape.suffix_lens]
        self.shape = shape
        # the top layer's G_Y = sum_i dY_P(i), summed in fp32 and rounded once
        self.g_y = (torch.stack([x.float() for x in dy_p]).sum(0).to(bf) if dy_p
                    else torch.zeros_like(self.x_p))
        self.dy_p = dy_p
        self.ws = torch.empty(DecoderLayer.workspace_bytes(shape), dtype=torch.uint8, device=self.dev)
        self.layers = [DecoderLayer.of_weights(shape, w, self.dev, self.ws) for w in weights]
        self.offload = offload
        self.budget = budget or HbmBudget()
        self.copy_stream = torch.cuda.Stream(self.dev) if offload else None
        P, hid, I = shape.prefix_len, shape.hidden, shape.intermediate
        hq, d = shape.num_q_heads, shape.head_dim
        # bytes of one layer's dormant set: bf16 rows of the hidden width
        # (x, n1, h, n2), the query width (q, o) and the MLP width (g, u, m),
        # fp32 norm statistics (r1, r2) and LSE
        self.layer_dormant_bytes = P * (2 * (4 * hid + 2 * hq * d + 3 * I) + 4 * (2 + hq))
        self.dormant_bytes = self.layer_dormant_bytes * layers
        self.pool = PinnedPool(int(self.dormant_bytes * pool_factor)) if offload else None
        self.stats = {"prefetched": 0, "demand_loaded": 0, "pool_fallbacks": 0}
        L = layers
        self._saved: List[Optional[Dict[str, torch.Tensor]]] = [None] * L
        self._host: List[Dict[str, torch.Tensor]] = [dict() for _ in range(L)]
        self._ready: List[Optional[torch.cuda.Event]] = [None] * L
        self._packed: List[Optional[torch.cuda.Event]] = [None] * L

    # ------------------------------------------------------ offload helpers
    def _pack(self, l: int) -> None:
        """Layer l's dormant set to pinned host memory, then released."""
        main = torch.cuda.current_stream(self.dev)
        done = torch.cuda.Event()
        done.record(main)
        cs = self.copy_stream
        cs.wait_event(done)
        c = self._saved[l]
        with torch.cuda.stream(cs):
            for k in _DORMANT:
                x = c[k]
                h = self.pool.take(x.numel() * x.element_size()).view(x.dtype).view(x.shape)
                h.copy_(x, non_blocking=True)
                self._host[l][k] = h
                x.record_stream(cs)
                c[k] = None
            packed = torch.cuda.Event()
            packed.record(cs)
            self._packed[l] = packed
        self.stats["pool_fallbacks"] = self.pool.fallbacks

    def _restore(self, l: int, prefetch: bool) -> None:
        """Layer l's dormant set back to the device: on the copy stream
        (prefetch) or on the compute stream right before use (demand load,
        after the pack's copies have landed)."""
        c = self._saved[l]
        stream = self.copy_stream if prefetch else torch.cuda.current_stream(self.dev)
        if not prefetch and self._packed[l] is not None:
            stream.wait_event(self._packed[l])
        with torch.cuda.stream(stream):
            for k in _DORMANT:
                h = self._host[l][k]
                x = torch.empty(h.shape, dtype=h.dtype, device=self.dev)
                x.copy_(h, non_blocking=True)
                c[k] = x
            if prefetch:
                e = torch.cuda.Event()
                e.record(stream)
                self._ready[l] = e
        self.stats["prefetched" if prefetch else "demand_loaded"] += 1

    def _try_prefetch(self, l: int) -> None:
        if l < 0 or not self.offload or self._saved[l]["q"] is not None or self._ready[l] is not None:
            return
        if self.budget.allows(self.layer_dormant_bytes):
            self._restore(l, prefetch=True)

    def _ensure_resident(self, l: int) -> None:
        c = self._saved[l]
        if c["q"] is None:
            self._restore(l, prefetch=False)
        elif self._ready[l] is not None:
            main = torch.cuda.current_stream(self.dev)
            main.wait_event(self._ready[l])
            for k in _DORMANT:
                c[k].record_stream(main)
            self._ready[l] = None

    # ------------------------------------------------------------ schedule
    def run_schedule(self, on_phase: Optional[Callable[[str], None]] = None) -> Dict:
        """The schedule over the stack; returns the top layer's outputs
        y_p, y_s, the bottom layer's input gradients dx_p, dx_s and every
        layer's weight gradients dw (fp32).  ``on_phase(name)`` is called
        after the launches of "A", "B" and "C" are issued."""
        mark = on_phase or (lambda name: None)
        shp, P, L = self.shape, self.shape.prefix_len, len(self.layers)
        if self.offload:
            self.pool.reset()
            self._ready = [None] * L
            self._packed = [None] * L
        dws = [layer._zero_dw() for layer in self.layers]
        # Phase A: the prefix through every layer once; each layer's dormant
        # set leaves for the host as soon as the layer is done
        x = self.x_p
        for l, layer in enumerate(self.layers):
            B.gkv_cache_zero(layer.dims, layer.gk, layer.gv)

            def prefix_attn(c, layer=layer):
                B.prefix_fwd(layer.dims, c["q"], c["k"], c["v"], c["o"], c["lse"])

            c = layer._forward(x, 0, prefix_attn)
            x = c.pop("y")
            self._saved[l] = c
            if self.offload:
                self._pack(l)
        y_p = x
        mark("A")
        # Phase B: each suffix microbatch forward through the layers and
        # backward from the top; its activations live only inside it
        y_s, dx_s = [], []
        for i, (x_s, dy_s) in enumerate(zip(self.x_s, self.dy_s)):
            s = x_s.shape[0]
            acts = []
            x = x_s
            for l, layer in enumerate(self.layers):
                kp, vp, cu = self._saved[l]["k"], self._saved[l]["v"], layer._cu_of(s)

                def suffix_attn(c, layer=layer, kp=kp, vp=vp, s=s, cu=cu):
                    B.suffix_attn_fwd(layer.dims, kp, vp, c["q"], c["k"], c["v"], cu, 1, s, s, c["o"], c["lse"],
                                      self.ws)

                c = layer._forward(x, P, suffix_attn)
                x = c["y"]
                acts.append(c)
            y_s.append(x)
            if i == len(self.x_s) - 1:
                self._try_prefetch(L - 1)  # the first Phase C layer, during the last backward
            g = dy_s
            for l in reversed(range(L)):
                layer, c = self.layers[l], acts[l]
                kp, vp, cu = self._saved[l]["k"], self._saved[l]["v"], layer._cu_of(s)

                def suffix_attn_bwd(c, do, dq, dk, dv, layer=layer, kp=kp, vp=vp, s=s, cu=cu):
                    B.suffix_attn_bwd_accum(layer.dims, kp, vp, c["q"], c["k"], c["v"], c["o"], c["lse"], do, cu,
                                            1, s, s, dq, dk, dv, layer.gk, layer.gv, self.ws)

                g = layer._backward(c, g, P, suffix_attn_bwd, dws[l])
                acts[l] = None
            dx_s.append(g)
            del acts
        mark("B")
        # Phase C: the prefix backward from the top layer down, each layer's
        # input adjoint chained to the layer below; the next layer's dormant
        # set prefetched while this one runs
        g = self.g_y
        for l in reversed(range(L)):
            if self.offload:
                self._ensure_resident(l)
                self._try_prefetch(l - 1)
            layer, c = self.layers[l], self._saved[l]

            def prefix_attn_bwd(c, do, dq, dk, dv, layer=layer):
                B.prefix_bwd(layer.dims, c["q"], c["k"], c["v"], c["o"], c["lse"], do, layer.gk, layer.gv,
                             dq, dk, dv, self.ws)

            g = layer._backward(c, g, 0, prefix_attn_bwd, dws[l])
            self._saved[l] = None
        mark("C")
        return {"y_p": y_p, "y_s": y_s, "dx_p": g, "dx_s": dx_s, "dw": dws}

    # --------------------------------------------------------------- dense
    def run_dense(self) -> Dict:
        """Every trajectory [P||S(i)] through all layers with causal
        attention over the whole sequence, upstream [dY_P(i); dY_S(i)] at
        the top; the prefix's and the weights' gradients summed."""
        shp, P, L = self.shape, self.shape.prefix_len, len(self.layers)
        dws = [layer._zero_dw() for layer in self.layers]
        y_s, dx_s, y_p = [], [], None
        dx_p = torch.zeros(P, shp.hidden, dtype=torch.float32, device=self.dev)
        for x_s, dy_s, dy_p in zip(self.x_s, self.dy_s, self.dy_p):
            x = torch.cat([self.x_p, x_s])
            Lt = x.shape[0]
            acts = []
            for layer in self.layers:
                dims, ws, zero = layer._dims_for(Lt)

                def attn(c, dims=dims):
                    B.prefix_fwd(dims, c["q"], c["k"], c["v"], c["o"], c["lse"])

                c = layer._forward(x, 0, attn)
                x = c["y"]
                acts.append(c)
            g = torch.cat([dy_p, dy_s])
            for l in reversed(range(L)):
                layer = self.layers[l]
                dims, ws, zero = layer._dims_for(Lt)

                def attn_bwd(c, do, dq, dk, dv, dims=dims, ws=ws, zero=zero):
                    B.prefix_bwd(dims, c["q"], c["k"], c["v"], c["o"], c["lse"], do, zero[0], zero[1], dq, dk, dv,
                                 ws)

                g = layer._backward(acts[l], g, 0, attn_bwd, dws[l])
                acts[l] = None
            dx_p += g[:P].float()
            dx_s.append(g[P:])
            y_s.append(x[P:])
            if y_p is None:
                y_p = x[:P]
        return {"y_p": y_p, "y_s": y_s, "dx_p": dx_p.to(torch.bfloat16), "dx_s": dx_s, "dw": dws}
