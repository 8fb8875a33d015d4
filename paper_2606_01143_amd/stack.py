"""A stack of attention layers run through the three-phase schedule with the
prefix-state lifecycle of paper Sec. 3.3 and Sec. 4.3.

Per layer the schedule keeps a *hot* set resident (K_1, V_1 and the gK/gV
cache: Phase B reads and updates them) and a *dormant* set that Phase A
produces and only Phase C consumes: here the prefix queries, the prefix
outputs and LSE, and the prefix-row adjoint G_Y (the attention part of the
saved prefix activations).  With ``offload=True`` the dormant set of each
layer is packed to pinned host memory right after the layer's Phase A
(asynchronously, on a copy stream) and restored for Phase C: prefetched one
layer ahead when an HBM budget check allows, otherwise demand-loaded right
before use.  That turns the dormant set into Phase-B HBM headroom (the
measurement of the paper's Table 6).

Layers are independent attention problems (the projections that would link
them are outside the hot path), each with seeded synthetic inputs generated
on the device.  Phase B takes one suffix per microbatch: the microbatch's
tensors for every layer are made at its start and released after its
backward, as a trainer's activations are.  Every launch is the same in both
modes, so outputs and caches are bitwise identical with and without offload
(with ``atomic_dq=True`` dQ agrees to rounding only).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import torch

from . import binding as B


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
@dataclass(frozen=True)
class StackShape:
    layers: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    prefix_len: int
    suffix_lens: Tuple[int, ...]


_DORMANT = ("q_p", "o_p", "lse_p", "g_y")


class StackedGroup:
    def __init__(self, shape: StackShape, seed: int = 0, device="cuda:0", offload: bool = False,
                 pool_factor: float = 1.5, budget: Optional[HbmBudget] = None,
                 keep_suffix_grads: bool = False, atomic_dq: bool = False):
        self.shape = shape
        self.dev = torch.device(device)
        self.seed = seed
        self.offload = offload
        self.budget = budget or HbmBudget()
        self.keep_suffix_grads = keep_suffix_grads
        L, hq, hkv, d, P = shape.layers, shape.num_q_heads, shape.num_kv_heads, shape.head_dim, shape.prefix_len
        self.dims = B.make_dims(hq, hkv, d, P, "bf16", atomic_dq=atomic_dq)
        bf = torch.bfloat16
        # hot set and prefix outputs stay resident; dormant set may move
        self.layers: List[Dict[str, torch.Tensor]] = []
        for l in range(L):
            g = self._gen(l, 0)
            t = {"q_p": self._randn((P, hq, d), g), "k_p": self._randn((P, hkv, d), g),
                 "v_p": self._randn((P, hkv, d), g), "g_y": self._randn((P, hq, d), g),
                 "o_p": torch.empty(P, hq, d, dtype=bf, device=self.dev),
                 "lse_p": torch.empty(P, hq, dtype=torch.float32, device=self.dev),
                 "gk": torch.empty(P, hkv, d, dtype=torch.float32, device=self.dev),
                 "gv": torch.empty(P, hkv, d, dtype=torch.float32, device=self.dev),
                 "dq_p": torch.empty(P, hq, d, dtype=bf, device=self.dev),
                 "dk_p": torch.empty(P, hkv, d, dtype=bf, device=self.dev),
                 "dv_p": torch.empty(P, hkv, d, dtype=bf, device=self.dev)}
            self.layers.append(t)
        self.dormant_bytes = sum(self.layers[0][k].numel() * self.layers[0][k].element_size()
                                 for k in _DORMANT) * L
        mx = max(shape.suffix_lens)
        need = max(B.workspace_size(B.OP_SUFFIX_FWD, self.dims, 1, mx, mx),
                   B.workspace_size(B.OP_SUFFIX_BWD, self.dims, 1, mx, mx),
                   B.workspace_size(B.OP_PREFIX_BWD, self.dims), 256)
        self.ws = torch.empty(need, dtype=torch.uint8, device=self.dev)
        self.cu = {s: torch.tensor([0, s], dtype=torch.int32, device=self.dev) for s in set(shape.suffix_lens)}
        self.copy_stream = torch.cuda.Stream(self.dev) if offload else None
        self.pool = PinnedPool(int(self.dormant_bytes * pool_factor)) if offload else None
        self.host: List[Dict[str, torch.Tensor]] = [dict() for _ in range(L)]
        self.ready: List[Optional[torch.cuda.Event]] = [None] * L
        self.packed: List[Optional[torch.cuda.Event]] = [None] * L
        self.stats = {"prefetched": 0, "demand_loaded": 0, "pool_fallbacks": 0}
        self.suffix_grads: List[Dict[str, torch.Tensor]] = []

    # -------------------------------------------------------------- inputs
    def _gen(self, layer: int, mb: int) -> torch.Generator:
        g = torch.Generator(device=self.dev)
        g.manual_seed(self.seed * 1_000_003 + layer * 1009 + mb)
        return g

    def _randn(self, shape, g) -> torch.Tensor:
        return torch.randn(shape, generator=g, device=self.dev, dtype=torch.float32).to(torch.bfloat16)

    # ------------------------------------------------------ offload helpers
    def _pack(self, l: int) -> None:
        """Dormant set of layer l to pinned host memory, then release it."""
        main = torch.cuda.current_stream(self.dev)
        done = torch.cuda.Event()
        done.record(main)
        cs = self.copy_stream
        cs.wait_event(done)
        t = self.layers[l]
        with torch.cuda.stream(cs):
            for k in _DORMANT:
                x = t[k]
                h = self.pool.take(x.numel() * x.element_size()).view(x.dtype).view(x.shape)
                h.copy_(x, non_blocking=True)
                self.host[l][k] = h
                x.record_stream(cs)
                t[k] = None
            # the host copies are complete once this event has passed: a
            # restore on another stream waits for it
            packed = torch.cuda.Event()
            packed.record(cs)
            self.packed[l] = packed
        self.stats["pool_fallbacks"] = self.pool.fallbacks

    def _restore(self, l: int, prefetch: bool) -> None:
        """Dormant set of layer l back to the device: on the copy stream
        (prefetch) or on the compute stream right before use (demand load)."""
        t = self.layers[l]
        stream = self.copy_stream if prefetch else torch.cuda.current_stream(self.dev)
        # the pack of this layer ran on the copy stream: a demand load on
        # the compute stream must not read the pinned slices before it ends
        if not prefetch and self.packed[l] is not None:
            stream.wait_event(self.packed[l])
        with torch.cuda.stream(stream):
            for k in _DORMANT:
                h = self.host[l][k]
                x = torch.empty(h.shape, dtype=h.dtype, device=self.dev)
                x.copy_(h, non_blocking=True)
                t[k] = x
            if prefetch:
                e = torch.cuda.Event()
                e.record(stream)
                self.ready[l] = e
        self.stats["prefetched" if prefetch else "demand_loaded"] += 1

    def _try_prefetch(self, l: int) -> None:
        if l < 0 or not self.offload or self.layers[l]["q_p"] is not None or self.ready[l] is not None:
            return
        need = self.dormant_bytes // self.shape.layers
        if self.budget.allows(need):
            self._restore(l, prefetch=True)

    def _ensure_resident(self, l: int) -> None:
        t = self.layers[l]
        if t["q_p"] is None:
            self._restore(l, prefetch=False)
        elif self.ready[l] is not None:
            main = torch.cuda.current_stream(self.dev)
            main.wait_event(self.ready[l])
            for k in _DORMANT:
                t[k].record_stream(main)
            self.ready[l] = None

    # ------------------------------------------------------------ schedule
    def run(self, on_phase: Optional[Callable[[str], None]] = None) -> None:
        mark = on_phase or (lambda name: None)
        shp, dims = self.shape, self.dims
        L, hq, hkv, d = shp.layers, shp.num_q_heads, shp.num_kv_heads, shp.head_dim
        bf = torch.bfloat16
        if self.offload:
            self.pool.reset()
            self.ready = [None] * L
            self.packed = [None] * L
        # Phase A: prefix forward layer by layer; each layer's dormant set
        # leaves for the host as soon as the layer is done
        for l in range(L):
            t = self.layers[l]
            B.gkv_cache_zero(dims, t["gk"], t["gv"])
            B.prefix_fwd(dims, t["q_p"], t["k_p"], t["v_p"], t["o_p"], t["lse_p"])
            if self.offload:
                self._pack(l)
        mark("A")
        # Phase B: one suffix per microbatch, forward through the layers and
        # backward in reverse; the microbatch's tensors live only inside it
        self.suffix_grads = []
        for i, s in enumerate(shp.suffix_lens):
            acts = []
            for l in range(L):
                g = self._gen(l, 1 + i)
                a = {"q": self._randn((s, hq, d), g), "k": self._randn((s, hkv, d), g),
                     "v": self._randn((s, hkv, d), g), "do": self._randn((s, hq, d), g),
                     "o": torch.empty(s, hq, d, dtype=bf, device=self.dev),
                     "lse": torch.empty(s, hq, dtype=torch.float32, device=self.dev)}
                t = self.layers[l]
                B.suffix_attn_fwd(dims, t["k_p"], t["v_p"], a["q"], a["k"], a["v"], self.cu[s], 1, s, s,
                                  a["o"], a["lse"], self.ws)
                acts.append(a)
            if i == len(shp.suffix_lens) - 1:
                self._try_prefetch(L - 1)  # the first Phase C layer, during the last backward
            grads = {}
            for l in reversed(range(L)):
                a, t = acts[l], self.layers[l]
                dq = torch.empty_like(a["q"])
                dk = torch.empty_like(a["k"])
                dv = torch.empty_like(a["v"])
                B.suffix_attn_bwd_accum(dims, t["k_p"], t["v_p"], a["q"], a["k"], a["v"], a["o"], a["lse"],
                                        a["do"], self.cu[s], 1, s, s, dq, dk, dv, t["gk"], t["gv"], self.ws)
                if self.keep_suffix_grads:
                    grads[l] = (dq, dk, dv)
                acts[l] = None
            self.suffix_grads.append(grads)
            del acts
        mark("B")
        # Phase C: prefix backward from the last layer down, the next layer's
        # dormant set prefetched while this one runs
        for l in reversed(range(L)):
            if self.offload:
                self._ensure_resident(l)
                self._try_prefetch(l - 1)
            t = self.layers[l]
            B.prefix_bwd(dims, t["q_p"], t["k_p"], t["v_p"], t["o_p"], t["lse_p"], t["g_y"], t["gk"],
                         t["gv"], t["dq_p"], t["dk_p"], t["dv_p"], self.ws)
        mark("C")
