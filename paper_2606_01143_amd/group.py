"""One GRPO prompt group resident in HBM, run through libspr.

PyTorch only provides device memory and the stream here; every step of the
schedule runs in the HIP library through ``binding``.

``DeviceGroup.run_schedule`` is the paper's three-phase schedule (Sec. 3.2):
zero the gK/gV cache, Phase A ``prefix_fwd`` once, Phase B
``suffix_attn_fwd`` + ``suffix_attn_bwd_accum`` per suffix microbatch (a
microbatch is a contiguous run of the packed suffixes; packed layout of
Sec. 4.2), Phase C ``prefix_bwd`` once.  ``run_dense`` is the comparison:
``dense_recompute_baseline`` over every [P||S(i)].

Streams: the Phase B suffix forwards read only inputs, so by default they
run in order on a side stream while the backwards run in order on the
caller's stream.  A suffix backward waits for its own forward.  Phase A and
Phase C run on the caller's stream after the last backward; the gK/gV
cache updates therefore stay in microbatch order.  The work items are the
same launches with the same arguments, so the results are identical to the
serial order.  The overlap only fills the idle compute units at the tail of
each launch.  Phase A stays off the side stream: beside the backwards it
competes for the L2 their row-tile order relies on.  Measured, that made
the step up to 3% slower than the serial order at long prefixes, and never
faster than running Phase A just before Phase C.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch

from . import binding as B

_TORCH_DT = {"bf16": torch.bfloat16, "f32": torch.float32}
OUTPUT_KEYS = ["o_p", "lse_p", "o_s", "lse_s", "dq_p", "dk_p", "dv_p", "dq_s", "dk_s", "dv_s"]


def plan_suffix_waves(lens: Sequence[int], budget_tokens: int,
                      layout: str = "packed") -> List[Tuple[int, int]]:
    """Split the suffixes, in order, into microbatches ("suffix waves", paper
    Sec. 4.2) whose token footprint stays within ``budget_tokens``: the sum of
    the lengths for the packed layout, the count times the longest length
    for the padded layout.  Greedy: each wave takes suffixes while the next
    one still fits; a suffix larger than the budget gets a wave of its own.
    Any split gives the same group gradients (Prop. 1), so the split only
    trades memory for launch count."""
    if layout not in ("packed", "padded"):
        raise ValueError(f"unknown layout {layout!r}")
    if budget_tokens < 1:
        raise ValueError("budget_tokens must be >= 1")
    waves, a = [], 0
    n = len(lens)
    while a < n:
        b, tot, mx = a, 0, 0
        while b < n:
            t2, m2 = tot + lens[b], max(mx, lens[b])
            cost = t2 if layout == "packed" else (b + 1 - a) * m2
            if b > a and cost > budget_tokens:
                break
            tot, mx, b = t2, m2, b + 1
        waves.append((a, b))
        a = b
    return waves


class DeviceGroup:
    """Inputs, outputs, cache and workspace of one prompt group on one GPU.

    ``inp`` is a synthetic group (see ``synthetic.make_group``): float32
    arrays holding values exactly representable in the storage dtype.
    ``layout="padded"`` runs Phase B through the batch-plus-padding calls:
    each microbatch's suffixes are held as [n, longest, H, d] tensors (built
    once per microbatch) and the padded outputs are kept per microbatch
    (``gather_padded_outputs`` copies their valid rows into ``self.out``).
    """

    def __init__(self, inp: Dict, device="cuda:0", softmax_scale: float = 0.0,
                 deterministic: bool = False, dense: bool = True, atomic_dq: bool = False,
                 microbatch_splits: Optional[Sequence[Sequence[Tuple[int, int]]]] = None,
                 layout: str = "packed"):
        if layout not in ("packed", "padded"):
            raise ValueError(f"unknown layout {layout!r}")
        self.layout = layout
        self._padded: Dict[Tuple[int, int], Dict[str, torch.Tensor]] = {}
        shp = inp["shape"]
        self.shape = shp
        self.device = torch.device(device)
        dt = _TORCH_DT[shp.dtype]
        self.dtype = dt
        hq, hkv, d, p = shp.num_q_heads, shp.num_kv_heads, shp.head_dim, shp.prefix_len
        t = shp.total_suffix
        self.dims = B.make_dims(hq, hkv, d, p, shp.dtype, softmax_scale, deterministic, atomic_dq)
        self.lens = [int(x) for x in inp["suffix_lens"]]
        self.cu_host = [int(x) for x in inp["cu_seqlens"]]

        def up(x, dtype=dt):
            return torch.from_numpy(np.ascontiguousarray(x)).to(device=self.device, dtype=dtype)

        self.q_p, self.k_p, self.v_p = up(inp["q_p"]), up(inp["k_p"]), up(inp["v_p"])
        self.q_s, self.k_s, self.v_s = up(inp["q_s"]), up(inp["k_s"]), up(inp["v_s"])
        self.do_s = up(inp["do_s"])
        self.g_y = up(inp["g_y"])
        self.do_p = up(inp["do_p"]) if dense else None
        self.cu = up(inp["cu_seqlens"], torch.int32)
        self._cu_cache: Dict[Tuple[int, int], torch.Tensor] = {}

        def empty(*shape, dtype=dt):
            return torch.empty(*shape, device=self.device, dtype=dtype)

        self.out = {
            "o_p": empty(p, hq, d), "lse_p": empty(p, hq, dtype=torch.float32),
            "o_s": empty(t, hq, d), "lse_s": empty(t, hq, dtype=torch.float32),
            "dq_p": empty(p, hq, d), "dk_p": empty(p, hkv, d), "dv_p": empty(p, hkv, d),
            "dq_s": empty(t, hq, d), "dk_s": empty(t, hkv, d), "dv_s": empty(t, hkv, d),
        }
        self.gk = empty(p, hkv, d, dtype=torch.float32)
        self.gv = empty(p, hkv, d, dtype=torch.float32)
        self.dense_out = None
        if dense:
            self.dense_out = {k: torch.empty_like(v) for k, v in self.out.items()}

        # one workspace large enough for every call this group makes
        splits = list(microbatch_splits or []) + [self.default_microbatches(),
                                                  [(0, shp.n)]]
        need = B.workspace_size(B.OP_PREFIX_BWD, self.dims)
        for mbs in splits:
            for a, b in mbs:
                nmb, mx, tot = self._mb_sizes(a, b)
                need = max(need, B.workspace_size(B.OP_SUFFIX_FWD, self.dims, nmb, mx, tot),
                           B.workspace_size(B.OP_SUFFIX_BWD, self.dims, nmb, mx, tot))
        if dense:
            need = max(need, B.workspace_size(B.OP_DENSE_BASELINE, self.dims, shp.n,
                                              max(self.lens), t))
        self.ws = torch.empty(max(need, 256), device=self.device, dtype=torch.uint8)
        # the suffix forwards' own workspace: they run beside the backwards
        need_f = 256
        for mbs in splits:
            for a, b in mbs:
                nmb, mx, tot = self._mb_sizes(a, b)
                need_f = max(need_f, B.workspace_size(B.OP_SUFFIX_FWD, self.dims, nmb, mx, tot))
        if layout == "padded":
            for mbs in splits:
                for a, b in mbs:
                    nmb, mx, _ = self._mb_sizes(a, b)
                    need = max(need, B.workspace_size(B.OP_SUFFIX_BWD_PADDED, self.dims, nmb, mx),
                               B.workspace_size(B.OP_SUFFIX_FWD_PADDED, self.dims, nmb, mx))
                    need_f = max(need_f, B.workspace_size(B.OP_SUFFIX_FWD_PADDED, self.dims, nmb, mx))
            self.ws = torch.empty(max(need, 256), device=self.device, dtype=torch.uint8)
        self.ws_fwd = torch.empty(need_f, device=self.device, dtype=torch.uint8)
        self._side = None  # suffix forward stream, made on first use

    # ------------------------------------------------------------------
    def default_microbatches(self) -> List[Tuple[int, int]]:
        """One suffix per microbatch, in order (the paper's timing choice)."""
        return [(i, i + 1) for i in range(self.shape.n)]

    def _mb_sizes(self, a: int, b: int):
        return b - a, max(self.lens[a:b]), self.cu_host[b] - self.cu_host[a]

    def _mb_cu(self, a: int, b: int) -> torch.Tensor:
        key = (a, b)
        if key not in self._cu_cache:
            base = self.cu_host[a]
            host = [x - base for x in self.cu_host[a:b + 1]]
            nmb, mx, tot = self._mb_sizes(a, b)
            B.check_cu_seqlens(host, nmb, mx, tot)  # once per microbatch, before any launch
            self._cu_cache[key] = torch.tensor(host, dtype=torch.int32, device=self.device)
        return self._cu_cache[key]

    def prepare(self, microbatches: Sequence[Tuple[int, int]]) -> None:
        """Build the per-microbatch cu_seqlens tensors (and, for the padded
        layout, the padded tensors) ahead of a timed run."""
        for a, b in microbatches:
            self._mb_cu(a, b)
            if self.layout == "padded":
                self._mb_padded(a, b)

    def _mb_padded(self, a: int, b: int) -> Dict[str, torch.Tensor]:
        key = (a, b)
        if key not in self._padded:
            shp = self.shape
            nmb, mx, _ = self._mb_sizes(a, b)
            hq, hkv, d = shp.num_q_heads, shp.num_kv_heads, shp.head_dim

            def pad(x, h):
                y = torch.zeros(nmb, mx, h, d, device=self.device, dtype=self.dtype)
                for i in range(a, b):
                    y[i - a, :self.lens[i]] = x[self.cu_host[i]:self.cu_host[i + 1]]
                return y

            def empty(h, dtype=None):
                return torch.empty(nmb, mx, h, d, device=self.device, dtype=dtype or self.dtype)

            self._padded[key] = {
                "q": pad(self.q_s, hq), "k": pad(self.k_s, hkv), "v": pad(self.v_s, hkv),
                "do": pad(self.do_s, hq),
                "lens": torch.tensor(self.lens[a:b], dtype=torch.int32, device=self.device),
                "o": empty(hq), "lse": torch.empty(nmb, mx, hq, device=self.device, dtype=torch.float32),
                "dq": empty(hq), "dk": empty(hkv), "dv": empty(hkv)}
        return self._padded[key]

    def gather_padded_outputs(self) -> None:
        """Copy the valid rows of every padded microbatch output into the
        packed ``self.out`` tensors."""
        for (a, b), t in self._padded.items():
            for i in range(a, b):
                r0, r1, L = self.cu_host[i], self.cu_host[i + 1], self.lens[i]
                for src, dst in (("o", "o_s"), ("lse", "lse_s"), ("dq", "dq_s"), ("dk", "dk_s"),
                                 ("dv", "dv_s")):
                    self.out[dst][r0:r1] = t[src][i - a, :L]

    # ------------------------------------------------------------------
    def run_schedule(self, microbatches: Optional[Sequence[Tuple[int, int]]] = None,
                     use_gy: bool = True, stream=None, mark=None, overlap: bool = True) -> None:
        """Three-phase schedule; results land in ``self.out``, ``self.gk``, ``self.gv``.

        ``overlap`` runs the suffix forwards on a side stream (see the
        module docstring); ``overlap=False`` issues every launch in
        order on ``stream``.  ``mark(name)``, if given, is called after each
        phase's launches are issued ("zero", "A", "B_fwd", "B_bwd" per
        microbatch, "C"), e.g. to record events for per-phase times; it
        implies the serial order."""
        mbs = list(microbatches) if microbatches is not None else self.default_microbatches()
        if overlap and mark is None:
            self._run_overlapped(mbs, use_gy, stream)
            return
        dims, o = self.dims, self.out
        mark = mark or (lambda name: None)
        B.gkv_cache_zero(dims, self.gk, self.gv, stream)
        mark("zero")
        # Phase A: prefix forward once
        B.prefix_fwd(dims, self.q_p, self.k_p, self.v_p, o["o_p"], o["lse_p"], stream)
        mark("A")
        # Phase B: suffix microbatches read K_P/V_P and accumulate gK/gV
        for a, b in mbs:
            self._suffix_fwd(a, b, self.ws, stream)
            mark("B_fwd")
            self._suffix_bwd(a, b, stream)
            mark("B_bwd")
        # Phase C: prefix backward once on the accumulated cache
        self._prefix_bwd(use_gy, stream)
        mark("C")

    def _suffix_fwd(self, a: int, b: int, ws, stream) -> None:
        nmb, mx, tot = self._mb_sizes(a, b)
        if self.layout == "padded":
            t = self._mb_padded(a, b)
            B.suffix_attn_fwd_padded(self.dims, self.k_p, self.v_p, t["q"], t["k"], t["v"], t["lens"],
                                     nmb, mx, t["o"], t["lse"], ws, stream)
            return
        r0, r1 = self.cu_host[a], self.cu_host[b]
        o = self.out
        B.suffix_attn_fwd(self.dims, self.k_p, self.v_p, self.q_s[r0:r1], self.k_s[r0:r1],
                          self.v_s[r0:r1], self._mb_cu(a, b), nmb, mx, tot, o["o_s"][r0:r1],
                          o["lse_s"][r0:r1], ws, stream)

    def _suffix_bwd(self, a: int, b: int, stream) -> None:
        nmb, mx, tot = self._mb_sizes(a, b)
        if self.layout == "padded":
            t = self._mb_padded(a, b)
            B.suffix_attn_bwd_accum_padded(self.dims, self.k_p, self.v_p, t["q"], t["k"], t["v"], t["o"],
                                           t["lse"], t["do"], t["lens"], nmb, mx, t["dq"], t["dk"],
                                           t["dv"], self.gk, self.gv, self.ws, stream)
            return
        r0, r1 = self.cu_host[a], self.cu_host[b]
        o = self.out
        B.suffix_attn_bwd_accum(self.dims, self.k_p, self.v_p, self.q_s[r0:r1], self.k_s[r0:r1],
                                self.v_s[r0:r1], o["o_s"][r0:r1], o["lse_s"][r0:r1],
                                self.do_s[r0:r1], self._mb_cu(a, b), nmb, mx, tot,
                                o["dq_s"][r0:r1], o["dk_s"][r0:r1], o["dv_s"][r0:r1], self.gk,
                                self.gv, self.ws, stream)

    def _prefix_bwd(self, use_gy: bool, stream) -> None:
        o = self.out
        B.prefix_bwd(self.dims, self.q_p, self.k_p, self.v_p, o["o_p"], o["lse_p"],
                     self.g_y if use_gy else None, self.gk, self.gv, o["dq_p"], o["dk_p"],
                     o["dv_p"], self.ws, stream)

    def _run_overlapped(self, mbs, use_gy: bool, stream) -> None:
        main = stream if stream is not None else torch.cuda.current_stream(self.device)
        if self._side is None:
            # default priority: the side stream only fills idle compute units
            self._side = torch.cuda.Stream(self.device)
        s_f = self._side
        with torch.cuda.stream(main):
            self.prepare(mbs)  # any cu_seqlens upload is ordered before `start`
        start = torch.cuda.Event()
        start.record(main)
        B.gkv_cache_zero(self.dims, self.gk, self.gv, main)
        # suffix forwards in order on the side stream, one event each
        s_f.wait_event(start)
        fwd_done = []
        for a, b in mbs:
            self._suffix_fwd(a, b, self.ws_fwd, s_f)
            e = torch.cuda.Event()
            e.record(s_f)
            fwd_done.append(e)
        # backwards in microbatch order on the caller's stream
        for (a, b), e in zip(mbs, fwd_done):
            main.wait_event(e)
            self._suffix_bwd(a, b, main)
        # Phase A, then Phase C (only Phase C reads Phase A's outputs)
        o = self.out
        B.prefix_fwd(self.dims, self.q_p, self.k_p, self.v_p, o["o_p"], o["lse_p"], main)
        self._prefix_bwd(use_gy, main)

    def run_dense(self, use_dop: bool = True, stream=None) -> None:
        """Dense recompute baseline; results land in ``self.dense_out``."""
        o = self.dense_out
        shp = self.shape
        if not getattr(self, "_cu_checked", False):
            B.check_cu_seqlens(self.cu_host, shp.n, max(self.lens), shp.total_suffix)
            self._cu_checked = True
        B.dense_recompute_baseline(
            self.dims, self.q_p, self.k_p, self.v_p, self.do_p if use_dop else None, self.q_s,
            self.k_s, self.v_s, self.do_s, self.cu, shp.n, max(self.lens), shp.total_suffix,
            o["o_p"], o["lse_p"], o["o_s"], o["lse_s"], o["dq_s"], o["dk_s"], o["dv_s"],
            o["dq_p"], o["dk_p"], o["dv_p"], self.ws, stream)

    # ------------------------------------------------------------------
    def prepare_dense_packed(self) -> None:
        """Materialize every trajectory [P||S(i)] (Q, K, V and dO = [dO_P(i);
        dO_S(i)]) as one packed varlen batch of N sequences, as a dense
        trainer that packs the whole wave into one microbatch holds it.
        Built once, outside any timed region."""
        if getattr(self, "_dp", None) is not None:
            return
        if self.do_p is None:
            raise ValueError("the dense baseline needs the group built with dense=True")
        shp = self.shape
        hq, hkv, d, P = shp.num_q_heads, shp.num_kv_heads, shp.head_dim, shp.prefix_len
        seq = [P + L for L in self.lens]
        cu = [0] + list(np.cumsum(seq))
        T = int(cu[-1])

        def cat(pre, suf):
            return torch.cat([t for i in range(shp.n) for t in (pre(i), suf[self.cu_host[i]:self.cu_host[i + 1]])])

        dims = B.make_dims(hq, hkv, d, 0, shp.dtype, self.dims.softmax_scale,
                           bool(self.dims.flags & B.SPR_DETERMINISTIC), bool(self.dims.flags & B.SPR_ATOMIC_DQ))
        B.check_cu_seqlens(cu, shp.n, max(seq), T)
        e = lambda h, dt=None: torch.empty(T, h, d, device=self.device, dtype=dt or self.dtype)
        none_kv = torch.empty(0, hkv, d, device=self.device, dtype=self.dtype)
        none_c = torch.empty(0, hkv, d, device=self.device, dtype=torch.float32)
        dp = {"dims": dims, "cu_host": cu, "max_len": max(seq), "T": T,
              "cu": torch.tensor(cu, dtype=torch.int32, device=self.device),
              "q": cat(lambda i: self.q_p, self.q_s), "k": cat(lambda i: self.k_p, self.k_s),
              "v": cat(lambda i: self.v_p, self.v_s), "do": cat(lambda i: self.do_p[i], self.do_s),
              "o": e(hq), "lse": torch.empty(T, hq, device=self.device, dtype=torch.float32),
              "dq": e(hq), "dk": e(hkv), "dv": e(hkv), "none_kv": none_kv, "none_c": none_c}
        need = max(B.workspace_size(B.OP_SUFFIX_FWD, dims, shp.n, dp["max_len"], T),
                   B.workspace_size(B.OP_SUFFIX_BWD, dims, shp.n, dp["max_len"], T), 256)
        dp["ws"] = torch.empty(need, device=self.device, dtype=torch.uint8)
        self._dp = dp

    def release_dense_packed(self) -> None:
        self._dp = None

    def run_dense_packed(self, stream=None) -> None:
        """The dense baseline under the packed batching policy: the N
        materialized trajectories as one varlen microbatch, one forward and
        one backward call of causal attention over each whole sequence
        (the library's suffix calls with no shared prefix).  The
        prefix gradients stay per copy, as a dense trainer has them;
        ``fetch_dense_packed`` sums them for comparison."""
        self.prepare_dense_packed()
        t = self._dp
        dims, n, mx, T = t["dims"], self.shape.n, t["max_len"], t["T"]
        B.suffix_attn_fwd(dims, t["none_kv"], t["none_kv"], t["q"], t["k"], t["v"], t["cu"], n, mx, T,
                          t["o"], t["lse"], t["ws"], stream)
        B.suffix_attn_bwd_accum(dims, t["none_kv"], t["none_kv"], t["q"], t["k"], t["v"], t["o"], t["lse"],
                                t["do"], t["cu"], n, mx, T, t["dq"], t["dk"], t["dv"], t["none_c"],
                                t["none_c"], t["ws"], stream)

    def fetch_dense_packed(self) -> Dict[str, np.ndarray]:
        """The packed dense outputs in the layout of ``fetch``: the first
        copy's prefix outputs, the prefix gradients summed over the copies
        (in float64), the suffix rows as packed suffixes."""
        t, P = self._dp, self.shape.prefix_len
        f64 = lambda x: x.float().cpu().numpy().astype(np.float64)
        cu = t["cu_host"]
        res = {"o_p": f64(t["o"][:P]), "lse_p": f64(t["lse"][:P])}
        for k in ("dq", "dk", "dv"):
            res[k + "_p"] = sum(f64(t[k][cu[i]:cu[i] + P]) for i in range(self.shape.n))
        for k in ("o", "lse", "dq", "dk", "dv"):
            res[k + "_s"] = np.concatenate([f64(t[k][cu[i] + P:cu[i + 1]]) for i in range(self.shape.n)])
        return res

    # ------------------------------------------------------------------
    def fetch(self, which: str = "schedule") -> Dict[str, np.ndarray]:
        """Outputs as float64 numpy arrays (LSE as [T, Hq])."""
        src = self.out if which == "schedule" else self.dense_out
        res = {k: v.float().cpu().numpy().astype(np.float64) for k, v in src.items()}
        if which == "schedule":
            res["g_k"] = self.gk.cpu().numpy().astype(np.float64)
            res["g_v"] = self.gv.cpu().numpy().astype(np.float64)
        return res
