"""One GRPO prompt group resident in HBM, run through libspr.

PyTorch only provides device memory and the stream here; every step of the
schedule runs in the HIP library through ``binding``.

``DeviceGroup.run_schedule`` is the paper's three-phase schedule (Sec. 3.2):
zero the gK/gV cache, Phase A ``prefix_fwd`` once, Phase B
``suffix_attn_fwd`` + ``suffix_attn_bwd_accum`` per suffix microbatch (a
microbatch is a contiguous run of the packed suffixes; packed layout of
Sec. 4.2), Phase C ``prefix_bwd`` once.  ``run_dense`` is the comparison:
``dense_recompute_baseline`` over every [P||S(i)].
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch

from . import binding as B

_TORCH_DT = {"bf16": torch.bfloat16, "f32": torch.float32}
OUTPUT_KEYS = ["o_p", "lse_p", "o_s", "lse_s", "dq_p", "dk_p", "dv_p", "dq_s", "dk_s", "dv_s"]


class DeviceGroup:
    """Inputs, outputs, cache and workspace of one prompt group on one GPU.

    ``inp`` is a synthetic group (see ``synthetic.make_group``): float32
    arrays holding values exactly representable in the storage dtype.
    """

    def __init__(self, inp: Dict, device="cuda:0", softmax_scale: float = 0.0,
                 deterministic: bool = False, dense: bool = True,
                 microbatch_splits: Optional[Sequence[Sequence[Tuple[int, int]]]] = None):
        shp = inp["shape"]
        self.shape = shp
        self.device = torch.device(device)
        dt = _TORCH_DT[shp.dtype]
        self.dtype = dt
        hq, hkv, d, p = shp.num_q_heads, shp.num_kv_heads, shp.head_dim, shp.prefix_len
        t = shp.total_suffix
        self.dims = B.make_dims(hq, hkv, d, p, shp.dtype, softmax_scale, deterministic)
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
            self._cu_cache[key] = torch.tensor([x - base for x in self.cu_host[a:b + 1]],
                                               dtype=torch.int32, device=self.device)
        return self._cu_cache[key]

    def prepare(self, microbatches: Sequence[Tuple[int, int]]) -> None:
        """Build the per-microbatch cu_seqlens tensors ahead of a timed run."""
        for a, b in microbatches:
            self._mb_cu(a, b)

    # ------------------------------------------------------------------
    def run_schedule(self, microbatches: Optional[Sequence[Tuple[int, int]]] = None,
                     use_gy: bool = True, stream=None, mark=None) -> None:
        """Three-phase schedule; results land in ``self.out``, ``self.gk``, ``self.gv``.

        ``mark(name)``, if given, is called after each phase's launches are
        issued ("zero", "A", "B_fwd", "B_bwd" per microbatch, "C"), e.g. to
        record events for per-phase times."""
        dims, o = self.dims, self.out
        mark = mark or (lambda name: None)
        mbs = list(microbatches) if microbatches is not None else self.default_microbatches()
        B.gkv_cache_zero(dims, self.gk, self.gv, stream)
        mark("zero")
        # Phase A: prefix forward once
        B.prefix_fwd(dims, self.q_p, self.k_p, self.v_p, o["o_p"], o["lse_p"], stream)
        mark("A")
        # Phase B: suffix microbatches read K_P/V_P and accumulate gK/gV
        for a, b in mbs:
            nmb, mx, tot = self._mb_sizes(a, b)
            r0, r1 = self.cu_host[a], self.cu_host[b]
            cu = self._mb_cu(a, b)
            B.suffix_attn_fwd(dims, self.k_p, self.v_p, self.q_s[r0:r1], self.k_s[r0:r1],
                              self.v_s[r0:r1], cu, nmb, mx, tot, o["o_s"][r0:r1],
                              o["lse_s"][r0:r1], self.ws, stream)
            mark("B_fwd")
            B.suffix_attn_bwd_accum(dims, self.k_p, self.v_p, self.q_s[r0:r1], self.k_s[r0:r1],
                                    self.v_s[r0:r1], o["o_s"][r0:r1], o["lse_s"][r0:r1],
                                    self.do_s[r0:r1], cu, nmb, mx, tot, o["dq_s"][r0:r1],
                                    o["dk_s"][r0:r1], o["dv_s"][r0:r1], self.gk, self.gv,
                                    self.ws, stream)
            mark("B_bwd")
        # Phase C: prefix backward once on the accumulated cache
        B.prefix_bwd(dims, self.q_p, self.k_p, self.v_p, o["o_p"], o["lse_p"],
                     self.g_y if use_gy else None, self.gk, self.gv, o["dq_p"], o["dk_p"],
                     o["dv_p"], self.ws, stream)
        mark("C")

    def run_dense(self, use_dop: bool = True, stream=None) -> None:
        """Dense recompute baseline; results land in ``self.dense_out``."""
        o = self.dense_out
        shp = self.shape
        B.dense_recompute_baseline(
            self.dims, self.q_p, self.k_p, self.v_p, self.do_p if use_dop else None, self.q_s,
            self.k_s, self.v_s, self.do_s, self.cu, shp.n, max(self.lens), shp.total_suffix,
            o["o_p"], o["lse_p"], o["o_s"], o["lse_s"], o["dq_s"], o["dk_s"], o["dv_s"],
            o["dq_p"], o["dk_p"], o["dv_p"], self.ws, stream)

    # ------------------------------------------------------------------
    def fetch(self, which: str = "schedule") -> Dict[str, np.ndarray]:
        """Outputs as float64 numpy arrays (LSE as [T, Hq])."""
        src = self.out if which == "schedule" else self.dense_out
        res = {k: v.float().cpu().numpy().astype(np.float64) for k, v in src.items()}
        if which == "schedule":
            res["g_k"] = self.gk.cpu().numpy().astype(np.float64)
            res["g_v"] = self.gv.cpu().numpy().astype(np.float64)
        return res
