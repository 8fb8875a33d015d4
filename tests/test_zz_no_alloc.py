"""The allocation-free suffix forward (the library's static device scratch
as workspace) against the workspace call: bitwise equal outputs, over two
calls in a row whose second is smaller, and both within the bf16 gate of
the fp64 oracle.  Both cases need the scratch: the prefixes are long enough
that the forward splits its key range into fp32 partials."""
import sys

import numpy as np
import pytest

from oracle import max_abs_rel, three_phase_reference
from synthetic import GroupShape, make_group

pytestmark = pytest.mark.gpu

CASES = [("first", GroupShape(8, 2, 128, 4096, (100, 60), "bf16"), 11),
         ("second_smaller", GroupShape(4, 1, 128, 2048, (40,), "bf16"), 12)]


def test_noalloc_suffix_forward_equals_workspace_call(gpu):
    import torch
    from paper_2606_01143_amd import binding as B
    from paper_2606_01143_amd.group import DeviceGroup
    for name, shape, seed in CASES:
        sys.stderr.write(f"\n[gpu no-alloc] {name} {shape}\n")
        sys.stderr.flush()
        inp = make_group(shape, seed=seed)
        grp = DeviceGroup(inp, dense=False)
        n, lens, T = shape.n, list(shape.suffix_lens), shape.total_suffix
        need = B.workspace_size(B.OP_SUFFIX_FWD, grp.dims, n, max(lens), T)
        assert 0 < need <= B.STATIC_SCRATCH_BYTES
        cu = grp._mb_cu(0, n)
        o_ws, lse_ws = torch.empty_like(grp.out["o_s"]), torch.empty_like(grp.out["lse_s"])
        o_na, lse_na = torch.full_like(o_ws, float("nan")), torch.full_like(lse_ws, float("nan"))
        B.suffix_attn_fwd(grp.dims, grp.k_p, grp.v_p, grp.q_s, grp.k_s, grp.v_s, cu, n, max(lens), T,
                          o_ws, lse_ws, grp.ws_fwd)
        B.suffix_attn_fwd_noalloc(grp.dims, grp.k_p, grp.v_p, grp.q_s, grp.k_s, grp.v_s, cu, n, max(lens),
                                  T, o_na, lse_na, cu_host=grp.cu_host)
        torch.cuda.synchronize()
        assert torch.equal(o_na, o_ws) and torch.equal(lse_na, lse_ws), name
        ref = three_phase_reference(inp)
        got_o = o_na.float().cpu().numpy().astype(np.float64)
        got_l = lse_na.cpu().numpy().astype(np.float64)
        assert max_abs_rel(got_o, ref["o_s"]) <= 2e-2, name
        assert max_abs_rel(got_l, ref["lse_s"].T) <= 2e-2, name
        del grp
