"""Full-length groups of the sweep and the long-context shape on one kv
group (4 q heads), where the full oracle is too slow: sampled rows against
the oracle's per-row definition (O, LSE, dQ of prefix and suffix rows),
and every key's dK/dV through identities that hold at any size:
  sum over all keys of dK = 0 (softmax-backward rows sum to zero), and
  sum over all keys of dV = sum over all rows and group heads of dO, with
  G_Y for the prefix rows (probability rows sum to one)."""
import numpy as np
import pytest

from oracle.attention import sampled_rows_reference
from synthetic import GroupShape, make_group

TOL = 2e-2


def _announce(what):
    print(f"\n[gpu fullsize] {what}", flush=True)


CASES = [
    ("qwen3_8b_p16384_n16_kvgroup", GroupShape(4, 1, 128, 16384, (1024,) * 16, "bf16"), None),
    ("llama3_8b_p28672_n8_s128_kvgroup", GroupShape(4, 1, 128, 28672, (128,) * 8, "bf16"), None),
    ("qwen3_moe_p8192_n16_ragged_kvgroup", GroupShape(8, 1, 128, 8192, (0,) * 16, "bf16"), (128, 2048)),
    # the longest prefix tested: 128k tokens, two ragged suffixes
    ("longest_prefix_p131072_n2_kvgroup", GroupShape(4, 1, 128, 131072, (1000, 37), "bf16"), None),
]


@pytest.mark.gpu
@pytest.mark.parametrize("name,shape,ragged", CASES, ids=[c[0] for c in CASES])
def test_full_length_sampled_rows_and_identities(gpu, name, shape, ragged):
    import torch
    from paper_2606_01143_amd.group import DeviceGroup
    _announce(name)
    inp = make_group(shape, seed=1, ragged=ragged)
    shp = inp["shape"]
    grp = DeviceGroup(inp, dense=False)
    grp.run_schedule()
    torch.cuda.synchronize()
    got = grp.fetch("schedule")
    P, n, lens = shp.prefix_len, shp.n, [int(x) for x in inp["suffix_lens"]]
    rng = np.random.default_rng(0)
    prefix_rows = sorted({0, 1, 63, 64, P // 2, P - 2, P - 1, *rng.integers(0, P, 5).tolist()})
    suffix_rows = [(0, 0), (0, lens[0] - 1), (n - 1, lens[-1] - 1), (n // 2, lens[n // 2] // 2)]
    ref = sampled_rows_reference(inp, prefix_rows, suffix_rows)
    cu = inp["cu_seqlens"]
    errs = {}
    for key, rows, gk in (("prefix", prefix_rows, "_p"), ("suffix", suffix_rows, "_s")):
        for f in ("o", "dq", "lse"):
            g, r = [], []
            for row in rows:
                idx = row if key == "prefix" else int(cu[row[0]]) + row[1]
                g.append(got[f + gk][idx])
                r.append(ref[key][row][f])
            g, r = np.stack(g), np.stack(r)
            errs[f"{f}{gk}"] = float(np.max(np.abs(g - r)) / max(np.max(np.abs(r)), 1e-30))
    bad = {k: v for k, v in errs.items() if not v <= TOL}
    assert not bad, (bad, errs)
    # identities over every key
    dk = np.concatenate([got["dk_p"], got["dk_s"]]).sum(axis=0)
    dk_scale = np.abs(np.concatenate([got["dk_p"], got["dk_s"]])).sum(axis=0).max()
    assert np.abs(dk).max() <= 1e-3 * dk_scale, np.abs(dk).max() / dk_scale
    dv = np.concatenate([got["dv_p"], got["dv_s"]]).sum(axis=0)
    g_y = np.asarray(inp["do_p"], np.float64).sum(axis=0)
    do_sum = g_y.sum(axis=0) + np.asarray(inp["do_s"], np.float64).sum(axis=0)  # [Hq, d]
    G = shp.num_q_heads // shp.num_kv_heads
    want = do_sum.reshape(shp.num_kv_heads, G, -1).sum(axis=1)
    assert np.abs(dv - want).max() <= TOL * np.abs(want).max(), np.abs(dv - want).max() / np.abs(want).max()
