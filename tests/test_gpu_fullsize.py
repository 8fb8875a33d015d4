"""Full-length groups of the sweep and the long-context shape on one kv
group, where the whole fp64 oracle is too slow, checked element by element
on sampled rows and sampled keys, both computed by the oracle from each
row's own sequence:

* rows (``sampled_rows_reference``): O, LSE and dQ of prefix rows (first,
  tile edges, middle, last, random) and suffix rows (first, last and both
  sides of row-tile edges of three suffixes).  Every row's O and dQ sum over
  all its key tiles, so they also cover every key-split range of the split
  suffix forward and backward launches and their combine kernels.
* keys (``sampled_keys_reference``): dK and dV of prefix keys (first, both
  sides of 64-key tile edges, the middle, the last, random) with the cache
  values G_K, G_V, and of suffix keys (first, tile edges, middle, last of
  three suffixes).  Every sampled prefix key is swept by all rows that see
  it, so its dK/dV/G_K/G_V check the cache accumulation over every suffix
  microbatch and the row shares of the key-outer role.

The longest-prefix case samples prefix keys in its last 2048 positions
only (each sampled prefix key costs a forward over the rows that see it).
Identities that hold at any size are checked on every key as well:
sum over all keys of dK = 0, and sum over all keys of dV = sum over all
rows and group heads of dO (G_Y for the prefix rows)."""
import numpy as np
import pytest

from oracle.attention import sampled_keys_reference, sampled_rows_reference
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


def _rel(got, ref):
    g, r = np.stack(got), np.stack(ref)
    return float(np.max(np.abs(g - r)) / max(np.max(np.abs(r)), 1e-30))


def sample_rows(P, lens, rng):
    n = len(lens)
    prefix = sorted({0, 1, 63, 64, 127, 128, 255, 256, P // 2, P - 2, P - 1,
                     *rng.integers(0, P, 5).tolist()})
    suffix = sorted({(i, t) for i in (0, n // 2, n - 1)
                     for t in (0, 31, 32, 127, 128, lens[i] // 2, lens[i] - 1) if t < lens[i]})
    return prefix, suffix


def sample_keys(P, lens, rng):
    n = len(lens)
    if P > 32768:
        lo = P - 2048
        prefix = sorted({lo, lo + 63, lo + 64, P - 1025, P - 1024, P - 65, P - 64, P - 2, P - 1,
                         *rng.integers(lo, P, 3).tolist()})
    else:
        prefix = sorted({0, 1, 63, 64, 127, 128, P // 2 - 1, P // 2, P - 65, P - 64, P - 2, P - 1,
                         *rng.integers(0, P, 4).tolist()})
    suffix = sorted({(i, t) for i in (0, n // 2, n - 1)
                     for t in (0, 1, 63, 64, lens[i] // 2, lens[i] - 1) if t < lens[i]})
    return prefix, suffix


@pytest.mark.gpu
@pytest.mark.parametrize("name,shape,ragged", CASES, ids=[c[0] for c in CASES])
def test_full_length_sampled_rows_keys_and_identities(gpu, name, shape, ragged):
    import torch
    from paper_2606_01143_amd.group import DeviceGroup
    _announce(name)
    inp = make_group(shape, seed=1, ragged=ragged)
    shp = inp["shape"]
    grp = DeviceGroup(inp, dense=False)
    grp.run_schedule()
    torch.cuda.synchronize()
    got = grp.fetch("schedule")
    del grp
    P, n, lens = shp.prefix_len, shp.n, [int(x) for x in inp["suffix_lens"]]
    cu = inp["cu_seqlens"]
    rng = np.random.default_rng(0)
    errs = {}
    # ---- rows
    prefix_rows, suffix_rows = sample_rows(P, lens, rng)
    ref = sampled_rows_reference(inp, prefix_rows, suffix_rows)
    for key, rows, sfx in (("prefix", prefix_rows, "_p"), ("suffix", suffix_rows, "_s")):
        for f in ("o", "dq", "lse"):
            g, r = [], []
            for row in rows:
                idx = row if key == "prefix" else int(cu[row[0]]) + row[1]
                g.append(got[f + sfx][idx])
                r.append(ref[key][row][f])
            errs[f"{f}{sfx}"] = _rel(g, r)
    # ---- keys
    prefix_keys, suffix_keys = sample_keys(P, lens, rng)
    kref = sampled_keys_reference(inp, prefix_keys, suffix_keys)
    for f, gk in (("dk", "dk_p"), ("dv", "dv_p"), ("g_k", "g_k"), ("g_v", "g_v")):
        errs[gk + "@keys"] = _rel([got[gk][j] for j in prefix_keys], [kref["prefix"][j][f] for j in prefix_keys])
    for f in ("dk", "dv"):
        errs[f + "_s@keys"] = _rel([got[f + "_s"][int(cu[i]) + t] for i, t in suffix_keys],
                                   [kref["suffix"][(i, t)][f] for i, t in suffix_keys])
    bad = {k: v for k, v in errs.items() if not v <= TOL}
    assert not bad, (bad, errs)
    # ---- identities over every key
    dk = np.concatenate([got["dk_p"], got["dk_s"]]).sum(axis=0)
    dk_scale = np.abs(np.concatenate([got["dk_p"], got["dk_s"]])).sum(axis=0).max()
    assert np.abs(dk).max() <= 1e-3 * dk_scale, np.abs(dk).max() / dk_scale
    dv = np.concatenate([got["dv_p"], got["dv_s"]]).sum(axis=0)
    g_y = np.asarray(inp["do_p"], np.float64).sum(axis=0)
    do_sum = g_y.sum(axis=0) + np.asarray(inp["do_s"], np.float64).sum(axis=0)  # [Hq, d]
    G = shp.num_q_heads // shp.num_kv_heads
    want = do_sum.reshape(shp.num_kv_heads, G, -1).sum(axis=1)
    assert np.abs(dv - want).max() <= TOL * np.abs(want).max(), np.abs(dv - want).max() / np.abs(want).max()
