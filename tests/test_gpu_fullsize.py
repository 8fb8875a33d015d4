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
  sides of 64-key and 192-key tile edges, the middle, the last, random) with the cache
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

from sampled_checks import identity_errors, sampled_errors
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
def test_full_length_sampled_rows_keys_and_identities(gpu, name, shape, ragged):
    import torch
    from paper_2606_01143_amd.group import DeviceGroup
    _announce(name)
    inp = make_group(shape, seed=1, ragged=ragged)
    grp = DeviceGroup(inp, dense=False)
    grp.run_schedule()
    torch.cuda.synchronize()
    got = grp.fetch("schedule")
    del grp
    rng = np.random.default_rng(0)
    errs = sampled_errors(inp, got, rng)
    bad = {k: v for k, v in errs.items() if not v <= TOL}
    assert not bad, (bad, errs)
    # ---- identities over every key
    dk_res, dv_res = identity_errors(inp, got)
    assert dk_res <= 1e-3, dk_res
    assert dv_res <= TOL, dv_res
