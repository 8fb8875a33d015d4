"""The prefix forward's twelve-wave form (Phase A, Sec. 3.2; the forward of
App. A.1 on the prefix rows): one workgroup holds 96 prefix rows of four q
heads of one kv head, three waves on every SIMD, all twelve waves reading
each K/V tile.  ``spr_prefix_fwd`` takes it for bf16 groups whose q heads
per kv head are a multiple of four, once there are at least 1024 such
workgroups (ceil(P / 96) * Hkv * G / 4); the rule is restated below.

Checked element by element against the oracle (``causal_forward_rows``,
each row against its own causal keys) on sampled rows of every q head: the
first rows, both sides of the 64-key and 96-row tile edges, the middle,
the first row of the last (partial) row tile, the last rows, and random
rows.  Prefix lengths are multiples of neither tile; d = 128 and 64; four
and eight q heads per kv head (eight: two workgroups per row tile)."""
import numpy as np
import pytest

from oracle.attention import causal_forward_rows
from oracle.compare import max_abs_rel
from synthetic import GroupShape, make_group

TOL = 2e-2


def _wide(hq, hkv, P):
    g = hq // hkv
    return g % 4 == 0 and -(-P // 96) * hkv * (g // 4) >= 1024


CASES = [
    ("hq32_hkv8_d128_p12345", GroupShape(32, 8, 128, 12345, (1,), "bf16")),
    ("hq32_hkv4_d128_p12300", GroupShape(32, 4, 128, 12300, (1,), "bf16")),
    ("hq32_hkv8_d64_p12289", GroupShape(32, 8, 64, 12289, (1,), "bf16")),
]


def _rows(P, rng):
    last_tile = 96 * ((P - 1) // 96)
    fixed = [0, 1, 31, 32, 63, 64, 95, 96, 127, 128, 191, 192, 287, 288, P // 2, P // 2 + 1,
             last_tile - 1, last_tile, P - 65, P - 64, P - 2, P - 1]
    extra = rng.integers(0, P, size=6).tolist()
    return sorted({r for r in fixed + extra if 0 <= r < P})


def test_rule_picks_the_twelve_wave_form_at_these_shapes():
    for _, shp in CASES:
        assert _wide(shp.num_q_heads, shp.num_kv_heads, shp.prefix_len)
    # the long-context group takes it, a P = 4096 group and one kv group do not
    assert _wide(32, 8, 28672) and _wide(32, 8, 16384)
    assert not _wide(32, 8, 8192) and not _wide(32, 8, 4096)
    assert not _wide(4, 1, 28672) and not _wide(32, 32, 28672)


@pytest.mark.gpu
@pytest.mark.parametrize("name,shape", CASES, ids=[c[0] for c in CASES])
def test_twelve_wave_prefix_forward_matches_oracle(gpu, name, shape):
    import torch
    from paper_2606_01143_amd import binding as B
    print(f"\n[gpu prefix fwd wide] {name}", flush=True)
    inp = make_group(shape, seed=3)
    P, hq, hkv, d = shape.prefix_len, shape.num_q_heads, shape.num_kv_heads, shape.head_dim
    dev = torch.device("cuda:0")
    up = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(device=dev, dtype=torch.bfloat16)
    q, k, v = up(inp["q_p"]), up(inp["k_p"]), up(inp["v_p"])
    o = torch.empty(P, hq, d, device=dev, dtype=torch.bfloat16)
    lse = torch.empty(P, hq, device=dev, dtype=torch.float32)
    dims = B.make_dims(hq, hkv, d, P, "bf16")
    B.prefix_fwd(dims, q, k, v, o, lse)
    torch.cuda.synchronize()
    o_got = o.float().cpu().numpy().astype(np.float64)
    lse_got = lse.cpu().numpy().astype(np.float64)
    rows = _rows(P, np.random.default_rng(0))
    scale = 1.0 / np.sqrt(d)
    o_ref = np.zeros((len(rows), hq, d))
    lse_ref = np.zeros((len(rows), hq))
    for i, r in enumerate(rows):
        orow, lrow = causal_forward_rows(inp["q_p"][r:r + 1], inp["k_p"][:r + 1], inp["v_p"][:r + 1], scale,
                                         first_query_pos=r)
        o_ref[i], lse_ref[i] = orow[0], lrow[:, 0]
    e_o = max_abs_rel(o_got[rows], o_ref)
    e_lse = max_abs_rel(lse_got[rows], lse_ref)
    assert e_o <= TOL and e_lse <= TOL, (name, e_o, e_lse)
