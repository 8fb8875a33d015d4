"""The forward's twelve-wave form (the forward of App. A.1; Phase A and
Phase B of Sec. 3.2, and the dense baseline's forward): one workgroup holds
96 rows of the four q heads of one kv head, three waves on every SIMD, all
twelve waves reading each K/V tile.  A bf16 forward launch takes it when
its q heads per kv head are a multiple of four, it needs no key splits,
and it has at least 1024 such workgroups (96-row tiles over all its
sequences, times Hkv * G / 4); the rule is restated below.  That covers
Phase A of long prefixes, one microbatch of long suffixes (the packed
dense baseline's whole trajectories among them) and the dense baseline's
per-trajectory forward over a long prefix.

Checked element by element against the oracle: the prefix forward alone on
sampled rows of every q head (the first rows, both sides of the 64-key and
96-row tile edges, the middle, the first row of the last partial row tile,
the last rows, random rows) at prefix lengths that are multiples of
neither tile, d = 128 and 64, four and eight q heads per kv head (eight:
two workgroups per row tile); then whole schedules whose suffix forward
takes the twelve-wave form (with and without a prefix; d = 128 and 64;
four and eight q heads per kv head), and a dense baseline whose
per-trajectory forward takes it, on sampled rows and keys (O, LSE, dQ, dK,
dV and the cache), as the full-length tests check them."""
import numpy as np
import pytest

from oracle.attention import causal_forward_rows
from oracle.compare import max_abs_rel
from sampled_checks import sampled_errors
from synthetic import GroupShape, make_group

TOL = 2e-2


def _wide(hq, hkv, tiles96):
    """tiles96: 96-row tiles of the launch over all its sequences"""
    g = hq // hkv
    return g % 4 == 0 and tiles96 * hkv * (g // 4) >= 1024


def _t96(n):
    return -(-n // 96)


def _suffix_splits(hq, n_mb, max_len, P):
    """the suffix forward's key splits (bf16): enough workgroups of 128
    rows of one q head for two per CU, each split keeping four 64-key
    prefix tiles"""
    nrb = -(-max_len // 128) * hq * n_mb
    ns = -(-512 // nrb)
    return max(1, min(ns, max(1, P // 256), 16))


PREFIX_CASES = [
    ("hq32_hkv8_d128_p12345", GroupShape(32, 8, 128, 12345, (1,), "bf16")),
    ("hq32_hkv4_d128_p12300", GroupShape(32, 4, 128, 12300, (1,), "bf16")),
    ("hq32_hkv8_d64_p12289", GroupShape(32, 8, 64, 12289, (1,), "bf16")),
]
# one microbatch of every suffix: its suffix forward runs unsplit in the
# twelve-wave form (Phase A and the backward take their usual forms)
SUFFIX_CASES = [
    ("p0_two_sequences_6200", GroupShape(32, 8, 128, 0, (6200, 6131), "bf16")),
    ("p1000_three_ragged_suffixes", GroupShape(32, 8, 128, 1000, (6000, 4999, 5537), "bf16")),
    ("p0_g8_d64_two_sequences", GroupShape(32, 4, 64, 0, (6200, 6100), "bf16")),
]
# the dense baseline: each trajectory's forward over P + S rows
DENSE_CASE = ("dense_p12300_n2", GroupShape(32, 8, 128, 12300, (64, 37), "bf16"))


def _rows(P, rng):
    last_tile = 96 * ((P - 1) // 96)
    fixed = [0, 1, 31, 32, 63, 64, 95, 96, 127, 128, 191, 192, 287, 288, P // 2, P // 2 + 1,
             last_tile - 1, last_tile, P - 65, P - 64, P - 2, P - 1]
    extra = rng.integers(0, P, size=6).tolist()
    return sorted({r for r in fixed + extra if 0 <= r < P})


def test_rule_picks_the_twelve_wave_form_at_these_shapes():
    for _, shp in PREFIX_CASES:
        assert _wide(shp.num_q_heads, shp.num_kv_heads, _t96(shp.prefix_len))
    for _, shp in SUFFIX_CASES:
        n, ml = len(shp.suffix_lens), max(shp.suffix_lens)
        assert _suffix_splits(shp.num_q_heads, n, ml, shp.prefix_len) == 1
        assert _wide(shp.num_q_heads, shp.num_kv_heads, n * _t96(ml))
        assert not _wide(shp.num_q_heads, shp.num_kv_heads, _t96(shp.prefix_len))  # Phase A: four waves
    _, shp = DENSE_CASE
    assert _wide(32, 8, _t96(shp.prefix_len) + _t96(max(shp.suffix_lens)))
    # the long-context group's Phase A takes it, its suffix forwards (split)
    # and a P = 4096 group's Phase A do not, nor a single kv group
    assert _wide(32, 8, _t96(28672)) and _wide(32, 8, _t96(16384))
    assert _suffix_splits(32, 1, 128, 28672) > 1
    assert not _wide(32, 8, _t96(8192)) and not _wide(32, 8, _t96(4096))
    assert not _wide(4, 1, _t96(28672)) and not _wide(32, 32, _t96(28672))


@pytest.mark.gpu
@pytest.mark.parametrize("name,shape", PREFIX_CASES, ids=[c[0] for c in PREFIX_CASES])
def test_twelve_wave_prefix_forward_matches_oracle(gpu, name, shape):
    import torch
    from paper_2606_01143_amd import binding as B
    print(f"\n[gpu fwd wide] {name}", flush=True)
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


@pytest.mark.gpu
@pytest.mark.parametrize("name,shape", SUFFIX_CASES, ids=[c[0] for c in SUFFIX_CASES])
def test_schedule_with_twelve_wave_suffix_forward_matches_oracle(gpu, name, shape):
    import torch
    from paper_2606_01143_amd.group import DeviceGroup
    print(f"\n[gpu fwd wide] {name}", flush=True)
    inp = make_group(shape, seed=4)
    grp = DeviceGroup(inp, dense=False)
    grp.run_schedule(microbatches=[(0, len(shape.suffix_lens))])
    torch.cuda.synchronize()
    got = grp.fetch("schedule")
    del grp
    errs = sampled_errors(inp, got, np.random.default_rng(0), cache=shape.prefix_len > 0)
    bad = {k: v for k, v in errs.items() if not v <= TOL}
    assert not bad, (name, bad, errs)


@pytest.mark.gpu
def test_dense_baseline_with_twelve_wave_forward_matches_oracle(gpu):
    import torch
    from paper_2606_01143_amd.group import DeviceGroup
    name, shape = DENSE_CASE
    print(f"\n[gpu fwd wide] {name}", flush=True)
    inp = make_group(shape, seed=5)
    grp = DeviceGroup(inp, dense=True)
    grp.run_dense()
    torch.cuda.synchronize()
    got = grp.fetch("dense")
    del grp
    errs = sampled_errors(inp, got, np.random.default_rng(0), cache=False)
    bad = {k: v for k, v in errs.items() if not v <= TOL}
    assert not bad, (name, bad, errs)
