"""Backward launches whose key-outer work fills the GPU several times over
(bf16, default mode: at least 32768 (32-row tile, q head) steps of 192-key
tiles over all kv heads) run the key-outer role alone, six wave pairs (192
keys) per workgroup, then the query-outer role in a launch of its own:
Phase C of a long prefix, the dense baseline's per-trajectory backward of
long sequences, and the suffix backward (the packed dense baseline's whole
trajectories; Phase B when its prefix key tiles also fill their rounds of
256 workgroups to 85%).  Checked at full length on one or two kv heads
against the oracle's sampled rows and keys (each from its own sequence;
both sampled references are pinned to the whole oracle on small groups) and
the identities that hold at any size, with row shares (3 to 6), head_dim
64, and prefixes that are not a multiple of 192 keys (a partial last tile
whose last pairs have no key); the Phase C halves bitwise equal to the
whole call; reruns bitwise equal."""
import sys

import numpy as np
import pytest

from sampled_checks import identity_errors, sampled_errors
from synthetic import GroupShape, make_group

pytestmark = pytest.mark.gpu

TOL = 2e-2

CASES = [
    # one kv head of four q heads, 6 row shares in Phase C
    ("hkv1_gqa4_p16384", GroupShape(4, 1, 128, 16384, (100, 37), "bf16")),
    # d = 64, no GQA, 16400 = 85 * 192 + 80: the last tile's pairs 3-5 have no key
    ("hkv2_d64_p16400", GroupShape(2, 2, 64, 16400, (33,), "bf16")),
    # 16500 = 85 * 192 + 180: the last pair of the last tile is partial; ragged suffixes of 1 to 200
    ("hkv1_gqa2_p16500", GroupShape(2, 1, 128, 16500, (64, 200, 1), "bf16")),
]


def _announce(msg):
    sys.stderr.write(f"\n[gpu-case] {msg}\n")
    sys.stderr.flush()


def _assert_sampled(inp, got, what, cache):
    errs = sampled_errors(inp, got, np.random.default_rng(5), cache=cache)
    bad = {k: v for k, v in errs.items() if not v <= TOL}
    assert not bad, f"{what}: {bad} (all: {errs})"
    dk_res, dv_res = identity_errors(inp, got)
    assert dk_res <= 1e-3 and dv_res <= TOL, (what, dk_res, dv_res)


@pytest.mark.parametrize("name,shape", CASES, ids=[c[0] for c in CASES])
def test_long_prefix_phase_c_matches_oracle(gpu, name, shape):
    import torch
    from paper_2606_01143_amd import binding as B
    from paper_2606_01143_amd.group import DeviceGroup
    _announce(f"long-prefix Phase C {name} {shape}")
    inp = make_group(shape, seed=23)
    grp = DeviceGroup(inp, dense=False)
    B.profile_reset()
    B.profile_enable(True)
    try:
        grp.run_schedule(overlap=False)
        torch.cuda.synchronize()
        _, n_bwd = B.profile_query("bwd_bf16")
    finally:
        B.profile_enable(False)
    # N suffix backwards, then Phase C as two launches
    assert n_bwd == shape.n + 2, n_bwd
    _assert_sampled(inp, grp.fetch("schedule"), f"schedule {name}", cache=True)


@pytest.mark.parametrize("name,shape", CASES[:2], ids=[c[0] for c in CASES[:2]])
def test_long_prefix_halves_and_reruns_bitwise(gpu, name, shape):
    import torch
    from paper_2606_01143_amd import binding as B
    from paper_2606_01143_amd.group import DeviceGroup
    _announce(f"long-prefix Phase C halves {name}")
    inp = make_group(shape, seed=29)
    grp = DeviceGroup(inp, dense=False)
    grp.run_schedule(overlap=False)
    torch.cuda.synchronize()
    o = grp.out
    whole = {k: o[k].clone() for k in ("dq_p", "dk_p", "dv_p")}
    # a rerun of the whole call
    B.prefix_bwd(grp.dims, grp.q_p, grp.k_p, grp.v_p, o["o_p"], o["lse_p"], grp.g_y, grp.gk, grp.gv,
                 o["dq_p"], o["dk_p"], o["dv_p"], grp.ws)
    torch.cuda.synchronize()
    for k in whole:
        assert torch.equal(whole[k], o[k]), ("rerun", k)
    dq, dk, dv = (torch.empty_like(whole[k]) for k in ("dq_p", "dk_p", "dv_p"))
    B.prefix_bwd_dq(grp.dims, grp.q_p, grp.k_p, grp.v_p, o["o_p"], o["lse_p"], grp.g_y, dq, grp.ws)
    B.prefix_bwd_dkv(grp.dims, grp.q_p, grp.k_p, grp.v_p, o["o_p"], o["lse_p"], grp.g_y, grp.gk, grp.gv,
                     dk, dv, grp.ws)
    torch.cuda.synchronize()
    assert torch.equal(whole["dq_p"], dq) and torch.equal(whole["dk_p"], dk) and torch.equal(whole["dv_p"], dv)


@pytest.mark.parametrize("name,shape", CASES[:2], ids=[c[0] for c in CASES[:2]])
def test_long_sequence_dense_baseline_matches_oracle(gpu, name, shape):
    """The dense baseline's per-trajectory backward of sequences this long
    takes the same two launches; its outputs against the sampled oracle."""
    import torch
    from paper_2606_01143_amd import binding as B
    from paper_2606_01143_amd.group import DeviceGroup
    _announce(f"long-sequence dense {name} {shape}")
    inp = make_group(shape, seed=31)
    grp = DeviceGroup(inp, dense=True)
    B.profile_reset()
    B.profile_enable(True)
    try:
        grp.run_dense()
        torch.cuda.synchronize()
        _, n_bwd = B.profile_query("bwd_bf16")
    finally:
        B.profile_enable(False)
    assert n_bwd == 2 * shape.n, n_bwd
    _assert_sampled(inp, grp.fetch("dense"), f"dense {name}", cache=False)


@pytest.mark.parametrize("name,shape", CASES[:2], ids=[c[0] for c in CASES[:2]])
def test_long_sequences_packed_dense_baseline_matches_oracle(gpu, name, shape):
    """The packed dense baseline's whole trajectories (one varlen microbatch,
    no shared prefix) are this long: the suffix backward takes the same two
    launches; its outputs against the sampled oracle."""
    import torch
    from paper_2606_01143_amd import binding as B
    from paper_2606_01143_amd.group import DeviceGroup
    _announce(f"long-sequence packed dense {name} {shape}")
    inp = make_group(shape, seed=37)
    grp = DeviceGroup(inp, dense=True)
    grp.prepare_dense_packed()
    B.profile_reset()
    B.profile_enable(True)
    try:
        grp.run_dense_packed()
        torch.cuda.synchronize()
        _, n_bwd = B.profile_query("bwd_bf16")
    finally:
        B.profile_enable(False)
    assert n_bwd == 2, n_bwd
    _assert_sampled(inp, grp.fetch_dense_packed(), f"packed dense {name}", cache=False)


LONG_SUFFIX = [
    # two kv heads, 21000 keys: 220 prefix key tiles of 192, 86% of one round
    # of 256 workgroups.  The 3000-token suffix's Phase B takes the two
    # launches, the 100-token one the shared launch; Phase C two launches.
    ("hkv2_p21000_s3000", GroupShape(4, 2, 128, 21000, (3000, 100), "bf16"), 5),
    # d = 64, no GQA, 21100 = 109 * 192 + 172: a partial last prefix tile
    ("hkv2_d64_p21100_s5000", GroupShape(2, 2, 64, 21100, (5000,), "bf16"), 4),
]
@pytest.mark.parametrize("name,shape,launches", LONG_SUFFIX, ids=[c[0] for c in LONG_SUFFIX])
def test_long_suffix_phase_b_matches_oracle(gpu, name, shape, launches):
    import torch
    from paper_2606_01143_amd import binding as B
    from paper_2606_01143_amd.group import DeviceGroup
    _announce(f"long-suffix Phase B {name} {shape}")
    inp = make_group(shape, seed=41)
    grp = DeviceGroup(inp, dense=False)
    B.profile_reset()
    B.profile_enable(True)
    try:
        grp.run_schedule(overlap=False)
        torch.cuda.synchronize()
        _, n_bwd = B.profile_query("bwd_bf16")
    finally:
        B.profile_enable(False)
    assert n_bwd == launches, n_bwd
    _assert_sampled(inp, grp.fetch("schedule"), f"schedule {name}", cache=True)


def test_long_and_short_suffix_in_one_microbatch_matches_oracle(gpu):
    """Both suffixes of the first long-suffix group as one microbatch: the
    key-outer-only launch also sweeps the short suffix's keys and rows."""
    import torch
    from paper_2606_01143_amd import binding as B
    from paper_2606_01143_amd.group import DeviceGroup
    name, shape, _ = LONG_SUFFIX[0]
    _announce(f"long and short suffix packed {name} {shape}")
    inp = make_group(shape, seed=43)
    mb = [(0, shape.n)]
    grp = DeviceGroup(inp, dense=False, microbatch_splits=[mb])
    B.profile_reset()
    B.profile_enable(True)
    try:
        grp.run_schedule(microbatches=mb, overlap=False)
        torch.cuda.synchronize()
        _, n_bwd = B.profile_query("bwd_bf16")
    finally:
        B.profile_enable(False)
    assert n_bwd == 4, n_bwd  # Phase B and Phase C, two launches each
    _assert_sampled(inp, grp.fetch("schedule"), f"schedule packed {name}", cache=True)
