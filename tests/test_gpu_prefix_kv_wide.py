"""Backward launches over long sequences (bf16, default mode): a Phase C of
a prefix of 16384 keys or more runs the key-outer role alone, six wave
pairs (192 keys) per workgroup, then the query-outer role in a launch of its
own; the dense baseline's per-trajectory backward of sequences that long
does the same, and so does the suffix backward of suffixes that long (the
packed dense baseline's whole trajectories, or a long suffix behind a short
prefix in Phase B).  Checked at full length on one or two kv heads against the
oracle's sampled rows and keys (each from its own sequence; both sampled
references are pinned to the whole oracle on small groups) and the
identities that hold at any size, with row shares (3 to 6), head_dim 64,
and prefixes that are not a multiple of 192 keys (a partial last tile whose
last pairs have no key); the Phase C halves bitwise equal to the whole
call; reruns bitwise equal."""
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
    # a suffix of 16400 = 85 * 192 + 80 tokens behind a prefix of 512, and a
    # short one: Phase B takes the two launches for the first microbatch only
    ("hkv1_gqa4_s16400", GroupShape(4, 1, 128, 512, (16400, 300), "bf16")),
    ("hkv2_d64_s16500", GroupShape(2, 2, 64, 200, (16500,), "bf16")),
]


@pytest.mark.parametrize("name,shape", LONG_SUFFIX, ids=[c[0] for c in LONG_SUFFIX])
def test_long_suffix_phase_b_matches_oracle(gpu, name, shape):
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
    n_long = sum(1 for s in shape.suffix_lens if s >= 16384)
    # one launch per short suffix, two per long one, one for Phase C
    assert n_bwd == shape.n + n_long + 1, n_bwd
    _assert_sampled(inp, grp.fetch("schedule"), f"schedule {name}", cache=True)
