"""Batch-plus-padding suffix layout (paper Sec. 2.1, Sec. 4.2): the padded
calls must give bitwise the packed calls' results on the valid rows, zero on
the padding rows, and the same gK/gV cache; and their valid rows and cache
must match the fp64 oracle's three-phase reference on the same inputs (the
max-abs-relative gate: 1e-4 fp32, 2e-2 bf16).  The padding rows of every
input hold NaN, so any read of them would show."""
import numpy as np
import pytest

from oracle import max_abs_rel, three_phase_reference
from synthetic import GroupShape, make_group

TOL = {"f32": 1e-4, "bf16": 2e-2}


def _against_oracle(inp, rows, gk, gv, what, microbatches=None):
    """rows: packed [T, ...] valid-row outputs o, lse, dq, dk, dv (torch);
    gk, gv: the cache after Phase B.  Compared with the oracle's Phase B
    outputs and cache."""
    ref = three_phase_reference(inp, microbatches=microbatches)
    f64 = lambda x: x.float().cpu().numpy().astype(np.float64)
    errs = {k: max_abs_rel(f64(rows[k]), ref[k + "_s"].T if k == "lse" else ref[k + "_s"])
            for k in ("o", "lse", "dq", "dk", "dv")}
    errs["g_k"] = max_abs_rel(f64(gk), ref["g_k"])
    errs["g_v"] = max_abs_rel(f64(gv), ref["g_v"])
    tol = TOL[inp["shape"].dtype]
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, (what, bad, errs)


def _announce(what):
    print(f"\n[gpu padded] {what}", flush=True)


def _run_packed_and_padded(shape, seed, ragged=None, deterministic=True):
    import torch
    from paper_2606_01143_amd import binding as B
    inp = make_group(shape, seed=seed, ragged=ragged)
    shape = inp["shape"]
    dev = torch.device("cuda:0")
    dt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    up = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(device=dev, dtype=dt)
    hq, hkv, d, P = shape.num_q_heads, shape.num_kv_heads, shape.head_dim, shape.prefix_len
    lens = [int(x) for x in inp["suffix_lens"]]
    n, s_max, T = len(lens), max(lens), sum(lens)
    cu_h = [0] + list(np.cumsum(lens))
    dims = B.make_dims(hq, hkv, d, P, shape.dtype, atomic_dq=not deterministic)
    k_p, v_p = up(inp["k_p"]), up(inp["v_p"])
    t = {k: up(inp[k]) for k in ("q_s", "k_s", "v_s", "do_s")}
    cu = torch.tensor(cu_h, dtype=torch.int32, device=dev)
    # packed reference
    o = torch.empty(T, hq, d, dtype=dt, device=dev)
    lse = torch.empty(T, hq, dtype=torch.float32, device=dev)
    dq, dk, dv = (torch.empty(T, h, d, dtype=dt, device=dev) for h in (hq, hkv, hkv))
    gk = torch.zeros(P, hkv, d, dtype=torch.float32, device=dev)
    gv = torch.zeros_like(gk)
    ws = torch.empty(max(B.workspace_size(B.OP_SUFFIX_FWD, dims, n, s_max, T),
                         B.workspace_size(B.OP_SUFFIX_BWD, dims, n, s_max, T), 256), dtype=torch.uint8, device=dev)
    B.suffix_attn_fwd(dims, k_p, v_p, t["q_s"], t["k_s"], t["v_s"], cu, n, s_max, T, o, lse, ws)
    B.suffix_attn_bwd_accum(dims, k_p, v_p, t["q_s"], t["k_s"], t["v_s"], o, lse, t["do_s"], cu, n, s_max, T,
                            dq, dk, dv, gk, gv, ws)
    # padded: NaN everywhere, then the valid rows
    def pad(x, h):
        y = torch.full((n, s_max, h, d), float("nan"), dtype=dt, device=dev)
        for i in range(n):
            y[i, :lens[i]] = x[cu_h[i]:cu_h[i + 1]]
        return y
    pq, pk, pv, pdo = pad(t["q_s"], hq), pad(t["k_s"], hkv), pad(t["v_s"], hkv), pad(t["do_s"], hq)
    lens_d = torch.tensor(lens, dtype=torch.int32, device=dev)
    po = torch.full((n, s_max, hq, d), 7.0, dtype=dt, device=dev)
    plse = torch.full((n, s_max, hq), 7.0, dtype=torch.float32, device=dev)
    pdq, pdk, pdv = (torch.full((n, s_max, h, d), 7.0, dtype=dt, device=dev) for h in (hq, hkv, hkv))
    gk2 = torch.zeros_like(gk)
    gv2 = torch.zeros_like(gk)
    wsp = torch.empty(max(B.workspace_size(B.OP_SUFFIX_FWD_PADDED, dims, n, s_max),
                          B.workspace_size(B.OP_SUFFIX_BWD_PADDED, dims, n, s_max)), dtype=torch.uint8, device=dev)
    B.suffix_attn_fwd_padded(dims, k_p, v_p, pq, pk, pv, lens_d, n, s_max, po, plse, wsp)
    # the backward reads O as the padded forward wrote it (zero padding rows)
    B.suffix_attn_bwd_accum_padded(dims, k_p, v_p, pq, pk, pv, po, plse, pdo, lens_d, n, s_max, pdq, pdk, pdv,
                                   gk2, gv2, wsp)
    torch.cuda.synchronize()
    packed = {"o": o, "lse": lse, "dq": dq, "dk": dk, "dv": dv}
    padded = {"o": po, "lse": plse, "dq": pdq, "dk": pdk, "dv": pdv}
    exact = deterministic or shape.dtype == "f32"  # dQ of the atomic mode agrees to rounding only
    for key in packed:
        for i in range(n):
            got = padded[key][i, :lens[i]]
            want = packed[key][cu_h[i]:cu_h[i + 1]]
            if exact or key != "dq":
                assert torch.equal(got, want), (key, i)
            else:
                assert max_abs_rel(got.float().cpu().numpy(), want.float().cpu().numpy(), floor=1e-3) <= 2e-2
            assert not padded[key][i, lens[i]:].float().abs().sum().item(), (key, i, "padding not zero")
    assert torch.equal(gk, gk2) and torch.equal(gv, gv2)
    # the padded call's own valid rows and cache against the oracle
    valid = {k: torch.cat([padded[k][i, :lens[i]] for i in range(n)]) for k in padded}
    _against_oracle(inp, valid, gk2, gv2, f"padded {shape}")


CASES = [
    ("bf16_gqa4_ragged", GroupShape(8, 2, 128, 300, (70, 129, 33), "bf16")),
    ("bf16_d64", GroupShape(4, 2, 64, 130, (65, 1, 128), "bf16")),
    ("bf16_split", GroupShape(4, 2, 128, 1100, (70, 129, 33), "bf16")),
    ("f32_gqa", GroupShape(4, 2, 128, 75, (33, 70, 5), "f32")),
    ("bf16_n1", GroupShape(4, 1, 128, 257, (100,), "bf16")),
]


@pytest.mark.gpu
@pytest.mark.parametrize("deterministic", [True, False], ids=["deterministic", "atomic_dq"])
@pytest.mark.parametrize("name,shape", CASES, ids=[c[0] for c in CASES])
def test_padded_layout_is_bitwise_the_packed_layout(gpu, name, shape, deterministic):
    _announce(f"{name} {shape} deterministic={deterministic}")
    _run_packed_and_padded(shape, seed=31, deterministic=deterministic)


@pytest.mark.gpu
def test_padded_layout_with_many_suffixes(gpu):
    """1100 suffixes of 1..3 tokens: more than the gather derives offsets
    for by itself, so the separate offsets launch runs."""
    shape = GroupShape(2, 1, 64, 40, (0,) * 1100, "bf16")
    _announce(f"many suffixes {shape}")
    _run_packed_and_padded(shape, seed=41, ragged=(1, 3))


@pytest.mark.gpu
@pytest.mark.parametrize("budget", [10 ** 9, 300])
def test_padded_schedule_equals_packed_schedule(gpu, budget):
    """The whole schedule (streams overlapped) in the padded layout, with
    waves planned under a padded token budget, gives bitwise the packed
    schedule's outputs and cache on the same waves."""
    import torch
    from paper_2606_01143_amd.group import DeviceGroup, plan_suffix_waves
    shape = GroupShape(8, 2, 128, 700, (70, 129, 33, 128, 5), "bf16")
    _announce(f"padded schedule budget {budget} {shape}")
    inp = make_group(shape, seed=37)
    waves = plan_suffix_waves([int(x) for x in inp["suffix_lens"]], budget, "padded")
    packed = DeviceGroup(inp, dense=False, microbatch_splits=[waves])
    padded = DeviceGroup(inp, dense=False, microbatch_splits=[waves], layout="padded")
    packed.run_schedule(waves)
    padded.run_schedule(waves)
    padded.gather_padded_outputs()
    torch.cuda.synchronize()
    for k in packed.out:
        assert torch.equal(packed.out[k], padded.out[k]), k
    assert torch.equal(packed.gk, padded.gk) and torch.equal(packed.gv, padded.gv)
    # the padded schedule's outputs against the oracle's schedule on the same waves
    ref = three_phase_reference(inp, microbatches=[list(range(a, b)) for a, b in waves])
    got = padded.fetch("schedule")
    errs = {k: max_abs_rel(got[k], ref[k].T if k.startswith("lse") else ref[k])
            for k in ("o_p", "lse_p", "o_s", "lse_s", "dq_p", "dk_p", "dv_p", "dq_s", "dk_s", "dv_s",
                      "g_k", "g_v")}
    bad = {k: v for k, v in errs.items() if not v <= 2e-2}
    assert not bad, (bad, errs)
