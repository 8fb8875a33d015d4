"""GPU parity of the MoE router aux-loss accounting (paper App. B) against
the fp64 oracle's materialized batch (every prefix copy explicit).

Counts, totals and the invalid-id count are integers: bit-exact.  Mass, f,
P and the loss are fp64 sums of fp32 inputs times integers on both sides
(different order): 1e-12 relative.  The gradient is stored in fp32: 2^-23
relative per element, checked at 1e-6.
"""
import numpy as np
import pytest

from oracle.moe_aux import materialized_reference, reuse_reference, logical_stats
from synthetic.moe import RouterShape, make_router_group, ROUTER_SHAPES

LAM = 0.01


def _announce(what):
    print(f"\n[gpu moe] {what}", flush=True)


class _Dev:
    """Router outputs of one group on the GPU, statistics and workspace."""

    def __init__(self, inp):
        import torch
        from paper_2606_01143_amd import binding as B
        self.B, self.torch = B, torch
        shp = inp["shape"]
        self.E, self.k = shp.num_experts, shp.top_k
        dev = torch.device("cuda:0")
        t = lambda x, dt: torch.from_numpy(np.ascontiguousarray(x)).to(device=dev, dtype=dt)
        self.p_p, self.r_p = t(inp["p_p"], torch.float32), t(inp["r_p"], torch.int32)
        self.p_s, self.r_s = t(inp["p_s"], torch.float32), t(inp["r_s"], torch.int32)
        self.cu = [int(x) for x in inp["cu_seqlens"]]
        self.stats = torch.empty(B.moe_stats_bytes(self.E), dtype=torch.uint8, device=dev)
        n_max = max(shp.prefix_len, int(inp["suffix_lens"].sum()), 1) * (shp.n + 1)
        self.ws = torch.empty(max(B.moe_aux_workspace_size(self.E, n_max), 16), dtype=torch.uint8, device=dev)
        self.f = torch.empty(self.E, dtype=torch.float64, device=dev)
        self.pe = torch.empty(self.E, dtype=torch.float64, device=dev)
        self.loss = torch.empty(1, dtype=torch.float64, device=dev)
        self.n = shp.n

    def schedule(self, per_microbatch=True):
        """Reuse accounting: prefix once with m = N, suffixes with m = 1."""
        B = self.B
        B.moe_stats_zero(self.E, self.stats)
        B.moe_aux_accumulate(self.E, self.k, self.p_p, self.r_p, self.stats, multiplicity=self.n, ws=self.ws)
        spans = [(self.cu[i], self.cu[i + 1]) for i in range(self.n)] if per_microbatch else [(0, self.cu[-1])]
        for a, b in spans:
            B.moe_aux_accumulate(self.E, self.k, self.p_s[a:b], self.r_s[a:b], self.stats, multiplicity=1,
                                 ws=self.ws)
        B.moe_aux_loss(self.E, self.k, LAM, self.stats, self.f, self.pe, self.loss)
        dp_p = self.torch.empty_like(self.p_p)
        dp_s = self.torch.empty_like(self.p_s)
        B.moe_aux_grad(self.E, self.k, LAM, 1.0, self.stats, dp_p, multiplicity=self.n)
        B.moe_aux_grad(self.E, self.k, LAM, 1.0, self.stats, dp_s, multiplicity=1)
        self.torch.cuda.synchronize()
        return self.read(), dp_p.cpu().numpy(), dp_s.cpu().numpy()

    def read(self):
        raw = self.stats.cpu().numpy()
        E = self.E
        return {"C": raw[:8 * E].view(np.int64).copy(), "R": raw[8 * E:16 * E].view(np.float64).copy(),
                "M": int(raw[16 * E:16 * E + 8].view(np.int64)[0]),
                "invalid": int(raw[16 * E + 8:16 * E + 16].view(np.int64)[0]),
                "f": self.f.cpu().numpy(), "P": self.pe.cpu().numpy(), "L": float(self.loss.item())}


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)) if a.size else 0.0


def _check(got, dp_p, dp_s, ref):
    assert np.array_equal(got["C"], ref["C"]), "counts"
    assert got["M"] == ref["M"] and got["invalid"] == 0
    for key in ("R", "f", "P"):
        assert _rel(got[key], ref[key]) <= 1e-12, key
    assert abs(got["L"] - ref["L"]) <= 1e-12 * abs(ref["L"])
    assert _rel(dp_p, ref["dp_p"]) <= 1e-6 and _rel(dp_s, ref["dp_s"]) <= 1e-6


CASES = [
    ("tiny", RouterShape(8, 2, 24, (5, 9, 3)), None),
    ("e4_k1", RouterShape(4, 1, 70, (65, 1)), None),
    ("e60_k4_ragged", RouterShape(60, 4, 130, (0,) * 5), (1, 90)),
    ("e1024_k2", RouterShape(1024, 2, 33, (20, 7)), None),
    ("p0", RouterShape(16, 2, 0, (40, 3)), None),
]


@pytest.mark.gpu
@pytest.mark.parametrize("name,shape,ragged", CASES, ids=[c[0] for c in CASES])
def test_moe_accounting_matches_materialized_copies(gpu, name, shape, ragged):
    _announce(f"{name} {shape}")
    inp = make_router_group(shape, seed=11, ragged=ragged)
    ref = materialized_reference(inp, LAM)
    got, dp_p, dp_s = _Dev(inp).schedule()
    _check(got, dp_p, dp_s, ref)


@pytest.mark.gpu
def test_moe_full_size_qwen3_router_and_reproducibility(gpu):
    """The Qwen3-MoE router group (E = 128, top-8, P = 8192, N = 16 ragged
    suffixes of 128..2048): per-suffix microbatches, then one packed
    microbatch, both bitwise equal to each other in C/M and within 1e-12
    of the materialized batch; a rerun is bitwise identical."""
    shape = ROUTER_SHAPES["qwen3_moe_router_p8192_n16_ragged"]
    _announce(f"qwen3 router {shape}")
    inp = make_router_group(shape, seed=0, ragged=(128, 2048))
    ref = materialized_reference(inp, LAM)
    dev = _Dev(inp)
    got, dp_p, dp_s = dev.schedule()
    _check(got, dp_p, dp_s, ref)
    again, dp_p2, dp_s2 = dev.schedule()
    assert all(np.array_equal(got[k], again[k]) for k in ("C", "R", "f", "P")) and got["L"] == again["L"]
    assert np.array_equal(dp_p, dp_p2) and np.array_equal(dp_s, dp_s2)
    packed, _, _ = dev.schedule(per_microbatch=False)
    assert np.array_equal(packed["C"], got["C"]) and packed["M"] == got["M"]
    assert _rel(packed["R"], got["R"]) <= 1e-13


@pytest.mark.gpu
def test_moe_per_token_multiplicities_and_invalid_ids(gpu):
    """A per-token multiplicity array gives the scalar path's statistics;
    expert ids outside [0, E) are skipped and counted."""
    import torch
    from paper_2606_01143_amd import binding as B
    shape = RouterShape(16, 3, 50, (7, 9))
    _announce(f"multiplicity array / invalid ids {shape}")
    inp = make_router_group(shape, seed=13)
    dev = _Dev(inp)
    rng = np.random.default_rng(5)
    m = rng.integers(0, 6, size=shape.prefix_len).astype(np.int32)
    r_bad = inp["r_p"].copy()
    bad = [(0, 0, -1), (3, 2, 16), (7, 1, 1000)]
    for u, j, v in bad:
        r_bad[u, j] = v
    mt = torch.from_numpy(m).cuda()
    rb = torch.from_numpy(r_bad).cuda()
    B.moe_stats_zero(dev.E, dev.stats)
    B.moe_aux_accumulate(dev.E, dev.k, dev.p_p, rb, dev.stats, token_multiplicity=mt, ws=dev.ws)
    dp = torch.empty_like(dev.p_p)
    B.moe_aux_grad(dev.E, dev.k, LAM, 2.5, dev.stats, dp, token_multiplicity=mt)
    torch.cuda.synchronize()
    got = dev.read()
    counts, mass, total = logical_stats(inp["p_p"], inp["r_p"], m, dev.E)
    for u, j, _ in bad:
        counts[inp["r_p"][u, j]] -= m[u]
    assert np.array_equal(got["C"], counts) and got["M"] == total and got["invalid"] == len(bad)
    assert _rel(got["R"], mass) <= 1e-12
    f = counts / (dev.k * total)
    ref_dp = 2.5 * LAM * dev.E * np.outer(m, f) / total
    assert _rel(dp.cpu().numpy(), ref_dp) <= 1e-6


@pytest.mark.gpu
def test_moe_zero_total_gives_zeros(gpu):
    import torch
    from paper_2606_01143_amd import binding as B
    inp = make_router_group(RouterShape(8, 2, 10, (3,)), seed=17)
    dev = _Dev(inp)
    B.moe_stats_zero(dev.E, dev.stats)
    B.moe_aux_accumulate(dev.E, dev.k, dev.p_p, dev.r_p, dev.stats, multiplicity=0, ws=dev.ws)
    dp = torch.full_like(dev.p_p, 3.0)
    B.moe_aux_loss(dev.E, dev.k, LAM, dev.stats, dev.f, dev.pe, dev.loss)
    B.moe_aux_grad(dev.E, dev.k, LAM, 1.0, dev.stats, dp, multiplicity=0)
    torch.cuda.synchronize()
    got = dev.read()
    assert got["M"] == 0 and not got["C"].any() and got["L"] == 0.0
    assert not got["f"].any() and not got["P"].any() and not dp.cpu().numpy().any()


@pytest.mark.gpu
def test_moe_step_in_a_hip_graph_replays_exactly(gpu):
    """The reuse step (stats zero, accumulates, loss, gradients) captured in a
    HIP graph: every replay, with eager library work and synchronizations in
    between, reproduces the eager result bitwise."""
    import torch
    from paper_2606_01143_amd import binding as B
    shape = RouterShape(64, 4, 300, (70, 129, 33))
    _announce(f"graph replay {shape}")
    inp = make_router_group(shape, seed=19)
    dev = _Dev(inp)
    dp_p, dp_s = torch.empty_like(dev.p_p), torch.empty_like(dev.p_s)

    def step():
        B.moe_stats_zero(dev.E, dev.stats)
        B.moe_aux_accumulate(dev.E, dev.k, dev.p_p, dev.r_p, dev.stats, multiplicity=dev.n, ws=dev.ws)
        for i in range(dev.n):
            a, b = dev.cu[i], dev.cu[i + 1]
            B.moe_aux_accumulate(dev.E, dev.k, dev.p_s[a:b], dev.r_s[a:b], dev.stats, ws=dev.ws)
        B.moe_aux_loss(dev.E, dev.k, LAM, dev.stats, dev.f, dev.pe, dev.loss)
        B.moe_aux_grad(dev.E, dev.k, LAM, 1.0, dev.stats, dp_p, multiplicity=dev.n)
        B.moe_aux_grad(dev.E, dev.k, LAM, 1.0, dev.stats, dp_s)

    step()
    torch.cuda.synchronize()
    ref = (dev.stats.clone(), dev.loss.clone(), dp_p.clone(), dp_s.clone())
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    other = torch.empty_like(dev.stats)
    for rep in range(3):
        # eager work on the same buffers between replays
        dp_p.fill_(5.0)
        B.moe_stats_zero(dev.E, other)
        B.moe_aux_accumulate(dev.E, dev.k, dev.p_s, dev.r_s, other, ws=dev.ws)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = (dev.stats, dev.loss, dp_p, dp_s)
        assert all(torch.equal(x, y) for x, y in zip(got, ref)), rep
