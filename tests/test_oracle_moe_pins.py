"""Pins of the MoE auxiliary-loss accounting oracle (CPU only).

* App. B's claim: multiplicity-weighted statistics over the physical tokens
  equal the statistics of the materialized batch with N explicit prefix
  copies, and the prefix gradient equals the sum over the copies.
* Closed forms of the Switch-style loss: perfect balance gives lambda,
  collapse onto k experts gives lambda E / k.
* Invariants: sum_e f_e = 1 and sum_e P_e = 1.
* The gradient against torch autograd in fp64 (C_e held constant) and
  against central finite differences.
* Planted mistakes in the oracle are caught by at least one pin.
"""
import numpy as np
import pytest
import torch

import oracle.moe_aux as om
from synthetic.moe import RouterShape, make_router_group

LAM = 0.01


def _both(shape, seed, lam=LAM, n_copies=-1, ragged=None):
    inp = make_router_group(shape, seed=seed, ragged=ragged)
    return inp, om.reuse_reference(inp, lam, n_copies), om.materialized_reference(inp, lam, n_copies)


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)) if a.size else 0.0


def pin_materialized(shape, seed, n_copies=-1, ragged=None):
    inp, a, b = _both(shape, seed, n_copies=n_copies, ragged=ragged)
    assert np.array_equal(a["C"], b["C"]) and a["M"] == b["M"]
    return max(_rel(a["R"], b["R"]), _rel(a["L"], b["L"]), _rel(a["dp_p"], b["dp_p"]),
               _rel(a["dp_s"], b["dp_s"]))


@pytest.mark.parametrize("shape,seed,n_copies,ragged", [
    (RouterShape(8, 2, 24, (5, 9, 3)), 1, -1, None),
    (RouterShape(16, 1, 7, (1,)), 2, -1, None),          # N = 1: nothing shared
    (RouterShape(6, 6, 10, (4, 4)), 3, -1, None),        # k = E
    (RouterShape(12, 3, 0, (5, 2, 8)), 4, -1, None),     # P = 0
    (RouterShape(128, 8, 96, (0,) * 5), 5, -1, (3, 40)),  # ragged, Qwen3-MoE router shape
    (RouterShape(8, 2, 24, (5, 9, 3)), 6, 7, None),      # reduction scope of 7 logical copies
])
def test_logical_accounting_equals_materialized_copies(shape, seed, n_copies, ragged):
    assert pin_materialized(shape, seed, n_copies, ragged) < 1e-12


def _balanced(e, k, c):
    """c * e tokens, uniform probabilities, token u selects experts u .. u+k-1 mod e."""
    n = c * e
    p = np.full((n, e), 1.0 / e)
    r = (np.arange(n)[:, None] + np.arange(k)[None, :]) % e
    return p, r


def pin_balance(e=8, k=3, c=5, m=4):
    p, r = _balanced(e, k, c)
    counts, mass, total = om.logical_stats(p, r, np.full(len(p), m), e)
    _, _, loss = om.aux_loss(counts, mass, total, k, LAM)
    return abs(loss - LAM) / LAM


def pin_collapse(e=8, k=3, n=11):
    p = np.zeros((n, e))
    p[:, :k] = 1.0 / k
    r = np.tile(np.arange(k), (n, 1))
    m = np.arange(1, n + 1)
    counts, mass, total = om.logical_stats(p, r, m, e)
    _, _, loss = om.aux_loss(counts, mass, total, k, LAM)
    return abs(loss - LAM * e / k) / (LAM * e / k)


def test_closed_forms():
    assert pin_balance() < 1e-14
    assert pin_collapse() < 1e-14


def test_invariants():
    inp, a, _ = _both(RouterShape(10, 3, 13, (4, 7, 1)), 7)
    assert abs(a["f"].sum() - 1) < 1e-14
    assert abs(a["P"].sum() - 1) < 1e-6  # float32 probability rows
    assert a["C"].sum() == inp["shape"].top_k * a["M"]


def pin_autograd(shape=RouterShape(9, 2, 6, (3, 5)), seed=8):
    inp = make_router_group(shape, seed=seed)
    a = om.reuse_reference(inp, LAM)
    n = shape.n
    m = np.concatenate([np.full(shape.prefix_len, n), np.ones(int(sum(shape.suffix_lens)))])
    p = torch.tensor(np.concatenate([inp["p_p"], inp["p_s"]]), dtype=torch.float64, requires_grad=True)
    c = torch.tensor(a["C"], dtype=torch.float64)  # hard count: a constant
    mt = torch.tensor(m, dtype=torch.float64)
    total = mt.sum()
    loss = LAM * shape.num_experts * torch.sum((c / (shape.top_k * total)) * ((mt[:, None] * p).sum(0) / total))
    loss.backward()
    g = p.grad.numpy()
    got = np.concatenate([a["dp_p"], a["dp_s"]])
    return max(_rel(got, g), abs(loss.item() - a["L"]) / abs(a["L"]))


def pin_finite_differences(shape=RouterShape(5, 2, 4, (2, 3)), seed=9, h=1e-6):
    inp = make_router_group(shape, seed=seed)
    a = om.reuse_reference(inp, LAM)
    worst = 0.0
    for key, gkey in (("p_p", "dp_p"), ("p_s", "dp_s")):
        for idx in [(0, 0), (1, 3), (0, 4)]:
            if idx[0] >= inp[key].shape[0]:
                continue
            vals = []
            for sgn in (1, -1):
                x = {k: (v.astype(np.float64).copy() if isinstance(v, np.ndarray) and v.dtype.kind == "f" else v)
                     for k, v in inp.items()}
                x[key][idx] += sgn * h
                # the counts stay those of the unperturbed selection (hard, no gradient)
                vals.append(om.reuse_reference(x, LAM)["L"])
            fd = (vals[0] - vals[1]) / (2 * h)
            worst = max(worst, abs(fd - a[gkey][idx]) / max(abs(a[gkey][idx]), 1e-12))
    return worst


def test_gradient_against_autograd_and_finite_differences():
    assert pin_autograd() < 1e-12
    assert pin_finite_differences() < 1e-6


def _stats_without_multiplicity_in_mass(p, r, m, n_experts):
    counts, _, total = _orig_stats(p, r, m, n_experts)
    return counts, np.asarray(p, np.float64).sum(axis=0), total


def _stats_unweighted_total(p, r, m, n_experts):
    counts, mass, _ = _orig_stats(p, r, m, n_experts)
    return counts, mass, len(m)


def _loss_without_k(counts, mass, total, top_k, lam):
    return _orig_loss(counts, mass, total, 1, lam)


def _grad_without_multiplicity(f, total, m, lam):
    return _orig_grad(f, total, np.ones_like(np.asarray(m)), lam)


_orig_stats, _orig_loss, _orig_grad = om.logical_stats, om.aux_loss, om.aux_grad


@pytest.mark.parametrize("mutation", ["mass_without_m", "unweighted_total", "loss_without_k",
                                      "grad_without_m"])
def test_planted_mistakes_are_caught(monkeypatch, mutation):
    if mutation == "mass_without_m":
        monkeypatch.setattr(om, "logical_stats", _stats_without_multiplicity_in_mass)
    elif mutation == "unweighted_total":
        monkeypatch.setattr(om, "logical_stats", _stats_unweighted_total)
    elif mutation == "loss_without_k":
        monkeypatch.setattr(om, "aux_loss", _loss_without_k)
    elif mutation == "grad_without_m":
        monkeypatch.setattr(om, "aux_grad", _grad_without_multiplicity)
    caught = []
    try:
        caught.append(pin_materialized(RouterShape(8, 2, 24, (5, 9, 3)), 1) > 1e-9)
    except AssertionError:
        caught.append(True)
    caught.append(pin_balance() > 1e-9)
    caught.append(pin_collapse() > 1e-9)
    caught.append(pin_autograd() > 1e-9)
    caught.append(pin_finite_differences() > 1e-5)
    assert any(caught), f"mutation {mutation} escaped every pin"
