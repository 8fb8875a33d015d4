"""Pins of the decoder-layer oracle (CPU only).

* The schedule reordered at the layer level (prefix forward once, suffix
  forward/backward with the prefix K/V gradients accumulated, one prefix
  backward with the injected cache) equals the dense per-trajectory
  computation in fp64, weights included (Prop. 1; App. A.6: the weight
  gradient is the prefix part once plus the suffix parts).
* Finite differences of the dense group loss on inputs and weights.
* Rotate-half RoPE: identity at position 0, norm-preserving, and the score
  between two rotated vectors depends only on their position difference.
* RMSNorm with unit gain gives rows of unit root-mean-square.
* Zero weights: the layer is the identity and passes dY through.
* Planted mistakes in the oracle are caught.
"""
import numpy as np
import pytest
import torch

import oracle.layer as ol
from synthetic.layer import LayerShape, make_layer_group


def _rel(x, y):
    x, y = np.asarray(x, np.float64), np.asarray(y, np.float64)
    return float(np.max(np.abs(x - y)) / max(np.max(np.abs(y)), 1e-300))


def pin_reordered(shape, seed, ragged=None):
    inp = make_layer_group(shape, seed=seed, ragged=ragged)
    a, b = ol.dense_layer_reference(inp), ol.reordered_layer_reference(inp)
    errs = [_rel(b["y_p"], a["y_p"]), _rel(b["dx_p"], a["dx_p"])]
    errs += [_rel(x, y) for x, y in zip(b["y_s"], a["y_s"])] + [_rel(x, y) for x, y in zip(b["dx_s"], a["dx_s"])]
    errs += [_rel(b["dw"][k], a["dw"][k]) for k in ol.W_KEYS]
    return max(errs)


@pytest.mark.parametrize("shape,seed", [
    (LayerShape(16, 2, 1, 8, 32, 7, (3, 5), "f32"), 1),
    (LayerShape(32, 4, 2, 8, 48, 12, (4, 1, 9), "f32"), 2),
    (LayerShape(24, 2, 2, 12, 40, 5, (6,), "f32"), 3),   # N = 1
])
def test_layer_reordered_equals_dense(shape, seed):
    assert pin_reordered(shape, seed) < 1e-12


def pin_finite_differences(seed=4, h=1e-4):
    inp = make_layer_group(LayerShape(8, 2, 1, 4, 16, 3, (2, 3), "f32"), seed=seed)
    ref = ol.dense_layer_reference(inp)
    worst = 0.0
    probes = [("x_p", None, (1, 2), "dx_p"), ("x_s", 1, (2, 5), None), ("wq", "w", (3, 1), "wq"),
              ("wk", "w", (0, 2), "wk"), ("wv", "w", (5, 3), "wv"), ("wo", "w", (2, 6), "wo"),
              ("wg", "w", (7, 11), "wg"), ("wd", "w", (13, 4), "wd")]
    for key, sel, idx, gkey in probes:
        vals = []
        for sgn in (1, -1):
            x = {"shape": inp["shape"], "weights": {k: v.astype(np.float64).copy() for k, v in inp["weights"].items()},
                 "x_p": inp["x_p"].astype(np.float64).copy(), "x_s": [v.astype(np.float64).copy() for v in inp["x_s"]],
                 "dy_s": inp["dy_s"], "dy_p": inp["dy_p"]}
            if sel == "w":
                x["weights"][key][idx] += sgn * h
            elif key == "x_s":
                x["x_s"][sel][idx] += sgn * h
            else:
                x[key][idx] += sgn * h
            vals.append(ol.group_loss(x))
        fd = (vals[0] - vals[1]) / (2 * h)
        if sel == "w":
            g = ref["dw"][gkey][idx]
        elif key == "x_s":
            g = ref["dx_s"][sel][idx]
        else:
            g = ref[gkey][idx]
        worst = max(worst, abs(fd - g) / max(abs(g), 1e-8))
    return worst


def test_layer_finite_differences():
    assert pin_finite_differences() < 1e-5


def test_rope_properties():
    torch.manual_seed(0)
    d, theta = 16, 500000.0
    q = torch.randn(1, 1, d, dtype=torch.float64)
    k = torch.randn(1, 1, d, dtype=torch.float64)
    # position 0 is the identity; rotations keep the norm
    assert torch.allclose(ol.rope(q, torch.tensor([0]), theta), q, atol=0, rtol=0)
    r = ol.rope(q, torch.tensor([123]), theta)
    assert abs(r.norm().item() - q.norm().item()) < 1e-12
    # the score depends only on the position difference
    def score(m, n):
        return float((ol.rope(q, torch.tensor([m]), theta) * ol.rope(k, torch.tensor([n]), theta)).sum())
    assert abs(score(7, 3) - score(104, 100)) < 1e-10
    assert abs(score(7, 3) - score(3, 7)) > 1e-6  # not symmetric: the angle's sign matters
    # the rotation itself: pair (j, j + d/2) as the complex number
    # x_j + i x_(j+d/2), multiplied by exp(i m theta^(-2j/d))
    half = d // 2
    z = torch.complex(q[..., :half], q[..., half:])
    ang = 123 * theta ** (-torch.arange(half, dtype=torch.float64) * 2.0 / d)
    zr = z * torch.exp(1j * ang)
    assert torch.allclose(r, torch.cat([zr.real, zr.imag], dim=-1), atol=1e-12, rtol=0)


def test_rmsnorm_unit_rms():
    x = torch.randn(5, 32, dtype=torch.float64) * 3.0
    y = ol.rms(x, 0.0)
    assert torch.allclose((y * y).mean(dim=-1), torch.ones(5, dtype=torch.float64), atol=1e-12)


def pin_zero_weights():
    """All weights zero: both sublayers add nothing, so Y = X and dX = dY
    (the prefix's summed over the trajectories)."""
    inp = make_layer_group(LayerShape(8, 2, 1, 4, 16, 3, (2, 3), "f32"), seed=5)
    inp["weights"] = {k: np.zeros_like(v) for k, v in inp["weights"].items()}
    ref = ol.dense_layer_reference(inp)
    errs = [_rel(ref["y_p"], inp["x_p"]), _rel(ref["dx_p"], np.sum(np.asarray(inp["dy_p"], np.float64), axis=0))]
    errs += [_rel(y, x) for y, x in zip(ref["y_s"], inp["x_s"])]
    errs += [_rel(g, dy) for g, dy in zip(ref["dx_s"], inp["dy_s"])]
    return max(errs)


def test_zero_weights_closed_form():
    assert pin_zero_weights() < 1e-14


_orig_rope, _orig_tail = ol.rope, ol._tail


def _rope_wrong_sign(x, pos, theta):
    return _orig_rope(x, -pos, theta)


def _rope_no_rotation(x, pos, theta):
    return x


def _tail_no_residual(x, o, W, shp):
    return _orig_tail(x, o, W, shp) - x


@pytest.mark.parametrize("mutation", ["rope_wrong_sign", "rope_missing", "no_residual"])
def test_planted_mistakes_are_caught(monkeypatch, mutation):
    fn = {"rope_wrong_sign": ("rope", _rope_wrong_sign), "rope_missing": ("rope", _rope_no_rotation),
          "no_residual": ("_tail", _tail_no_residual)}[mutation]
    monkeypatch.setattr(ol, fn[0], fn[1])
    caught = [pin_finite_differences() > 1e-3, pin_zero_weights() > 1e-9]
    try:
        test_rope_properties()
        caught.append(False)
    except AssertionError:
        caught.append(True)
    assert any(caught), mutation


# ---------------------------------------------------------------------------
# the stack of layers (App. A.7)
# ---------------------------------------------------------------------------
from synthetic.layer import make_stack_group  # noqa: E402


def pin_stack_reordered(shape, layers, seed, ragged=None):
    inp = make_stack_group(shape, layers, seed=seed, ragged=ragged)
    a, b = ol.dense_stack_reference(inp), ol.reordered_stack_reference(inp)
    errs = [_rel(b["y_p"], a["y_p"]), _rel(b["dx_p"], a["dx_p"])]
    errs += [_rel(x, y) for x, y in zip(b["y_s"], a["y_s"])] + [_rel(x, y) for x, y in zip(b["dx_s"], a["dx_s"])]
    errs += [_rel(bw[k], aw[k]) for bw, aw in zip(b["dw"], a["dw"]) for k in ol.W_KEYS]
    return max(errs)


@pytest.mark.parametrize("shape,layers,seed", [
    (LayerShape(16, 2, 1, 8, 32, 7, (3, 5), "f32"), 2, 1),
    (LayerShape(32, 4, 2, 8, 48, 12, (4, 1, 9), "f32"), 3, 2),
    (LayerShape(24, 2, 2, 12, 40, 5, (6,), "f32"), 2, 3),   # N = 1
])
def test_stack_reordered_equals_dense(shape, layers, seed):
    """Prop. 1 across layers: the schedule over the stack (prefix once
    through every layer, suffixes against each layer's cached prefix K/V,
    the prefix backward from the top with each layer's cache injected and
    the adjoint chained downwards) equals the dense per-trajectory stack,
    every layer's weight gradients included."""
    assert pin_stack_reordered(shape, layers, seed) < 1e-12


def test_stack_of_one_layer_is_the_layer():
    """One layer's stack is the single-layer reference (same draws up to
    the weight list)."""
    shape = LayerShape(16, 2, 1, 8, 32, 7, (3, 5), "f32")
    st = make_stack_group(shape, 1, seed=6)
    one = dict(st, weights=st["weights"][0])
    a, b = ol.dense_stack_reference(st), ol.dense_layer_reference(one)
    assert _rel(a["dx_p"], b["dx_p"]) < 1e-14 and _rel(a["y_p"], b["y_p"]) < 1e-14
    for k in ol.W_KEYS:
        assert _rel(a["dw"][0][k], b["dw"][k]) < 1e-14


def test_stack_finite_differences(h=1e-4):
    """The dense stack's gradients against central differences of the group
    loss, on the bottom input, a suffix input and weights of both layers
    (the adjoint chained through the layer above included)."""
    inp = make_stack_group(LayerShape(8, 2, 1, 4, 16, 3, (2, 3), "f32"), 2, seed=8)
    ref = ol.dense_stack_reference(inp)
    probes = [("x_p", None, (1, 2)), ("x_s", 1, (2, 5)), ("wq", 0, (3, 1)), ("wk", 0, (0, 2)),
              ("wv", 1, (5, 3)), ("wd", 0, (13, 4)), ("wg", 1, (7, 11))]
    worst = 0.0
    for key, sel, idx in probes:
        vals = []
        for sgn in (1, -1):
            x = {"shape": inp["shape"], "layers": 2,
                 "weights": [{k: v.astype(np.float64).copy() for k, v in w.items()} for w in inp["weights"]],
                 "x_p": inp["x_p"].astype(np.float64).copy(),
                 "x_s": [v.astype(np.float64).copy() for v in inp["x_s"]],
                 "dy_s": inp["dy_s"], "dy_p": inp["dy_p"]}
            if key == "x_p":
                x["x_p"][idx] += sgn * h
            elif key == "x_s":
                x["x_s"][sel][idx] += sgn * h
            else:
                x["weights"][sel][key][idx] += sgn * h
            vals.append(ol.stack_group_loss(x))
        fd = (vals[0] - vals[1]) / (2 * h)
        if key == "x_p":
            an = ref["dx_p"][idx]
        elif key == "x_s":
            an = ref["dx_s"][sel][idx]
        else:
            an = ref["dw"][sel][key][idx]
        worst = max(worst, abs(fd - an) / max(abs(an), 1e-3))
    assert worst < 1e-6, worst


def test_stack_planted_mistake_is_caught(monkeypatch):
    """Dropping the chained adjoint (every layer's Phase C starting from
    G_Y instead of the adjoint from the layer above) breaks the stack pin."""
    orig = ol.reordered_stack_reference

    def broken(inp):
        shp = inp["shape"]
        out = orig(inp)
        # recompute Phase C of the bottom layer alone with the top G_Y
        one = dict(inp, weights=inp["weights"][0], x_s=[np.zeros_like(x) for x in inp["x_s"]])
        return dict(out, dx_p=ol.reordered_layer_reference(one)["dx_p"])

    monkeypatch.setattr(ol, "reordered_stack_reference", broken)
    shape = LayerShape(16, 2, 1, 8, 32, 7, (3, 5), "f32")
    assert pin_stack_reordered(shape, 2, 1) > 1e-6
