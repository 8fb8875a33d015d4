"""The decoder layer through the three-phase schedule on the GPU, against
the fp64 oracle's dense per-trajectory layer (tolerance 2e-2 max-abs-
relative for bf16), and the layer's token-wise kernels against plain
PyTorch fp32 of the same formulas."""
import numpy as np
import pytest

from oracle.compare import max_abs_rel
from oracle.layer import dense_layer_reference
from synthetic.layer import LAYER_SHAPES, LayerShape, make_layer_group

TOL = 2e-2


def _announce(what):
    print(f"\n[gpu layer] {what}", flush=True)


def _np(t):
    return t.float().cpu().numpy().astype(np.float64)


def _check(got, ref, what):
    errs = {"y_p": max_abs_rel(_np(got["y_p"]), ref["y_p"]), "dx_p": max_abs_rel(_np(got["dx_p"]), ref["dx_p"])}
    for i, (y, dx) in enumerate(zip(got["y_s"], got["dx_s"])):
        errs[f"y_s{i}"] = max_abs_rel(_np(y), ref["y_s"][i])
        errs[f"dx_s{i}"] = max_abs_rel(_np(dx), ref["dx_s"][i])
    for k, v in got["dw"].items():
        errs[f"d{k}"] = max_abs_rel(_np(v), ref["dw"][k])
    bad = {k: v for k, v in errs.items() if not v <= TOL}
    assert not bad, f"{what}: {bad}"
    return errs


CASES = [
    ("small", LAYER_SHAPES["small_layer"]),
    ("llama3_width_p256", LayerShape(4096, 32, 8, 128, 14336, 256, (64, 33))),
]


@pytest.mark.gpu
@pytest.mark.parametrize("name,shape", CASES, ids=[c[0] for c in CASES])
def test_layer_schedule_and_dense_match_oracle(gpu, name, shape):
    from paper_2606_01143_amd.layer import DecoderLayer
    _announce(f"{name} {shape}")
    inp = make_layer_group(shape, seed=9)
    ref = dense_layer_reference(inp)
    layer = DecoderLayer(inp)
    _check(layer.run_schedule(), ref, "schedule")
    _check(layer.run_dense(), ref, "dense")


@pytest.mark.gpu
def test_token_ops_match_fp32_formulas(gpu):
    import torch
    from paper_2606_01143_amd import binding as B
    _announce("token-wise ops")
    g = torch.Generator(device="cuda").manual_seed(3)
    bf = torch.bfloat16
    rnd = lambda *s: torch.randn(*s, generator=g, device="cuda").to(bf)
    rel = lambda a, b: ((a.float() - b.float()).abs().max() / b.float().abs().max()).item()
    # RMSNorm forward and backward (with the residual add)
    x, dy, add = rnd(37, 4096), rnd(37, 4096), rnd(37, 4096)
    y = torch.empty_like(x)
    r = torch.empty(37, dtype=torch.float32, device="cuda")
    B.rmsnorm_fwd(x, y, r, 1e-5)
    xf = x.float()
    rf = torch.rsqrt((xf * xf).mean(-1, keepdim=True) + 1e-5)
    assert rel(y, xf * rf) < 1e-2 and rel(r, rf[:, 0]) < 1e-5
    dx = torch.empty_like(x)
    B.rmsnorm_bwd(x, r, dy, dx, add=add)
    dyf = dy.float()
    ref = rf * dyf - rf ** 3 * xf * (dyf * xf).mean(-1, keepdim=True) + add.float()
    assert rel(dx, ref) < 1e-2
    # RoPE forward, and backward as the inverse rotation
    q = rnd(50, 8, 128)
    qr, qb = torch.empty_like(q), torch.empty_like(q)
    B.rope_fwd(q, qr, 1000, 500000.0)
    pos = torch.arange(1000, 1050, dtype=torch.float64, device="cuda")
    inv = 500000.0 ** (-torch.arange(64, dtype=torch.float64, device="cuda") * 2 / 128)
    ang = pos[:, None] * inv[None, :]
    cos = torch.cat([ang.cos(), ang.cos()], -1)[:, None, :].float()
    sin = torch.cat([ang.sin(), ang.sin()], -1)[:, None, :].float()
    qf = q.float()
    ref = qf * cos + torch.cat([-qf[..., 64:], qf[..., :64]], -1) * sin
    assert rel(qr, ref) < 1e-2
    B.rope_bwd(qr, qb, 1000, 500000.0)
    assert rel(qb, q) < 2e-2
    # SwiGLU forward and backward
    gt, ut, dm = rnd(64, 14336), rnd(64, 14336), rnd(64, 14336)
    m, dg, du = torch.empty_like(gt), torch.empty_like(gt), torch.empty_like(gt)
    B.swiglu_fwd(gt, ut, m)
    B.swiglu_bwd(gt, ut, dm, dg, du)
    gf, uf, dmf = gt.float(), ut.float(), dm.float()
    s = torch.sigmoid(gf)
    assert rel(m, gf * s * uf) < 1e-2
    assert rel(dg, dmf * uf * s * (1 + gf * (1 - s))) < 1e-2 and rel(du, dmf * gf * s) < 1e-2
