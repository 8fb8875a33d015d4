"""Pins of the fp64 oracle to things other than itself (CPU only).

Each pin is chosen so that a plausible mistake in the oracle (a dropped term,
a wrong sign or index, a transposed operand, a missing scale) fails at least
one of them; ``test_planted_mistakes_are_caught`` plants such mistakes in the
oracle and checks that.

* Proposition 1 (paper Sec. 3.1, App. A.4): the reordered schedule equals the
  dense definition, for any microbatch split and order.
* N = 1 is ordinary causal attention (paper Sec. 6, "not useful at N=1"):
  torch's scaled_dot_product_attention + autograd in fp64 on the CPU.
* P = 0: N independent causal attentions (same library routine).
* Finite differences of the group loss on every input element (chain rule).
* Suffix-only loss (App. A.5): G_Y = 0 gives dQ_P = 0 exactly and
  dK_P = G_K, dV_P = G_V.
* Invariants: softmax-backward rows sum to zero (sum of dK over keys = 0),
  probability rows sum to one (value-sum identity), bilinearity of the
  scores <dQ,Q> = <dK,K>, linearity in V <dV,V> = sum <dO,O>.
* Uniform attention (Q = 0): closed forms for O and dV.
"""
import itertools

import numpy as np
import pytest
import torch

import oracle.attention as oa
from oracle import dense_group_reference, three_phase_reference, group_loss, max_abs_rel
from synthetic import GroupShape, make_group

KEYS = ["o_p", "lse_p", "o_s", "lse_s", "dq_p", "dk_p", "dv_p",
        "dq_s", "dk_s", "dv_s", "g_k", "g_v"]
GRAD_INPUTS = [("q_p", "dq_p"), ("k_p", "dk_p"), ("v_p", "dv_p"),
               ("q_s", "dq_s"), ("k_s", "dk_s"), ("v_s", "dv_s")]


def exact_gy(inp):
    return inp["do_p"].astype(np.float64).sum(axis=0)


def _sdpa_reference(q, k, v, do, scale):
    """fp64 torch SDPA + autograd for one sequence; [L,H,d] in, [L,H,d] out."""
    def t(x):
        return torch.tensor(np.asarray(x, np.float64).transpose(1, 0, 2)[None], requires_grad=True)
    tq, tk, tv = t(q), t(k), t(v)
    o = torch.nn.functional.scaled_dot_product_attention(
        tq, tk, tv, is_causal=True, scale=scale, enable_gqa=True)
    o.backward(torch.tensor(np.asarray(do, np.float64).transpose(1, 0, 2)[None]))
    back = lambda x: x.detach().numpy()[0].transpose(1, 0, 2)
    return back(o), back(tq.grad), back(tk.grad), back(tv.grad)


# --------------------------------------------------------------------------
# pin functions (return an error figure; the mutation test reuses them)
# --------------------------------------------------------------------------

def pin_prop1(inp, splits):
    dense = dense_group_reference(inp)
    err = 0.0
    for mbs in splits:
        sched = three_phase_reference(inp, microbatches=mbs, g_y=exact_gy(inp))
        err = max(err, max(max_abs_rel(sched[k], dense[k]) for k in KEYS))
    return err


def pin_sdpa_n1(inp):
    """N = 1: the group is one ordinary causal attention over [P||S]."""
    shp = inp["shape"]
    sc = 1.0 / np.sqrt(shp.head_dim)
    q = np.concatenate([inp["q_p"], inp["q_s"]])
    k = np.concatenate([inp["k_p"], inp["k_s"]])
    v = np.concatenate([inp["v_p"], inp["v_s"]])
    do = np.concatenate([inp["do_p"][0], inp["do_s"]])
    o, dq, dk, dv = _sdpa_reference(q, k, v, do, sc)
    p = shp.prefix_len
    err = 0.0
    for ref in (dense_group_reference(inp), three_phase_reference(inp, g_y=exact_gy(inp))):
        err = max(err,
                  max_abs_rel(ref["o_p"], o[:p]), max_abs_rel(ref["o_s"], o[p:]),
                  max_abs_rel(ref["dq_p"], dq[:p]), max_abs_rel(ref["dq_s"], dq[p:]),
                  max_abs_rel(ref["dk_p"], dk[:p]), max_abs_rel(ref["dk_s"], dk[p:]),
                  max_abs_rel(ref["dv_p"], dv[:p]), max_abs_rel(ref["dv_s"], dv[p:]))
    return err


def pin_finite_differences(inp, h=1e-6):
    """Central differences of L = sum_i <dO(i), O(i)> on every input element."""
    ref = dense_group_reference(inp)
    sched = three_phase_reference(inp, g_y=exact_gy(inp))
    err = 0.0
    for name, gname in GRAD_INPUTS:
        x = inp[name]
        fd = np.zeros(x.shape)
        for idx in itertools.product(*[range(s) for s in x.shape]):
            plus = dict(inp); minus = dict(inp)
            xp = x.astype(np.float64).copy(); xm = x.astype(np.float64).copy()
            xp[idx] += h; xm[idx] -= h
            plus[name] = xp; minus[name] = xm
            fd[idx] = (group_loss(plus) - group_loss(minus)) / (2 * h)
        scale = max(np.max(np.abs(fd)), 1e-30)
        err = max(err, np.max(np.abs(ref[gname] - fd)) / scale,
                  np.max(np.abs(sched[gname] - fd)) / scale)
    return err


def pin_invariants(inp):
    """Invariants that hold for the exact gradients of any inputs."""
    ref = three_phase_reference(inp, g_y=exact_gy(inp))
    shp = inp["shape"]
    g = shp.group
    dk_all = np.concatenate([ref["dk_p"], ref["dk_s"]])
    dv_all = np.concatenate([ref["dv_p"], ref["dv_s"]])
    # (a) softmax-backward rows sum to zero => sum over all keys of dK is 0
    key_shift = np.max(np.abs(dk_all.sum(axis=0))) / np.max(np.abs(dk_all))
    # (b) probability rows sum to one => sum over keys of dV equals the sum
    #     over all rows and group heads of the upstream adjoints
    dO_all = np.concatenate([exact_gy(inp), inp["do_s"].astype(np.float64)])
    rhs = dO_all.reshape(dO_all.shape[0], shp.num_kv_heads, g, shp.head_dim).sum(axis=(0, 2))
    value_sum = np.max(np.abs(dv_all.sum(axis=0) - rhs)) / np.max(np.abs(rhs))
    # (c) bilinear scores: <dQ,Q> = <dK,K>
    lq = np.sum(ref["dq_p"] * inp["q_p"]) + np.sum(ref["dq_s"] * inp["q_s"])
    lk = np.sum(ref["dk_p"] * inp["k_p"]) + np.sum(ref["dk_s"] * inp["k_s"])
    bilinear = abs(lq - lk) / max(abs(lq), abs(lk), 1e-30)
    # (d) linear in V: <dV,V> = <G_Y,O_P> + sum_i <dO_S(i),O_S(i)>
    lv = np.sum(ref["dv_p"] * inp["v_p"]) + np.sum(ref["dv_s"] * inp["v_s"])
    lo = np.sum(exact_gy(inp) * ref["o_p"]) + np.sum(inp["do_s"] * ref["o_s"])
    linear_v = abs(lv - lo) / max(abs(lo), 1e-30)
    return {"key_shift": key_shift, "value_sum": value_sum,
            "bilinear": bilinear, "linear_v": linear_v}


def pin_uniform_attention(inp):
    """Q = 0: every visible key gets weight 1/n_r, so O_r is the mean of the
    visible V rows, dK = 0, and dV_j = sum over rows r that see j of dO_r/n_r."""
    z = dict(inp)
    z["q_p"] = np.zeros_like(inp["q_p"]); z["q_s"] = np.zeros_like(inp["q_s"])
    ref = three_phase_reference(z, g_y=exact_gy(z))
    shp = inp["shape"]
    p, g = shp.prefix_len, shp.group
    cu = inp["cu_seqlens"]
    gy = exact_gy(z)
    vp = inp["v_p"].astype(np.float64)
    vs = inp["v_s"].astype(np.float64)
    dos = inp["do_s"].astype(np.float64)
    exp_op = np.zeros_like(ref["o_p"])
    exp_dvp = np.zeros_like(ref["dv_p"])
    for r in range(p):
        for h in range(shp.num_q_heads):
            exp_op[r, h] = vp[: r + 1, h // g].mean(axis=0)
            exp_dvp[: r + 1, h // g] += gy[r, h] / (r + 1)
    exp_os = np.zeros_like(ref["o_s"])
    exp_dvs = np.zeros_like(ref["dv_s"])
    for i in range(len(cu) - 1):
        a, b = cu[i], cu[i + 1]
        for t in range(b - a):
            n_r = p + t + 1
            for h in range(shp.num_q_heads):
                vis = np.concatenate([vp[:, h // g], vs[a:a + t + 1, h // g]])
                exp_os[a + t, h] = vis.mean(axis=0)
                exp_dvp[:, h // g] += dos[a + t, h] / n_r
                exp_dvs[a:a + t + 1, h // g] += dos[a + t, h] / n_r
    dk = max(np.max(np.abs(ref["dk_p"]), initial=0.0), np.max(np.abs(ref["dk_s"]), initial=0.0))
    return max(max_abs_rel(ref["o_p"], exp_op), max_abs_rel(ref["o_s"], exp_os),
               max_abs_rel(ref["dv_p"], exp_dvp), max_abs_rel(ref["dv_s"], exp_dvs), dk)


# --------------------------------------------------------------------------
# tests
# --------------------------------------------------------------------------

SHAPES = [
    GroupShape(2, 2, 8, 13, (4, 7, 1), "f32"),
    GroupShape(4, 2, 16, 37, (5, 11, 3, 9), "f32"),
    GroupShape(8, 1, 8, 20, (6, 2), "f32"),
]


@pytest.mark.parametrize("shape", SHAPES, ids=str)
def test_prop1_superposition_any_split_any_order(shape):
    inp = make_group(shape, seed=3)
    n = shape.n
    ids = list(range(n))
    splits = [
        [[i] for i in ids],                  # one suffix per microbatch
        [ids],                                # whole wave packed
        [[i] for i in reversed(ids)],         # reversed order
        [ids[::2], ids[1::2]],                # mixed packing
        [list(reversed(ids[1:])), [ids[0]]],  # permuted, packed
    ]
    assert pin_prop1(inp, splits) <= 1e-12


def test_microbatch_split_and_order_invariance_between_schedules():
    inp = make_group(GroupShape(4, 1, 8, 9, (3, 5, 2, 6), "f32"), seed=11)
    base = three_phase_reference(inp, microbatches=[[0], [1], [2], [3]])
    for mbs in ([[3, 1], [0, 2]], [[2], [0, 1, 3]], [[0, 1, 2, 3]], [[3], [2], [1], [0]]):
        other = three_phase_reference(inp, microbatches=mbs)
        assert max(max_abs_rel(other[k], base[k]) for k in KEYS) <= 1e-12


@pytest.mark.parametrize("shape", [GroupShape(4, 2, 8, 11, (6,), "f32"),
                                   GroupShape(3, 3, 16, 0, (9,), "f32"),
                                   GroupShape(2, 1, 8, 17, (1,), "f32")], ids=str)
def test_n1_is_ordinary_causal_attention(shape):
    inp = make_group(shape, seed=5)
    assert pin_sdpa_n1(inp) <= 1e-12


def test_p0_is_independent_causal_attentions():
    shape = GroupShape(4, 2, 8, 0, (5, 3, 7), "f32")
    inp = make_group(shape, seed=2)
    ref = three_phase_reference(inp)
    dense = dense_group_reference(inp)
    cu = inp["cu_seqlens"]
    sc = 1.0 / np.sqrt(8)
    for i in range(3):
        a, b = cu[i], cu[i + 1]
        o, dq, dk, dv = _sdpa_reference(inp["q_s"][a:b], inp["k_s"][a:b], inp["v_s"][a:b],
                                        inp["do_s"][a:b], sc)
        for r in (ref, dense):
            assert max_abs_rel(r["o_s"][a:b], o) <= 1e-12
            assert max_abs_rel(r["dq_s"][a:b], dq) <= 1e-12
            assert max_abs_rel(r["dk_s"][a:b], dk) <= 1e-12
            assert max_abs_rel(r["dv_s"][a:b], dv) <= 1e-12
    assert ref["dq_p"].size == 0 and ref["g_k"].size == 0


def test_finite_differences_tiny():
    inp = make_group(GroupShape(2, 1, 4, 3, (2, 3), "f32"), seed=7)
    assert pin_finite_differences(inp) <= 1e-7


def test_suffix_only_loss_gives_zero_query_gradient_and_pure_cache():
    inp = make_group(GroupShape(4, 2, 8, 10, (4, 6, 3), "f32"), seed=9, with_prefix_adjoint=False)
    ref = three_phase_reference(inp, g_y=np.zeros_like(inp["g_y"]))
    assert np.all(ref["dq_p"] == 0.0)
    assert np.array_equal(ref["dk_p"], ref["g_k"])
    assert np.array_equal(ref["dv_p"], ref["g_v"])
    assert np.max(np.abs(ref["g_k"])) > 0 and np.max(np.abs(ref["g_v"])) > 0
    dense = dense_group_reference(inp)
    assert max(max_abs_rel(ref[k], dense[k]) for k in KEYS if k != "dq_p") <= 1e-12
    assert np.max(np.abs(dense["dq_p"])) <= 1e-12


@pytest.mark.parametrize("shape", SHAPES, ids=str)
def test_invariants(shape):
    inp = make_group(shape, seed=13)
    res = pin_invariants(inp)
    for name, val in res.items():
        assert val <= 1e-12, (name, val)


def test_uniform_attention_closed_form():
    inp = make_group(GroupShape(4, 2, 8, 6, (3, 4), "f32"), seed=17)
    assert pin_uniform_attention(inp) <= 1e-12


def test_prefix_forward_identical_across_trajectories():
    inp = make_group(GroupShape(2, 1, 8, 12, (3, 9, 5), "f32"), seed=19)
    assert dense_group_reference(inp)["prefix_forward_spread"] <= 1e-13


# --------------------------------------------------------------------------
# planted mistakes in the oracle must be caught by the pins above
# --------------------------------------------------------------------------

def _dropped_rowsum(p, dp):
    return p * dp                                   # dropped the rowsum term


def _wrong_sign(p, dp):
    return p * (dp + np.sum(dp * p, axis=1, keepdims=True))


_ORIG_SBWD = oa._softmax_backward
_ORIG_PHASE_C = oa._phase_c_prefix_backward
_ORIG_PHASE_B = oa._phase_b_microbatch


def _phase_c_without_gv(q_p, k_p, v_p, o_p, g_y, g_k, g_v, sc, g):
    return _ORIG_PHASE_C(q_p, k_p, v_p, o_p, g_y, g_k, np.zeros_like(g_v), sc, g)


def _phase_b_swapped_heads(q_mb, k_mb, v_mb, do_mb, seg, k_p, v_p, sc, g):
    # reads kv head (h % Hkv) instead of h // G
    hq = q_mb.shape[1]
    perm = np.array([(h % k_p.shape[1]) * g + h // k_p.shape[1] for h in range(hq)])
    out = list(_ORIG_PHASE_B(q_mb[:, perm], k_mb, v_mb, do_mb[:, perm], seg, k_p, v_p, sc, g))
    inv = np.argsort(perm)
    out[0] = out[0][:, inv]; out[1] = out[1][inv]; out[2] = out[2][:, inv]
    return tuple(out)


def _causal_attention_no_scale_dk(q, k, v, do, scale, *, first_query_pos=0):
    o, lse, dq, dk, dv = _ORIG_CAUSAL(q, k, v, do, scale, first_query_pos=first_query_pos)
    return o, lse, dq, dk / scale, dv


_ORIG_CAUSAL = oa.causal_attention


@pytest.mark.parametrize("mutation", ["dropped_rowsum", "wrong_sign", "lost_gv_injection",
                                      "swapped_gqa_heads", "missing_dk_scale"])
def test_planted_mistakes_are_caught(monkeypatch, mutation):
    shape = GroupShape(4, 2, 4, 5, (3, 2), "f32")
    inp = make_group(shape, seed=23)
    if mutation == "dropped_rowsum":
        monkeypatch.setattr(oa, "_softmax_backward", _dropped_rowsum)
    elif mutation == "wrong_sign":
        monkeypatch.setattr(oa, "_softmax_backward", _wrong_sign)
    elif mutation == "lost_gv_injection":
        monkeypatch.setattr(oa, "_phase_c_prefix_backward", _phase_c_without_gv)
    elif mutation == "swapped_gqa_heads":
        monkeypatch.setattr(oa, "_phase_b_microbatch", _phase_b_swapped_heads)
    elif mutation == "missing_dk_scale":
        monkeypatch.setattr(oa, "causal_attention", _causal_attention_no_scale_dk)
    caught = []
    caught.append(pin_prop1(inp, [[[0], [1]]]) > 1e-6)
    caught.append(pin_finite_differences(make_group(GroupShape(2, 1, 3, 2, (2, 1), "f32"), seed=1)) > 1e-5)
    caught.append(max(pin_invariants(inp).values()) > 1e-6)
    one = make_group(GroupShape(4, 2, 4, 5, (3,), "f32"), seed=29)
    caught.append(pin_sdpa_n1(one) > 1e-6)
    assert any(caught), f"mutation {mutation} escaped every pin"


def test_sampled_rows_equal_full_oracle_rows():
    """The per-row reference used at full size equals the full oracle's rows."""
    from oracle.attention import sampled_rows_reference
    inp = make_group(GroupShape(4, 2, 16, 20, (5, 9), "f32"), seed=2)
    ref = dense_group_reference(inp)
    smp = sampled_rows_reference(inp, [0, 7, 19], [(0, 0), (1, 8), (1, 3)])
    for r, v in smp["prefix"].items():
        assert np.abs(v["o"] - ref["o_p"][r]).max() < 1e-12
        assert np.abs(v["dq"] - ref["dq_p"][r]).max() < 1e-12
        assert np.abs(v["lse"] - ref["lse_p"][:, r]).max() < 1e-12
    cu = inp["cu_seqlens"]
    for (i, t), v in smp["suffix"].items():
        row = cu[i] + t
        assert np.abs(v["o"] - ref["o_s"][row]).max() < 1e-12
        assert np.abs(v["dq"] - ref["dq_s"][row]).max() < 1e-12
        assert np.abs(v["lse"] - ref["lse_s"][:, row]).max() < 1e-12


@pytest.mark.parametrize("shape,ragged", [
    (GroupShape(4, 2, 16, 20, (5, 9), "f32"), None),
    (GroupShape(8, 2, 8, 70, (3, 1, 40), "bf16"), None),
    (GroupShape(4, 1, 8, 33, (0,) * 3, "bf16"), (1, 9)),
])
def test_sampled_keys_equal_full_oracle_keys(shape, ragged):
    """The per-key reference used at full size equals the full oracle's
    dK/dV rows and cache rows, at prefix keys including the first and last
    and at the first, middle and last key of each suffix."""
    from oracle.attention import sampled_keys_reference
    inp = make_group(shape, seed=5, ragged=ragged)
    shp = inp["shape"]
    ref = dense_group_reference(inp)
    P, lens = shp.prefix_len, shp.suffix_lens
    pk = sorted({0, 1, P // 2, P - 2, P - 1})
    sk = sorted({(i, t) for i in range(shp.n) for t in (0, lens[i] // 2, lens[i] - 1)})
    smp = sampled_keys_reference(inp, pk, sk)
    for j, v in smp["prefix"].items():
        for f, rk in (("dk", "dk_p"), ("dv", "dv_p"), ("g_k", "g_k"), ("g_v", "g_v")):
            assert np.abs(v[f] - ref[rk][j]).max() < 1e-11, (j, f)
    cu = inp["cu_seqlens"]
    for (i, t), v in smp["suffix"].items():
        assert np.abs(v["dk"] - ref["dk_s"][cu[i] + t]).max() < 1e-11, (i, t)
        assert np.abs(v["dv"] - ref["dv_s"][cu[i] + t]).max() < 1e-11, (i, t)


def test_causal_forward_rows_equals_full_oracle_forward():
    """The forward-only row function equals the full oracle's O and LSE, also
    for a row range that starts inside the sequence."""
    from oracle.attention import causal_forward_rows, causal_attention
    rng = np.random.default_rng(3)
    q, k, v, do = (rng.standard_normal((2500, 4, 8)), rng.standard_normal((2500, 2, 8)),
                   rng.standard_normal((2500, 2, 8)), rng.standard_normal((2500, 4, 8)))
    o, lse, *_ = causal_attention(q, k, v, do, 0.3)
    o2, lse2 = causal_forward_rows(q, k, v, 0.3)
    assert np.abs(o - o2).max() < 1e-12 and np.abs(lse - lse2).max() < 1e-12
    o3, lse3 = causal_forward_rows(q[1700:], k, v, 0.3, first_query_pos=1700)
    assert np.abs(o[1700:] - o3).max() < 1e-12 and np.abs(lse[:, 1700:] - lse3).max() < 1e-12
