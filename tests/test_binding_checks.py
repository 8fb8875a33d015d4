"""The binding's size and dtype checks (CPU): a tensor smaller than the dims
require, or of another element type, is refused before any pointer reaches
the library."""
import pytest
import torch

from paper_2606_01143_amd import binding as B


def _prefix_args(dims, P, dt=torch.bfloat16, short=None, wrong_dtype=None):
    hq, hkv, d = dims.num_q_heads, dims.num_kv_heads, dims.head_dim
    shapes = {"q_p": (P, hq, d), "k_p": (P, hkv, d), "v_p": (P, hkv, d), "o_p": (P, hq, d)}
    t = {}
    for k, shp in shapes.items():
        rows = shp[0] - 1 if k == short else shp[0]
        t[k] = torch.zeros((rows,) + shp[1:], dtype=torch.float32 if k == wrong_dtype else dt)
    t["lse_p"] = torch.zeros((P - 1 if short == "lse_p" else P, hq), dtype=torch.float32)
    return t


@pytest.mark.parametrize("short", ["q_p", "k_p", "v_p", "o_p", "lse_p"])
def test_short_tensor_is_refused(short):
    dims = B.make_dims(4, 2, 64, 33, "bf16")
    t = _prefix_args(dims, 33, short=short)
    with pytest.raises(ValueError, match=f"{short}: .* elements, the call needs"):
        B.prefix_fwd(dims, t["q_p"], t["k_p"], t["v_p"], t["o_p"], t["lse_p"])


def test_wrong_element_type_is_refused():
    dims = B.make_dims(4, 2, 64, 33, "bf16")
    t = _prefix_args(dims, 33, wrong_dtype="k_p")
    with pytest.raises(ValueError, match="k_p: elements of 4 bytes, the call needs 2"):
        B.prefix_fwd(dims, t["q_p"], t["k_p"], t["v_p"], t["o_p"], t["lse_p"])


def test_right_sizes_reach_the_device_check():
    dims = B.make_dims(4, 2, 64, 33, "bf16")
    t = _prefix_args(dims, 33)
    with pytest.raises(ValueError, match="GPU tensors only"):
        B.prefix_fwd(dims, t["q_p"], t["k_p"], t["v_p"], t["o_p"], t["lse_p"])


def test_suffix_backward_cache_and_offsets_are_checked():
    dims = B.make_dims(4, 2, 64, 16, "bf16")
    T, n = 10, 2
    bf = lambda *s: torch.zeros(s, dtype=torch.bfloat16)
    f32 = lambda *s: torch.zeros(s, dtype=torch.float32)
    args = dict(k_p=bf(16, 2, 64), v_p=bf(16, 2, 64), q_s=bf(T, 4, 64), k_s=bf(T, 2, 64), v_s=bf(T, 2, 64),
                o_s=bf(T, 4, 64), lse_s=f32(T, 4), do_s=bf(T, 4, 64),
                cu_seqlens=torch.zeros(n + 1, dtype=torch.int32), dq_s=bf(T, 4, 64), dk_s=bf(T, 2, 64),
                dv_s=bf(T, 2, 64), gk_cache=f32(16, 2, 64), gv_cache=f32(16, 2, 64))

    def call(**over):
        a = dict(args, **over)
        B.suffix_attn_bwd_accum(dims, a["k_p"], a["v_p"], a["q_s"], a["k_s"], a["v_s"], a["o_s"], a["lse_s"],
                                a["do_s"], a["cu_seqlens"], n, 6, T, a["dq_s"], a["dk_s"], a["dv_s"],
                                a["gk_cache"], a["gv_cache"])

    with pytest.raises(ValueError, match="gv_cache"):
        call(gv_cache=f32(15, 2, 64))
    with pytest.raises(ValueError, match="gk_cache: elements of 2 bytes"):
        call(gk_cache=bf(16, 2, 64))
    with pytest.raises(ValueError, match="cu_seqlens"):
        call(cu_seqlens=torch.zeros(n, dtype=torch.int32))
    with pytest.raises(ValueError, match="dq_s"):
        call(dq_s=bf(T - 1, 4, 64))
    with pytest.raises(ValueError, match="GPU tensors only"):
        call()


@pytest.mark.parametrize("call,args,bad", [
    ("rmsnorm_fwd", lambda: (torch.zeros(4, 16, dtype=torch.bfloat16), torch.zeros(3, 16, dtype=torch.bfloat16),
                             torch.zeros(4)), "y: 48 elements"),
    ("rmsnorm_fwd", lambda: (torch.zeros(4, 16, dtype=torch.bfloat16), torch.zeros(4, 16, dtype=torch.bfloat16),
                             torch.zeros(3)), "rstd: 3 elements"),
    ("rmsnorm_bwd", lambda: (torch.zeros(4, 16, dtype=torch.bfloat16), torch.zeros(4),
                             torch.zeros(4, 16, dtype=torch.bfloat16), torch.zeros(4, 16)), "dx: elements of 4 bytes"),
    ("rope_fwd", lambda: (torch.zeros(5, 2, 8, dtype=torch.bfloat16), torch.zeros(5, 2, 7, dtype=torch.bfloat16),
                          0, 1e4), "y: 70 elements"),
    ("rope_bwd", lambda: (torch.zeros(5, 2, 8, dtype=torch.bfloat16), torch.zeros(5, 2, 8),
                          0, 1e4), "dx: elements of 4 bytes"),
    ("swiglu_fwd", lambda: (torch.zeros(16, dtype=torch.bfloat16), torch.zeros(16, dtype=torch.bfloat16),
                            torch.zeros(8, dtype=torch.bfloat16)), "m: 8 elements"),
    ("swiglu_bwd", lambda: (torch.zeros(16, dtype=torch.bfloat16), torch.zeros(16, dtype=torch.bfloat16),
                            torch.zeros(16, dtype=torch.bfloat16), torch.zeros(16, dtype=torch.bfloat16),
                            torch.zeros(15, dtype=torch.bfloat16)), "du: 15 elements"),
])
def test_layer_op_wrappers_refuse_short_or_mistyped_tensors(call, args, bad):
    """The decoder-layer op wrappers check element size and count too."""
    with pytest.raises(ValueError, match=bad):
        getattr(B, call)(*args())
