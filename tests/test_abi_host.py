"""CPU tier for the C ABI: the library loads, exports every symbol the header
declares, and rejects bad arguments before launching anything.

No call here reaches a kernel launch: each one fails validation first, and
the fake device pointers are only compared, never dereferenced.
"""
import ctypes
import os
import re

import pytest

from paper_2606_01143_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "spr.h")
HEADERS = sorted(os.path.join(ROOT, "include", f) for f in os.listdir(os.path.join(ROOT, "include"))
                 if f.endswith(".h"))


def header_symbols():
    syms = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        syms.update(re.findall(r"\b(spr_[a-z_0-9]+)\s*\(", text))
    return sorted(syms)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        pytest.fail("libspr.so is not built: run `python -m paper_2606_01143_amd.build`")
    return B.lib()


def test_every_header_symbol_is_exported_and_bound(lib):
    syms = header_symbols()
    assert len(syms) >= 15
    for s in syms:
        assert hasattr(lib, s), s
        assert s in B._SIGNATURES, f"{s} has no Python binding"


def test_dims_struct_matches_header():
    text = open(HEADER).read()
    body = re.search(r"typedef struct spr_dims \{(.*?)\} spr_dims;", text, re.S).group(1)
    fields = re.findall(r"\b(?:int32_t|float|uint32_t)\s+(\w+);", body)
    assert fields == [f for f, _ in B.SprDims._fields_]
    assert ctypes.sizeof(B.SprDims) == 28


def test_version_and_status_strings(lib):
    assert "spr" in B.version()
    for code, name in B.STATUS.items():
        assert B.status_string(code) == name


A = 0x7F0000000000  # fake, 16-byte aligned device addresses (never dereferenced)


def _addr(i):
    return A + i * (1 << 30)


def _dims(**kw):
    base = dict(num_q_heads=4, num_kv_heads=2, head_dim=128, prefix_len=64, dtype="bf16")
    base.update(kw)
    return B.make_dims(**base)


def _call_prefix_fwd(dims, q=1, k=2, v=3, o=4, lse=5):
    args = [_addr(x) if x else None for x in (q, k, v, o, lse)]
    return B.lib().spr_prefix_fwd(ctypes.byref(dims), *args, None)


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=96), "SPR_ERR_UNSUPPORTED"),
    (dict(num_q_heads=6, num_kv_heads=4), "SPR_ERR_INVALID_ARG"),
    (dict(num_kv_heads=0), "SPR_ERR_INVALID_ARG"),
    (dict(prefix_len=-1), "SPR_ERR_INVALID_ARG"),
    (dict(softmax_scale=float("inf")), "SPR_ERR_INVALID_ARG"),
])
def test_dims_validation(lib, kw, status):
    assert B.STATUS[_call_prefix_fwd(_dims(**kw))] == status
    assert B.last_error()


def test_unknown_dtype_and_flags(lib):
    d = _dims()
    d.dtype = 7
    assert B.STATUS[_call_prefix_fwd(d)] == "SPR_ERR_UNSUPPORTED"
    d = _dims()
    d.flags = 0x80
    assert B.STATUS[_call_prefix_fwd(d)] == "SPR_ERR_UNSUPPORTED"


def test_null_and_misaligned_pointers(lib):
    assert B.STATUS[_call_prefix_fwd(_dims(), q=0)] == "SPR_ERR_INVALID_ARG"
    d = _dims()
    r = B.lib().spr_prefix_fwd(ctypes.byref(d), _addr(1) + 8, _addr(2), _addr(3), _addr(4),
                               _addr(5), None)
    assert B.STATUS[r] == "SPR_ERR_MISALIGNED"


def _bwd_accum(dims, n_mb=2, max_len=10, total=15, gk=None, ws_bytes=1 << 40, ws=100):
    ptr = [_addr(i) for i in range(1, 14)]
    gk_ptr = gk if gk is not None else _addr(20)
    return B.lib().spr_suffix_attn_bwd_accum(
        ctypes.byref(dims), ptr[0], ptr[1], ptr[2], ptr[3], ptr[4], ptr[5], ptr[6], ptr[7],
        ptr[8], n_mb, max_len, total, ptr[9], ptr[10], ptr[11], gk_ptr, _addr(21),
        _addr(ws) if ws else None, ws_bytes, None)


@pytest.mark.parametrize("n_mb,max_len,total", [(0, 4, 4), (2, 0, 4), (3, 4, 2), (2, 4, 9)])
def test_suffix_size_validation(lib, n_mb, max_len, total):
    assert B.STATUS[_bwd_accum(_dims(), n_mb, max_len, total)] == "SPR_ERR_INVALID_ARG"


def test_cache_aliasing_is_rejected(lib):
    # gk_cache placed inside q_s (argument 3)
    assert B.STATUS[_bwd_accum(_dims(), gk=_addr(3) + 256)] == "SPR_ERR_ALIASING"


def test_workspace_checks(lib):
    dims = _dims()
    need = B.workspace_size(B.OP_SUFFIX_BWD, dims, 2, 10, 15)
    assert need >= 15 * 4 * 4           # bf16: the row statistic only
    need32 = B.workspace_size(B.OP_SUFFIX_BWD, _dims(dtype="f32"), 2, 10, 15)
    assert need32 >= 15 * 4 * 128 * 4   # fp32 also accumulates dQ
    assert B.STATUS[_bwd_accum(dims, ws_bytes=need - 1)] == "SPR_ERR_WORKSPACE"
    assert B.STATUS[_bwd_accum(dims, ws=0)] == "SPR_ERR_WORKSPACE"


def test_workspace_sizes_are_consistent(lib):
    dims = _dims(prefix_len=4096, num_q_heads=32, num_kv_heads=8)
    assert B.workspace_size(B.OP_PREFIX_FWD, dims) == 0
    assert B.workspace_size(B.OP_PREFIX_BWD, dims) >= 4096 * 32 * 4
    assert B.workspace_size(B.OP_PREFIX_BWD, _dims(prefix_len=4096, num_q_heads=32, num_kv_heads=8,
                                                   dtype="f32")) >= 4096 * 32 * 128 * 4
    dense = B.workspace_size(B.OP_DENSE_BASELINE, dims, 8, 512, 4096)
    assert dense >= 4096 * 32 * 128 * 4 + 4096 * 8 * 128 * 4 * 2
    with pytest.raises(B.SprError):
        B.workspace_size(99, dims)


# ---------------------------------------------------------------- MoE accounting
def _moe_status(fn, *args):
    return getattr(B.lib(), fn)(*args)


@pytest.mark.parametrize("E,k,status", [(128, 8, "SPR_OK"), (6, 1, "SPR_ERR_UNSUPPORTED"),
                                        (2048, 8, "SPR_ERR_UNSUPPORTED"), (0, 1, "SPR_ERR_UNSUPPORTED"),
                                        (16, 0, "SPR_ERR_INVALID_ARG"), (16, 17, "SPR_ERR_INVALID_ARG")])
def test_moe_shape_validation(lib, E, k, status):
    st = lib.spr_moe_aux_loss(E, k, 0.01, _addr(1), None, None, _addr(2) if status != "SPR_OK" else None,
                              None)
    if status == "SPR_OK":
        # valid shape: the null loss pointer is what gets rejected, before any launch
        assert B.STATUS[st] == "SPR_ERR_INVALID_ARG"
    else:
        assert B.STATUS[st] == status


def test_moe_sizes(lib):
    assert B.moe_stats_bytes(128) == 16 * 128 + 16
    assert B.moe_aux_workspace_size(128, 0) == 0
    a, b = B.moe_aux_workspace_size(128, 100), B.moe_aux_workspace_size(128, 100000)
    assert 0 < a < b and b == 2048 * (128 * 16 + 16)


def test_moe_accumulate_checks(lib):
    f = lib.spr_moe_aux_accumulate
    ws = _addr(9)
    # null probs, misaligned probs, negative multiplicity, small workspace, aliasing stats
    assert B.STATUS[f(16, 2, 10, None, _addr(2), 1, None, _addr(3), ws, 1 << 20, None)] == "SPR_ERR_INVALID_ARG"
    assert B.STATUS[f(16, 2, 10, _addr(1) + 4, _addr(2), 1, None, _addr(3), ws, 1 << 20, None)] == \
        "SPR_ERR_MISALIGNED"
    assert B.STATUS[f(16, 2, 10, _addr(1), _addr(2), -1, None, _addr(3), ws, 1 << 20, None)] == \
        "SPR_ERR_INVALID_ARG"
    assert B.STATUS[f(16, 2, 10, _addr(1), _addr(2), 1, None, _addr(3), ws, 8, None)] == "SPR_ERR_WORKSPACE"
    assert B.STATUS[f(16, 2, 10, _addr(1), _addr(2), 1, None, _addr(1), ws, 1 << 20, None)] == \
        "SPR_ERR_ALIASING"
    # zero tokens: nothing to do, no launch
    assert B.STATUS[f(16, 2, 0, None, None, 1, None, _addr(3), None, 0, None)] == "SPR_OK"


# ------------------------------------------------------ padded suffix layout
def _fwd_padded(dims, n=2, s_max=10, lens=7, out=8, ws=20, ws_bytes=1 << 40):
    args = [_addr(1), _addr(2), _addr(3), _addr(4), _addr(5)]
    return B.lib().spr_suffix_attn_fwd_padded(ctypes.byref(dims), *args, _addr(lens) if lens else None, n, s_max,
                                              _addr(out), _addr(9), _addr(ws) if ws else None, ws_bytes, None)


def test_padded_validation(lib):
    dims = _dims()
    need = B.workspace_size(B.OP_SUFFIX_FWD_PADDED, dims, 2, 10)
    assert B.STATUS[_fwd_padded(dims, n=0)] == "SPR_ERR_INVALID_ARG"
    assert B.STATUS[_fwd_padded(dims, s_max=0)] == "SPR_ERR_INVALID_ARG"
    assert B.STATUS[_fwd_padded(dims, lens=None)] == "SPR_ERR_INVALID_ARG"
    assert B.STATUS[_fwd_padded(dims, ws_bytes=need - 1)] == "SPR_ERR_WORKSPACE"
    assert B.STATUS[_fwd_padded(dims, out=3)] == "SPR_ERR_ALIASING"  # o_s on q_s
    assert B.STATUS[_fwd_padded(dims, ws=1)] == "SPR_ERR_ALIASING"   # workspace on k_p


def test_padded_workspace_holds_packed_copies_and_inner_workspace(lib):
    dims = _dims(prefix_len=4096, num_q_heads=32, num_kv_heads=8)
    n, s = 8, 512
    fwd = B.workspace_size(B.OP_SUFFIX_FWD_PADDED, dims, n, s)
    bwd = B.workspace_size(B.OP_SUFFIX_BWD_PADDED, dims, n, s)
    rows = n * s
    assert fwd >= B.workspace_size(B.OP_SUFFIX_FWD, dims, n, s, rows) + rows * (2 * 32 + 2 * 8) * 128 * 2
    assert bwd >= B.workspace_size(B.OP_SUFFIX_BWD, dims, n, s, rows) + rows * (4 * 32 + 4 * 8) * 128 * 2


@pytest.mark.parametrize("cu,n,mx,tot,ok", [
    ([0, 3, 5], 2, 3, 5, True),
    ([0, 3, 3, 5], 3, 3, 5, False),     # a zero-length suffix
    ([0, 3, 2, 5], 3, 3, 5, False),     # decreasing offsets
    ([1, 3, 5], 2, 2, 5, False),        # cu[0] != 0
    ([0, 3, 6], 2, 3, 5, False),        # cu[n] != total_len
    ([0, 4, 5], 2, 3, 5, False),        # a suffix longer than max_len
    ([0, 2, 4], 2, 3, 4, False),        # max_len is not the longest suffix
    ([0, 1], 1, 1, 1, True),
])
def test_check_cu_seqlens(lib, cu, n, mx, tot, ok):
    """The host-side offset check: a zero-length suffix and offsets that
    disagree with n / max_len / total_len are INVALID_ARG, nothing else."""
    if ok:
        B.check_cu_seqlens(cu, n, mx, tot)
    else:
        with pytest.raises(B.SprError) as e:
            B.check_cu_seqlens(cu, n, mx, tot)
        assert e.value.status_name == "SPR_ERR_INVALID_ARG"


def test_suffix_calls_check_host_offsets_before_launching(lib):
    """With the host offsets given, a zero-length suffix is rejected before
    the binding reaches the library's launch path (fake pointers)."""
    with pytest.raises(B.SprError) as e:
        B.suffix_attn_fwd(_dims(), _addr(1), _addr(2), _addr(3), _addr(4), _addr(5), _addr(6),
                          2, 4, 4, _addr(7), _addr(8), cu_host=[0, 4, 4])
    assert e.value.status_name == "SPR_ERR_INVALID_ARG"
    assert "length 0" in str(e.value)


def test_atomic_dq_and_deterministic_flags_conflict(lib):
    """SPR_ATOMIC_DQ with SPR_DETERMINISTIC is contradictory: INVALID_ARG
    before anything is launched; either alone passes the dims check."""
    d = _dims()
    d.flags = B.SPR_ATOMIC_DQ | B.SPR_DETERMINISTIC
    assert B.status_string(_call_prefix_fwd(d)) == "SPR_ERR_INVALID_ARG"
    assert "SPR_ATOMIC_DQ" in B.last_error()
    for f in (B.SPR_ATOMIC_DQ, B.SPR_DETERMINISTIC):
        d.flags = f
        out = ctypes.c_size_t(0)
        assert B.lib().spr_workspace_size(B.OP_PREFIX_BWD, ctypes.byref(d), 0, 0, 0, ctypes.byref(out)) == 0
