"""ctypes binding of libspr: one Python function per C entry point, same
name without the ``spr_`` prefix, same argument order.  Argument
marshalling only (tensor -> device pointer, stream -> hipStream_t, status ->
exception); every step of the computation runs in the HIP library.

Tensors must be contiguous GPU tensors; ``None`` passes a NULL pointer.
The library must be built (``python -m paper_2606_01143_amd.build``);
loading fails loudly otherwise -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, byref, c_char_p, c_double, c_float, c_int32, c_int64, c_size_t, c_uint32, c_void_p

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "lib", "libspr.so")

SPR_F32 = 0
SPR_BF16 = 1
SPR_DETERMINISTIC = 1
SPR_ATOMIC_DQ = 2

OP_PREFIX_FWD = 0
OP_SUFFIX_FWD = 1
OP_SUFFIX_BWD = 2
OP_PREFIX_BWD = 3
OP_DENSE_BASELINE = 4
OP_SUFFIX_FWD_PADDED = 5
OP_SUFFIX_BWD_PADDED = 6

STATUS = {0: "SPR_OK", 1: "SPR_ERR_INVALID_ARG", 2: "SPR_ERR_UNSUPPORTED",
          3: "SPR_ERR_MISALIGNED", 4: "SPR_ERR_ALIASING", 5: "SPR_ERR_WORKSPACE",
          6: "SPR_ERR_HIP"}

# C symbol -> (argtypes, restype)
_P = c_void_p
_SIGNATURES = {
    "spr_prefix_fwd": ([_P, _P, _P, _P, _P, _P, _P], c_int32),
    "spr_suffix_attn_fwd": ([_P, _P, _P, _P, _P, _P, _P, c_int32, c_int32, c_int32, _P, _P, _P,
                             c_size_t, _P], c_int32),
    "spr_suffix_attn_fwd_noalloc": ([_P, _P, _P, _P, _P, _P, _P, c_int32, c_int32, c_int32, _P, _P,
                                     _P], c_int32),
    "spr_suffix_attn_bwd_accum": ([_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, c_int32, c_int32, c_int32,
                                   _P, _P, _P, _P, _P, _P, c_size_t, _P], c_int32),
    "spr_prefix_bwd": ([_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, c_size_t, _P], c_int32),
    "spr_suffix_attn_fwd_padded": ([_P, _P, _P, _P, _P, _P, _P, c_int32, c_int32, _P, _P, _P, c_size_t, _P],
                                   c_int32),
    "spr_suffix_attn_bwd_accum_padded": ([_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, c_int32, c_int32, _P, _P,
                                          _P, _P, _P, _P, c_size_t, _P], c_int32),
    "spr_prefix_bwd_dq": ([_P, _P, _P, _P, _P, _P, _P, _P, _P, c_size_t, _P], c_int32),
    "spr_prefix_bwd_dkv": ([_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, c_size_t, _P], c_int32),
    "spr_dense_recompute_baseline": ([_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, c_int32, c_int32,
                                      c_int32, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                      c_size_t, _P], c_int32),
    "spr_workspace_size": ([c_int32, _P, c_int32, c_int32, c_int32, POINTER(c_size_t)], c_int32),
    "spr_check_cu_seqlens": ([POINTER(c_int32), c_int32, c_int32, c_int32], c_int32),
    "spr_gkv_cache_zero": ([_P, _P, _P, _P], c_int32),
    "spr_gkv_accumulate": ([_P, _P, _P, _P, _P, _P], c_int32),
    "spr_rmsnorm_fwd": ([c_int32, c_int32, c_float, _P, _P, _P, _P], c_int32),
    "spr_rmsnorm_bwd": ([c_int32, c_int32, _P, _P, _P, _P, _P, _P], c_int32),
    "spr_rope_fwd": ([c_int32, c_int32, c_int32, c_int32, c_double, _P, _P, _P], c_int32),
    "spr_rope_bwd": ([c_int32, c_int32, c_int32, c_int32, c_double, _P, _P, _P], c_int32),
    "spr_swiglu_fwd": ([c_int64, _P, _P, _P, _P], c_int32),
    "spr_swiglu_bwd": ([c_int64, _P, _P, _P, _P, _P, _P], c_int32),
    "spr_moe_stats_bytes": ([c_int32, POINTER(c_size_t)], c_int32),
    "spr_moe_stats_zero": ([c_int32, _P, _P], c_int32),
    "spr_moe_aux_workspace_size": ([c_int32, c_int32, POINTER(c_size_t)], c_int32),
    "spr_moe_aux_accumulate": ([c_int32, c_int32, c_int32, _P, _P, c_int32, _P, _P, _P, c_size_t, _P],
                               c_int32),
    "spr_moe_aux_loss": ([c_int32, c_int32, c_double, _P, _P, _P, _P, _P], c_int32),
    "spr_moe_aux_grad": ([c_int32, c_int32, c_double, c_double, _P, c_int32, c_int32, _P, _P, _P],
                         c_int32),
    "spr_profile_enable": ([c_int32, c_char_p], c_int32),
    "spr_profile_reset": ([], c_int32),
    "spr_profile_query": ([c_char_p, POINTER(c_double), POINTER(c_int32)], c_int32),
    "spr_profile_num_kernels": ([], c_int32),
    "spr_profile_kernel_name": ([c_int32], c_char_p),
    "spr_status_string": ([c_int32], c_char_p),
    "spr_last_error": ([], c_char_p),
    "spr_version": ([], c_char_p),
}


class SprDims(ctypes.Structure):
    """Mirror of ``spr_dims`` in include/spr.h."""
    _fields_ = [("num_q_heads", c_int32), ("num_kv_heads", c_int32), ("head_dim", c_int32),
                ("prefix_len", c_int32), ("softmax_scale", c_float), ("dtype", c_int32),
                ("flags", c_uint32)]


class SprError(RuntimeError):
    def __init__(self, status: int, message: str):
        self.status = status
        self.status_name = STATUS.get(status, f"status {status}")
        super().__init__(f"{self.status_name}: {message}")


_lib = None


def lib() -> ctypes.CDLL:
    """Load libspr.so (once) and declare every entry point's signature."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"libspr.so is not built ({LIB_PATH}); build it with "
                "`python -m paper_2606_01143_amd.build` -- there is no fallback path")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (argtypes, restype) in _SIGNATURES.items():
            fn = getattr(handle, name)
            fn.argtypes = argtypes
            fn.restype = restype
        _lib = handle
    return _lib


def make_dims(num_q_heads: int, num_kv_heads: int, head_dim: int, prefix_len: int,
              dtype: str = "bf16", softmax_scale: float = 0.0,
              deterministic: bool = False, atomic_dq: bool = False) -> SprDims:
    code = {"f32": SPR_F32, "bf16": SPR_BF16}[dtype]
    flags = (SPR_DETERMINISTIC if deterministic else 0) | (SPR_ATOMIC_DQ if atomic_dq else 0)
    return SprDims(num_q_heads, num_kv_heads, head_dim, prefix_len, softmax_scale, code, flags)


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if not x.is_cuda:
        raise ValueError("libspr takes GPU tensors only")
    if not x.is_contiguous():
        raise ValueError("libspr takes contiguous tensors only")
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


class _Sizes:
    """Required sizes of one call's tensors, from the dims and the row counts.

    The C ABI takes plain pointers and cannot see a buffer's size; a tensor
    that is too small, or of another element type than the dims say, would
    be read or written past its end on the GPU.  Every attention wrapper
    therefore checks its tensors here first (None is a NULL pointer and is
    left to the library's own checks)."""

    def __init__(self, dims, rows_s: int = 0):
        self.P, self.hq, self.hkv, self.d = (int(dims.prefix_len), int(dims.num_q_heads),
                                             int(dims.num_kv_heads), int(dims.head_dim))
        self.eb = 4 if dims.dtype == SPR_F32 else 2
        self.T = int(rows_s)

    def _need(self, name, x, elems, esize):
        if x is None or isinstance(x, int):
            return
        if x.element_size() != esize:
            raise ValueError(f"{name}: elements of {x.element_size()} bytes, the call needs {esize}")
        if x.numel() < elems:
            raise ValueError(f"{name}: {x.numel()} elements, the call needs {elems}")

    def q(self, rows, **kw):   # [rows, Hq, d] storage dtype
        for k, v in kw.items():
            self._need(k, v, rows * self.hq * self.d, self.eb)

    def kv(self, rows, **kw):  # [rows, Hkv, d] storage dtype
        for k, v in kw.items():
            self._need(k, v, rows * self.hkv * self.d, self.eb)

    def lse(self, rows, **kw):  # [rows, Hq] fp32
        for k, v in kw.items():
            self._need(k, v, rows * self.hq, 4)

    def cache(self, **kw):     # [P, Hkv, d] fp32
        for k, v in kw.items():
            self._need(k, v, self.P * self.hkv * self.d, 4)

    def i32(self, n, **kw):
        for k, v in kw.items():
            self._need(k, v, n, 4)


def _check(status: int) -> None:
    if status != 0:
        raise SprError(status, lib().spr_last_error().decode())


def check_cu_seqlens(cu_host, n_mb, max_len, total_len) -> None:
    """Host-side check of a microbatch's suffix offsets (the values uploaded
    as cu_seqlens): raises SprError(SPR_ERR_INVALID_ARG) on a zero-length
    suffix or offsets inconsistent with n_mb / max_len / total_len."""
    vals = [int(x) for x in cu_host]
    if len(vals) != int(n_mb) + 1:
        raise SprError(1, f"cu_seqlens has {len(vals)} entries, n_mb + 1 = {int(n_mb) + 1} expected")
    arr = (c_int32 * len(vals))(*vals)
    _check(lib().spr_check_cu_seqlens(arr, n_mb, max_len, total_len))


def _nbytes(ws) -> int:
    return 0 if ws is None else ws.numel() * ws.element_size()


# ------------------------------------------------------------ entry points
def prefix_fwd(dims, q_p, k_p, v_p, o_p, lse_p, stream=None):
    z = _Sizes(dims)
    z.q(z.P, q_p=q_p, o_p=o_p)
    z.kv(z.P, k_p=k_p, v_p=v_p)
    z.lse(z.P, lse_p=lse_p)
    _check(lib().spr_prefix_fwd(byref(dims), _ptr(q_p), _ptr(k_p), _ptr(v_p), _ptr(o_p),
                                _ptr(lse_p), _stream(stream)))


def suffix_attn_fwd(dims, k_p, v_p, q_s, k_s, v_s, cu_seqlens, n_mb, max_len, total_len, o_s,
                    lse_s, ws=None, stream=None, cu_host=None):
    """``cu_host``: the host copy of cu_seqlens, checked first when given."""
    if cu_host is not None:
        check_cu_seqlens(cu_host, n_mb, max_len, total_len)
    z = _Sizes(dims, total_len)
    z.kv(z.P, k_p=k_p, v_p=v_p)
    z.q(z.T, q_s=q_s, o_s=o_s)
    z.kv(z.T, k_s=k_s, v_s=v_s)
    z.lse(z.T, lse_s=lse_s)
    z.i32(int(n_mb) + 1, cu_seqlens=cu_seqlens)
    _check(lib().spr_suffix_attn_fwd(byref(dims), _ptr(k_p), _ptr(v_p), _ptr(q_s), _ptr(k_s),
                                     _ptr(v_s), _ptr(cu_seqlens), n_mb, max_len, total_len,
                                     _ptr(o_s), _ptr(lse_s), _ptr(ws), _nbytes(ws),
                                     _stream(stream)))


# bytes of the static device scratch behind suffix_attn_fwd_noalloc
STATIC_SCRATCH_BYTES = 64 << 20


def suffix_attn_fwd_noalloc(dims, k_p, v_p, q_s, k_s, v_s, cu_seqlens, n_mb, max_len, total_len,
                            o_s, lse_s, stream=None, cu_host=None):
    """suffix_attn_fwd with the library's static scratch as its workspace:
    no device allocation anywhere (callers under graph capture, serving
    loops).  Calls that overlap on one GPU race on the scratch."""
    if cu_host is not None:
        check_cu_seqlens(cu_host, n_mb, max_len, total_len)
    z = _Sizes(dims, total_len)
    z.kv(z.P, k_p=k_p, v_p=v_p)
    z.q(z.T, q_s=q_s, o_s=o_s)
    z.kv(z.T, k_s=k_s, v_s=v_s)
    z.lse(z.T, lse_s=lse_s)
    z.i32(int(n_mb) + 1, cu_seqlens=cu_seqlens)
    _check(lib().spr_suffix_attn_fwd_noalloc(byref(dims), _ptr(k_p), _ptr(v_p), _ptr(q_s), _ptr(k_s),
                                             _ptr(v_s), _ptr(cu_seqlens), n_mb, max_len, total_len,
                                             _ptr(o_s), _ptr(lse_s), _stream(stream)))


def suffix_attn_bwd_accum(dims, k_p, v_p, q_s, k_s, v_s, o_s, lse_s, do_s, cu_seqlens, n_mb,
                          max_len, total_len, dq_s, dk_s, dv_s, gk_cache, gv_cache, ws=None,
                          stream=None, cu_host=None):
    """``cu_host``: the host copy of cu_seqlens, checked first when given."""
    if cu_host is not None:
        check_cu_seqlens(cu_host, n_mb, max_len, total_len)
    z = _Sizes(dims, total_len)
    z.kv(z.P, k_p=k_p, v_p=v_p)
    z.q(z.T, q_s=q_s, o_s=o_s, do_s=do_s, dq_s=dq_s)
    z.kv(z.T, k_s=k_s, v_s=v_s, dk_s=dk_s, dv_s=dv_s)
    z.lse(z.T, lse_s=lse_s)
    z.cache(gk_cache=gk_cache, gv_cache=gv_cache)
    z.i32(int(n_mb) + 1, cu_seqlens=cu_seqlens)
    _check(lib().spr_suffix_attn_bwd_accum(
        byref(dims), _ptr(k_p), _ptr(v_p), _ptr(q_s), _ptr(k_s), _ptr(v_s), _ptr(o_s),
        _ptr(lse_s), _ptr(do_s), _ptr(cu_seqlens), n_mb, max_len, total_len, _ptr(dq_s),
        _ptr(dk_s), _ptr(dv_s), _ptr(gk_cache), _ptr(gv_cache), _ptr(ws), _nbytes(ws),
        _stream(stream)))


def prefix_bwd(dims, q_p, k_p, v_p, o_p, lse_p, do_p, gk_cache, gv_cache, dq_p, dk_p, dv_p,
               ws=None, stream=None):
    z = _Sizes(dims)
    z.q(z.P, q_p=q_p, o_p=o_p, do_p=do_p, dq_p=dq_p)
    z.kv(z.P, k_p=k_p, v_p=v_p, dk_p=dk_p, dv_p=dv_p)
    z.lse(z.P, lse_p=lse_p)
    z.cache(gk_cache=gk_cache, gv_cache=gv_cache)
    _check(lib().spr_prefix_bwd(byref(dims), _ptr(q_p), _ptr(k_p), _ptr(v_p), _ptr(o_p),
                                _ptr(lse_p), _ptr(do_p), _ptr(gk_cache), _ptr(gv_cache),
                                _ptr(dq_p), _ptr(dk_p), _ptr(dv_p), _ptr(ws), _nbytes(ws),
                                _stream(stream)))


def suffix_attn_fwd_padded(dims, k_p, v_p, q_s, k_s, v_s, seq_lens, n, s_max, o_s, lse_s, ws=None,
                           stream=None):
    z = _Sizes(dims, int(n) * int(s_max))
    z.kv(z.P, k_p=k_p, v_p=v_p)
    z.q(z.T, q_s=q_s, o_s=o_s)
    z.kv(z.T, k_s=k_s, v_s=v_s)
    z.lse(z.T, lse_s=lse_s)
    z.i32(int(n), seq_lens=seq_lens)
    _check(lib().spr_suffix_attn_fwd_padded(byref(dims), _ptr(k_p), _ptr(v_p), _ptr(q_s), _ptr(k_s),
                                            _ptr(v_s), _ptr(seq_lens), n, s_max, _ptr(o_s), _ptr(lse_s),
                                            _ptr(ws), _nbytes(ws), _stream(stream)))


def suffix_attn_bwd_accum_padded(dims, k_p, v_p, q_s, k_s, v_s, o_s, lse_s, do_s, seq_lens, n, s_max,
                                 dq_s, dk_s, dv_s, gk_cache, gv_cache, ws=None, stream=None):
    z = _Sizes(dims, int(n) * int(s_max))
    z.kv(z.P, k_p=k_p, v_p=v_p)
    z.q(z.T, q_s=q_s, o_s=o_s, do_s=do_s, dq_s=dq_s)
    z.kv(z.T, k_s=k_s, v_s=v_s, dk_s=dk_s, dv_s=dv_s)
    z.lse(z.T, lse_s=lse_s)
    z.cache(gk_cache=gk_cache, gv_cache=gv_cache)
    z.i32(int(n), seq_lens=seq_lens)
    _check(lib().spr_suffix_attn_bwd_accum_padded(
        byref(dims), _ptr(k_p), _ptr(v_p), _ptr(q_s), _ptr(k_s), _ptr(v_s), _ptr(o_s), _ptr(lse_s),
        _ptr(do_s), _ptr(seq_lens), n, s_max, _ptr(dq_s), _ptr(dk_s), _ptr(dv_s), _ptr(gk_cache),
        _ptr(gv_cache), _ptr(ws), _nbytes(ws), _stream(stream)))


def prefix_bwd_dq(dims, q_p, k_p, v_p, o_p, lse_p, do_p, dq_p, ws=None, stream=None):
    z = _Sizes(dims)
    z.q(z.P, q_p=q_p, o_p=o_p, do_p=do_p, dq_p=dq_p)
    z.kv(z.P, k_p=k_p, v_p=v_p)
    z.lse(z.P, lse_p=lse_p)
    _check(lib().spr_prefix_bwd_dq(byref(dims), _ptr(q_p), _ptr(k_p), _ptr(v_p), _ptr(o_p),
                                   _ptr(lse_p), _ptr(do_p), _ptr(dq_p), _ptr(ws), _nbytes(ws),
                                   _stream(stream)))


def prefix_bwd_dkv(dims, q_p, k_p, v_p, o_p, lse_p, do_p, gk_cache, gv_cache, dk_p, dv_p,
                   ws=None, stream=None):
    z = _Sizes(dims)
    z.q(z.P, q_p=q_p, o_p=o_p, do_p=do_p)
    z.kv(z.P, k_p=k_p, v_p=v_p, dk_p=dk_p, dv_p=dv_p)
    z.lse(z.P, lse_p=lse_p)
    z.cache(gk_cache=gk_cache, gv_cache=gv_cache)
    _check(lib().spr_prefix_bwd_dkv(byref(dims), _ptr(q_p), _ptr(k_p), _ptr(v_p), _ptr(o_p),
                                    _ptr(lse_p), _ptr(do_p), _ptr(gk_cache), _ptr(gv_cache),
                                    _ptr(dk_p), _ptr(dv_p), _ptr(ws), _nbytes(ws),
                                    _stream(stream)))


def dense_recompute_baseline(dims, q_p, k_p, v_p, do_p_seq, q_s, k_s, v_s, do_s, cu_seqlens, n,
                             max_len, total_len, o_p, lse_p, o_s, lse_s, dq_s, dk_s, dv_s, dq_p,
                             dk_p, dv_p, ws=None, stream=None, cu_host=None):
    """``cu_host``: the host copy of cu_seqlens, checked first when given."""
    if cu_host is not None:
        check_cu_seqlens(cu_host, n, max_len, total_len)
    z = _Sizes(dims, total_len)
    z.q(z.P, q_p=q_p, o_p=o_p, dq_p=dq_p)
    z.q(int(n) * z.P, do_p_seq=do_p_seq)
    z.kv(z.P, k_p=k_p, v_p=v_p, dk_p=dk_p, dv_p=dv_p)
    z.lse(z.P, lse_p=lse_p)
    z.q(z.T, q_s=q_s, o_s=o_s, do_s=do_s, dq_s=dq_s)
    z.kv(z.T, k_s=k_s, v_s=v_s, dk_s=dk_s, dv_s=dv_s)
    z.lse(z.T, lse_s=lse_s)
    z.i32(int(n) + 1, cu_seqlens=cu_seqlens)
    _check(lib().spr_dense_recompute_baseline(
        byref(dims), _ptr(q_p), _ptr(k_p), _ptr(v_p), _ptr(do_p_seq), _ptr(q_s), _ptr(k_s),
        _ptr(v_s), _ptr(do_s), _ptr(cu_seqlens), n, max_len, total_len, _ptr(o_p), _ptr(lse_p),
        _ptr(o_s), _ptr(lse_s), _ptr(dq_s), _ptr(dk_s), _ptr(dv_s), _ptr(dq_p), _ptr(dk_p),
        _ptr(dv_p), _ptr(ws), _nbytes(ws), _stream(stream)))


def _need_all(elems, esize, **tensors):
    """Every named tensor holds at least `elems` elements of `esize` bytes
    (None: a NULL pointer, left to the library)."""
    for name, x in tensors.items():
        if x is None:
            continue
        if x.element_size() != esize:
            raise ValueError(f"{name}: elements of {x.element_size()} bytes, the call needs {esize}")
        if x.numel() < elems:
            raise ValueError(f"{name}: {x.numel()} elements, the call needs {elems}")


def rmsnorm_fwd(x, y, rstd, eps=1e-5, stream=None):
    rows, width = int(x.shape[0]), int(x.shape[-1])
    _need_all(rows * width, 2, x=x, y=y)
    _need_all(rows, 4, rstd=rstd)
    _check(lib().spr_rmsnorm_fwd(rows, width, eps, _ptr(x), _ptr(y), _ptr(rstd), _stream(stream)))


def rmsnorm_bwd(x, rstd, dy, dx, add=None, stream=None):
    rows, width = int(x.shape[0]), int(x.shape[-1])
    _need_all(rows * width, 2, x=x, dy=dy, dx=dx, add=add)
    _need_all(rows, 4, rstd=rstd)
    _check(lib().spr_rmsnorm_bwd(rows, width, _ptr(x), _ptr(rstd), _ptr(dy), _ptr(add), _ptr(dx),
                                 _stream(stream)))


def rope_fwd(x, y, pos0, theta, stream=None):
    t, h, d = (int(v) for v in x.shape)
    _need_all(t * h * d, 2, x=x, y=y)
    _check(lib().spr_rope_fwd(t, h, d, pos0, float(theta), _ptr(x), _ptr(y), _stream(stream)))


def rope_bwd(dy, dx, pos0, theta, stream=None):
    t, h, d = (int(v) for v in dy.shape)
    _need_all(t * h * d, 2, dy=dy, dx=dx)
    _check(lib().spr_rope_bwd(t, h, d, pos0, float(theta), _ptr(dy), _ptr(dx), _stream(stream)))


def swiglu_fwd(g, u, m, stream=None):
    n = int(g.numel())
    _need_all(n, 2, g=g, u=u, m=m)
    _check(lib().spr_swiglu_fwd(n, _ptr(g), _ptr(u), _ptr(m), _stream(stream)))


def swiglu_bwd(g, u, dm, dg, du, stream=None):
    n = int(g.numel())
    _need_all(n, 2, g=g, u=u, dm=dm, dg=dg, du=du)
    _check(lib().spr_swiglu_bwd(n, _ptr(g), _ptr(u), _ptr(dm), _ptr(dg), _ptr(du),
                                _stream(stream)))


def moe_stats_bytes(n_experts: int) -> int:
    out = c_size_t(0)
    _check(lib().spr_moe_stats_bytes(n_experts, byref(out)))
    return int(out.value)


def moe_stats_zero(n_experts, stats, stream=None):
    _check(lib().spr_moe_stats_zero(n_experts, _ptr(stats), _stream(stream)))


def moe_aux_workspace_size(n_experts: int, n_tokens: int) -> int:
    out = c_size_t(0)
    _check(lib().spr_moe_aux_workspace_size(n_experts, n_tokens, byref(out)))
    return int(out.value)


def moe_aux_accumulate(n_experts, top_k, probs, experts, stats, multiplicity=1,
                       token_multiplicity=None, ws=None, stream=None):
    n = int(probs.shape[0]) if probs is not None else 0
    _check(lib().spr_moe_aux_accumulate(n_experts, top_k, n, _ptr(probs), _ptr(experts),
                                        multiplicity, _ptr(token_multiplicity), _ptr(stats),
                                        _ptr(ws), _nbytes(ws), _stream(stream)))


def moe_aux_loss(n_experts, top_k, aux_coef, stats, f, p, loss, stream=None):
    _check(lib().spr_moe_aux_loss(n_experts, top_k, float(aux_coef), _ptr(stats), _ptr(f), _ptr(p),
                                  _ptr(loss), _stream(stream)))


def moe_aux_grad(n_experts, top_k, aux_coef, upstream, stats, dprobs, multiplicity=1,
                 token_multiplicity=None, stream=None):
    n = int(dprobs.shape[0])
    _check(lib().spr_moe_aux_grad(n_experts, top_k, float(aux_coef), float(upstream), _ptr(stats), n,
                                  multiplicity, _ptr(token_multiplicity), _ptr(dprobs),
                                  _stream(stream)))


def workspace_size(op, dims, n_mb=0, max_len=0, total_len=0) -> int:
    out = c_size_t(0)
    _check(lib().spr_workspace_size(op, byref(dims), n_mb, max_len, total_len, byref(out)))
    return int(out.value)


def gkv_cache_zero(dims, gk_cache, gv_cache, stream=None):
    _Sizes(dims).cache(gk_cache=gk_cache, gv_cache=gv_cache)
    _check(lib().spr_gkv_cache_zero(byref(dims), _ptr(gk_cache), _ptr(gv_cache), _stream(stream)))


def gkv_accumulate(dims, gk_cache, gv_cache, dgk, dgv, stream=None):
    _Sizes(dims).cache(gk_cache=gk_cache, gv_cache=gv_cache, dgk=dgk, dgv=dgv)
    _check(lib().spr_gkv_accumulate(byref(dims), _ptr(gk_cache), _ptr(gv_cache), _ptr(dgk),
                                    _ptr(dgv), _stream(stream)))


def profile_enable(on: bool = True, only_kernel: str = None):
    _check(lib().spr_profile_enable(1 if on else 0,
                                    only_kernel.encode() if only_kernel else None))


def profile_reset():
    _check(lib().spr_profile_reset())


def profile_query(kernel: str):
    ms, cnt = c_double(0.0), c_int32(0)
    _check(lib().spr_profile_query(kernel.encode(), byref(ms), byref(cnt)))
    return float(ms.value), int(cnt.value)


def profile_kernels():
    n = lib().spr_profile_num_kernels()
    return [lib().spr_profile_kernel_name(i).decode() for i in range(n)]


def status_string(status: int) -> str:
    return lib().spr_status_string(status).decode()


def last_error() -> str:
    return lib().spr_last_error().decode()


def version() -> str:
    return lib().spr_version().decode()
