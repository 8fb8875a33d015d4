"""The key-outer row-share rule, pinned on the CPU through the workspace
sizes the library reports: a backward launch that splits its key tiles'
row sweeps into R shares reserves R * (P + T) * Hkv * d fp32 partials for
dK and for dV.  The rule is restated here from its description (work in
(32-row tile, q head) steps of 64-key tiles; by default the query-outer
role adds 3/4, with SPR_ATOMIC_DQ there is no such role; two slots
per CU on 256 CUs; split when the longest sweep exceeds the average per slot
by over 10%, R = ceil(longest / average), 1 <= R <= 8, each share >= 16
steps) and compared with the library's choice.  The atomic mode also
reserves the fp32 dQ accumulator of the launch's rows and never splits the
query-outer keys (it has no query-outer role).  A backward launch whose key-outer work, counted in
steps of 192-key tiles over all kv heads, reaches 32768 (128 per CU) runs,
in the default mode, the key-outer role alone with 192-key tiles (six wave
pairs per workgroup, one workgroup per CU): its steps are counted over
192-key tiles, on 256 slots, and no query-outer work is added.  The same
rule serves the prefix backward and the suffix backward (the packed dense
baseline's whole trajectories among them); a suffix backward with a prefix
also needs its prefix key tiles, one workgroup each, to fill their rounds of
256 to at least 85%."""
import math

import pytest

from paper_2606_01143_amd import binding as B


def _tiles(n, b):
    return 0 if n <= 0 else (n + b - 1) // b


def _causal(length, g, bk=64):
    return sum(g * ((length - k0 + 31) // 32) for k0 in range(0, length, bk))


def _rule(kv_steps, max_steps, atomic, slots=512):
    if kv_steps <= 0 or max_steps <= 0:
        return 1
    per_slot = (1.0 if atomic else 1.75) * kv_steps / slots
    if max_steps <= 1.1 * per_slot:
        return 1
    return max(1, min(math.ceil(max_steps / per_slot), max_steps // 16, 8))


def _wide(steps, hkv, atomic):
    """the key-outer role alone on 192-key tiles"""
    return not atomic and steps * hkv >= 32768


def _suffix_r(hq, hkv, P, n, ml, atomic):
    g, rows = hq // hkv, n * ml
    crit = g * ((rows + 31) // 32) if P > 0 else g * ((ml + 31) // 32)
    wide = _tiles(P, 192) * g * ((rows + 31) // 32) + n * _causal(ml, g, 192)
    nt = _tiles(P, 192) * hkv  # equally long prefix sweeps, rounds of 256
    full = P == 0 or nt * 100 >= 85 * 256 * ((nt + 255) // 256)
    if _wide(wide, hkv, atomic) and full:
        return _rule(wide * hkv, crit, True, slots=256)
    kv = _tiles(P, 64) * g * ((rows + 31) // 32) + n * _causal(ml, g)
    return _rule(kv * hkv, crit, atomic)


def _prefix_r(hq, hkv, P, atomic):
    g = hq // hkv
    if _wide(_causal(P, g, 192), hkv, atomic):
        return _rule(_causal(P, g, 192) * hkv, g * ((P + 31) // 32), True, slots=256)
    return _rule(_causal(P, g) * hkv, g * ((P + 31) // 32), atomic)


def _qsplit(hq, P, n, ml):
    """key splits of the query-outer role (fill two slots per CU, at least
    16 key tiles per split, at most 8 splits)"""
    nrb = _tiles(ml, 128) * hq * n
    if nrb <= 0 or nrb >= 512:
        return 1
    nkt = _tiles(P, 64) + _tiles(ml, 64)
    return max(1, min(nkt // 16, (512 + nrb - 1) // nrb, 8))


def _align(x):
    return (x + 255) // 256 * 256


def _suffix_ws(hq, hkv, d, P, n, ml, T, atomic):
    off = _align(hq * T * 4) + _align(hq * T * 4)  # row statistic, log2 LSE
    if atomic:
        off += _align(T * hq * d * 4)  # fp32 dQ accumulator
    else:
        ns = _qsplit(hq, P, n, ml)
        if ns > 1:
            off += _align(ns * T * hq * d * 4)
    r = _suffix_r(hq, hkv, P, n, ml, atomic)
    if r > 1:
        off += 2 * _align(r * (P + T) * hkv * d * 4)
    return off, r


def _prefix_ws(hq, hkv, d, P, atomic):
    off = _align(hq * P * 4) * 2
    if atomic:
        off += _align(P * hq * d * 4)
    r = _prefix_r(hq, hkv, P, atomic)
    if r > 1:
        off += 2 * _align(r * P * hkv * d * 4)
    return off, r


CASES = [
    # (Hq, Hkv, d, P, n_mb, max_len, total)
    (32, 8, 128, 4096, 1, 512, 512),     # bench workload, one suffix: no split in Phase B
    (32, 8, 128, 2048, 1, 1024, 1024),   # Qwen3-8B sweep, P = 2048
    (4, 1, 128, 2048, 1, 700, 700),      # one kv head: 5 shares
    (4, 1, 128, 2048, 1, 333, 333),      # 2 shares
    (8, 1, 128, 1024, 1, 300, 300),
    (4, 2, 64, 1536, 3, 400, 747),       # ragged microbatch of three
    (4, 1, 128, 16384, 1, 1024, 1024),
    (4, 1, 128, 131072, 2, 1000, 1037),
    (4, 1, 128, 0, 2, 16500, 32900),     # long whole sequences, no prefix (packed dense)
    (32, 8, 128, 0, 8, 28800, 230400),   # the long-context group's packed dense baseline
    (4, 1, 64, 512, 2, 16400, 20000),    # long suffixes behind a prefix
]


MODES = pytest.mark.parametrize("atomic", [True, False], ids=["atomic_dq", "deterministic"])


@MODES
@pytest.mark.parametrize("hq,hkv,d,P,n,ml,T", CASES)
def test_suffix_backward_workspace_follows_the_rule(hq, hkv, d, P, n, ml, T, atomic):
    dims = B.make_dims(hq, hkv, d, P, "bf16", atomic_dq=atomic)
    want, r = _suffix_ws(hq, hkv, d, P, n, ml, T, atomic)
    assert B.workspace_size(B.OP_SUFFIX_BWD, dims, n, ml, T) == want, r


@MODES
@pytest.mark.parametrize("hq,hkv,d,P", sorted({(c[0], c[1], c[2], c[3]) for c in CASES if c[3] > 0}))
def test_prefix_backward_workspace_follows_the_rule(hq, hkv, d, P, atomic):
    dims = B.make_dims(hq, hkv, d, P, "bf16", atomic_dq=atomic)
    want, r = _prefix_ws(hq, hkv, d, P, atomic)
    assert B.workspace_size(B.OP_PREFIX_BWD, dims) == want, r


def test_rule_decisions_at_named_shapes():
    # Llama3-8B group at P = 4096: Phase B whole; Phase C in two shares of
    # the shared launch (atomic mode), or in three shares of the
    # key-outer-only launch (512 steps for key tile 0 against 179 per slot)
    assert _suffix_r(32, 8, 4096, 1, 512, True) == 1 and _prefix_r(32, 8, 4096, True) == 2
    assert _suffix_r(32, 8, 4096, 1, 512, False) == 1 and _prefix_r(32, 8, 4096, False) == 3
    # the launch choice at the measured points: key-outer-only from 175
    # steps per CU on, shared at 87 and fewer
    g = 4
    assert _wide(_causal(4096, g, 192), 8, False) and _wide(_causal(8192, g, 192), 2, False)
    assert not _wide(_causal(8192, g, 192), 1, False) and not _wide(_causal(2048, g, 192), 8, False)
    assert not _wide(_causal(4096, g, 192), 2, False)
    # the long-context group (P = 28672) fills the GPU without shares
    assert _prefix_r(32, 8, 28672, True) == 1 and _suffix_r(32, 8, 28672, 1, 128, True) == 1
    # one kv head, short prefix: the sweeps are cut
    assert _suffix_r(4, 1, 2048, 1, 700, False) == 5 and _prefix_r(4, 1, 2048, False) == 8
    # long prefixes fill the GPU without shares
    assert _prefix_r(32, 8, 16384, False) == 1 and _suffix_r(4, 1, 131072, 2, 1000, False) == 1
    # long whole sequences on 192-key tiles: one kv head's two sequences are
    # cut, the long-context group's eight trajectories are not
    assert _suffix_r(4, 1, 0, 2, 16500, False) > 1 and _suffix_r(32, 8, 0, 8, 28800, False) == 1


def test_fp32_storage_never_splits():
    dims = B.make_dims(4, 1, 128, 2048, "f32")  # fp32 storage has no atomic mode either
    base = B.workspace_size(B.OP_SUFFIX_BWD, dims, 1, 700, 700)
    # fp32: row statistic, log2 LSE and the fp32 dQ accumulator only
    assert base == _align(4 * 700 * 4) * 2 + _align(700 * 4 * 128 * 4)
