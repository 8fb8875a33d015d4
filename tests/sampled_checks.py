"""Element-wise checks of full-length outputs on sampled rows and keys,
each computed by the oracle from its own sequence
(``oracle.attention.sampled_rows_reference`` / ``sampled_keys_reference``,
both pinned to the whole oracle on small groups), plus the identities that
hold at any size.  Shared by the GPU tests of long groups."""
import numpy as np

from oracle.attention import sampled_keys_reference, sampled_rows_reference


def rel(got, ref):
    g, r = np.stack(got), np.stack(ref)
    return float(np.max(np.abs(g - r)) / max(np.max(np.abs(r)), 1e-30))


def sample_rows(P, lens, rng):
    n = len(lens)
    rand = rng.integers(0, P, 5).tolist() if P > 0 else []
    prefix = sorted({r for r in (0, 1, 63, 64, 127, 128, 255, 256, P // 2, P - 2, P - 1, *rand) if 0 <= r < P})
    suffix = sorted({(i, t) for i in (0, n // 2, n - 1)
                     for t in (0, 31, 32, 127, 128, lens[i] // 2, lens[i] - 1) if t < lens[i]})
    return prefix, suffix


def sample_keys(P, lens, rng):
    """Prefix keys at both sides of the 64-key and 192-key tile edges (the
    two key-outer workgroup widths), the middle, the end and random ones;
    suffix keys at tile edges of three suffixes."""
    n = len(lens)
    if P > 32768:
        lo = P - 2048
        prefix = {lo, lo + 63, lo + 64, lo + 191, lo + 192, P - 1025, P - 1024, P - 65, P - 64, P - 2, P - 1,
                  *rng.integers(lo, P, 3).tolist()}
    else:
        last = (P - 1) // 192 * 192  # first key of the last 192-key tile
        rand = rng.integers(0, P, 4).tolist() if P > 0 else []
        prefix = {0, 1, 63, 64, 127, 128, 191, 192, 383, 384, P // 2 - 1, P // 2, last - 1, last,
                  P - 65, P - 64, P - 2, P - 1, *rand}
    prefix = sorted(k for k in prefix if 0 <= k < P)
    suffix = sorted({(i, t) for i in (0, n // 2, n - 1)
                     for t in (0, 1, 63, 64, lens[i] // 2, lens[i] - 1) if t < lens[i]})
    return prefix, suffix


def sampled_errors(inp, got, rng, cache=True):
    """max-abs-relative error per output family on the sampled rows and keys;
    ``got`` is ``DeviceGroup.fetch`` of the schedule (``cache``: with G_K,
    G_V) or of the dense baseline."""
    shp = inp["shape"]
    P, lens = shp.prefix_len, [int(x) for x in inp["suffix_lens"]]
    cu = inp["cu_seqlens"]
    errs = {}
    prefix_rows, suffix_rows = sample_rows(P, lens, rng)
    ref = sampled_rows_reference(inp, prefix_rows, suffix_rows)
    for key, rows, sfx in (("prefix", prefix_rows, "_p"), ("suffix", suffix_rows, "_s")):
        if not rows:  # no prefix (P = 0)
            continue
        for f in ("o", "dq", "lse"):
            g, r = [], []
            for row in rows:
                idx = row if key == "prefix" else int(cu[row[0]]) + row[1]
                g.append(got[f + sfx][idx])
                r.append(ref[key][row][f])
            errs[f"{f}{sfx}"] = rel(g, r)
    prefix_keys, suffix_keys = sample_keys(P, lens, rng)
    kref = sampled_keys_reference(inp, prefix_keys, suffix_keys)
    fams = (("dk", "dk_p"), ("dv", "dv_p")) + ((("g_k", "g_k"), ("g_v", "g_v")) if cache else ())
    for f, gk in fams if prefix_keys else ():
        errs[gk + "@keys"] = rel([got[gk][j] for j in prefix_keys], [kref["prefix"][j][f] for j in prefix_keys])
    for f in ("dk", "dv"):
        errs[f + "_s@keys"] = rel([got[f + "_s"][int(cu[i]) + t] for i, t in suffix_keys],
                                  [kref["suffix"][(i, t)][f] for i, t in suffix_keys])
    return errs


def identity_errors(inp, got):
    """sum over all keys of dK = 0, and sum over all keys of dV = sum over
    all rows and group heads of dO (G_Y for the prefix rows): (dk residual,
    dv residual), each relative to its scale."""
    shp = inp["shape"]
    dk_all = np.concatenate([got["dk_p"], got["dk_s"]])
    dk_res = np.abs(dk_all.sum(axis=0)).max() / np.abs(dk_all).sum(axis=0).max()
    dv = np.concatenate([got["dv_p"], got["dv_s"]]).sum(axis=0)
    g_y = np.asarray(inp["do_p"], np.float64).sum(axis=0)
    do_sum = g_y.sum(axis=0) + np.asarray(inp["do_s"], np.float64).sum(axis=0)  # [Hq, d]
    G = shp.num_q_heads // shp.num_kv_heads
    want = do_sum.reshape(shp.num_kv_heads, G, -1).sum(axis=1)
    return dk_res, np.abs(dv - want).max() / np.abs(want).max()
