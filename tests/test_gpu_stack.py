"""Stacked layers with the prefix-state lifecycle (paper Sec. 3.3, 4.3):
offloading the dormant prefix state to pinned host memory and restoring it
for Phase C (prefetched, demand-loaded, or through per-tensor pinned
fallbacks) changes no result bit, over repeated steps."""
import pytest

SHAPE_ARGS = dict(layers=3, num_q_heads=4, num_kv_heads=2, head_dim=128, prefix_len=300,
                  suffix_lens=(70, 129, 33))


def _snapshot(sg):
    import torch
    out = []
    for t in sg.layers:
        out.append({k: t[k].clone() for k in ("o_p", "lse_p", "gk", "gv", "dq_p", "dk_p", "dv_p")})
    grads = [{l: tuple(x.clone() for x in g) for l, g in mb.items()} for mb in sg.suffix_grads]
    torch.cuda.synchronize()
    return out, grads


def _equal(a, b):
    import torch
    (la, ga), (lb, gb) = a, b
    for x, y in zip(la, lb):
        for k in x:
            assert torch.equal(x[k], y[k]), k
    for x, y in zip(ga, gb):
        for l in x:
            assert all(torch.equal(u, v) for u, v in zip(x[l], y[l])), l


@pytest.mark.gpu
@pytest.mark.parametrize("mode", ["prefetch", "demand", "pool_fallback"])
def test_offload_changes_no_result_bit(gpu, mode):
    from paper_2606_01143_amd.stack import HbmBudget, StackedGroup, StackShape
    shape = StackShape(**SHAPE_ARGS)
    print(f"\n[gpu stack] {mode} {shape}", flush=True)
    ref = StackedGroup(shape, seed=3, keep_suffix_grads=True)
    ref.run()
    want = _snapshot(ref)
    del ref
    kw = {}
    if mode == "demand":
        kw["budget"] = HbmBudget(limit=0)
    if mode == "pool_fallback":
        kw["pool_factor"] = 0.1
    sg = StackedGroup(shape, seed=3, offload=True, keep_suffix_grads=True, **kw)
    for _ in range(2):
        sg.run()
        _equal(_snapshot(sg), want)
    L = shape.layers
    if mode == "prefetch":
        assert sg.stats["prefetched"] == 2 * L and sg.stats["demand_loaded"] == 0
    if mode == "demand":
        assert sg.stats["demand_loaded"] == 2 * L and sg.stats["prefetched"] == 0
    if mode == "pool_fallback":
        assert sg.stats["pool_fallbacks"] > 0
