"""Host logic of the prefix-state lifecycle (paper Sec. 4.3), CPU only:
the pinned staging pool and its per-tensor fallback, and the HBM budget
guard of speculative prefetch, with faked memory figures."""
import torch

from paper_2606_01143_amd.stack import HbmBudget, PinnedPool


def test_pool_hands_out_aligned_slices_then_falls_back():
    made = []

    def alloc(n):  # host memory standing in for pinned memory
        made.append(n)
        return torch.empty(n, dtype=torch.uint8)

    pool = PinnedPool(10_000, alloc=alloc, align=4096)
    a = pool.take(100)
    b = pool.take(5000)
    assert a.numel() == 100 and b.numel() == 5000
    assert b.data_ptr() - pool.arena.data_ptr() == 4096  # aligned after the first slice
    c = pool.take(2000)  # 4096 + 5000 -> 12288: does not fit in 10 000
    assert pool.fallbacks == 1 and c.numel() == 2000 and made == [10_000, 2000]
    pool.reset()
    assert pool.take(9000).data_ptr() == pool.arena.data_ptr()


def test_empty_pool_always_falls_back():
    pool = PinnedPool(0, alloc=lambda n: torch.empty(n, dtype=torch.uint8))
    pool.take(10)
    pool.take(10)
    assert pool.fallbacks == 2


def _budget(free, total, allocated, reserved, limit=None, reserve=100, slack=1.1):
    return HbmBudget(reserve=reserve, slack=slack, limit=limit, mem_get_info=lambda: (free, total),
                     allocated=lambda: allocated, reserved=lambda: reserved)


def test_budget_counts_driver_free_and_cached_blocks():
    # 1000 free in the driver, 500 cached in the allocator
    b = _budget(free=1000, total=10_000, allocated=4000, reserved=4500)
    assert b.headroom() == 1500
    assert b.allows(1000)            # 1500 - 1100 = 400 >= 100
    assert not b.allows(1300)        # 1500 - 1430 = 70 < 100


def test_budget_limit_caps_headroom():
    b = _budget(free=5000, total=10_000, allocated=4000, reserved=4000, limit=5000)
    assert b.headroom() == 1000
    assert not b.allows(900)         # 1000 - 990 < 100
    assert b.allows(800)


def test_zero_limit_forces_demand_loads():
    b = _budget(free=10 ** 9, total=10 ** 10, allocated=10, reserved=10, limit=0)
    assert not b.allows(1)
