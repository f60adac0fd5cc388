"""Host-side logic of the residency planner (Algorithm 1's pin / fallback-encode
and refresh lines, section 3.3): budget accounting, level schedule and refresh
insertion.  No GPU."""
import pytest

from paper_2606_17421_amd.planner import LinearGroup, encoded_bytes, plan

N = 1 << 10


def stack(layers, d=8, tee_every=None):
    gs = []
    for i in range(layers):
        gs.append(LinearGroup(f"g{i}", d, d, tee_after=bool(tee_every) and (i + 1) % tee_every == 0))
    return gs


def test_everything_pinned_under_a_large_budget():
    gs = stack(6)
    p = plan(gs, 1 << 40, full_limbs=4, n=N)
    assert p.pinned == 6 and p.fallback == 0
    assert p.pinned_bytes == sum(s.encoded_bytes for s in p.steps)


def test_nothing_pinned_under_a_zero_budget():
    p = plan(stack(5), 0, full_limbs=4, n=N)
    assert p.pinned == 0 and p.fallback == 5 and p.pinned_bytes == 0


def test_pins_in_topological_order_until_the_budget_runs_out():
    gs = stack(6)
    one = encoded_bytes(gs[0], 4, N)
    p = plan(gs, 2 * one + 10, full_limbs=4, n=N, min_out_limbs=3)   # every group starts at 4 limbs
    assert [s.pinned for s in p.steps] == [True, True, False, False, False, False]
    assert p.pinned_bytes == 2 * one


def test_level_schedule_and_refresh_insertion():
    # 4 limbs: a group's output keeps >= 2 limbs, so groups start at 4 or 3 and a refresh
    # follows every group that starts at 3
    p = plan(stack(5), 1 << 40, full_limbs=4, n=N)
    assert [s.level for s in p.steps] == [4, 3, 4, 3, 4]
    assert [s.refresh_after for s in p.steps] == [False, True, False, True, False]
    # smaller groups later in the chain are cheaper to pin (fewer limbs)
    assert p.steps[1].encoded_bytes * 4 == p.steps[0].encoded_bytes * 3


def test_tee_window_forces_a_refresh():
    p = plan(stack(4, tee_every=1), 1 << 40, full_limbs=5, n=N)
    assert [s.level for s in p.steps] == [5, 5, 5, 5]
    assert [s.refresh_after for s in p.steps] == [True, True, True, False]   # none after the last


def test_a_later_smaller_group_can_still_be_pinned():
    gs = [LinearGroup("big", 16, 8), LinearGroup("small", 8, 16)]
    small_bytes = encoded_bytes(gs[1], 3, N)
    p = plan(gs, small_bytes, full_limbs=4, n=N)
    assert [s.pinned for s in p.steps] == [False, True]


def test_shape_mismatch_and_short_chain_are_rejected():
    with pytest.raises(ValueError):
        plan([LinearGroup("a", 8, 8), LinearGroup("b", 8, 4)], 0, full_limbs=4, n=N)
    with pytest.raises(ValueError):
        plan(stack(2), 0, full_limbs=2, n=N)          # no rescale would keep 2 limbs


class _FakeTensor:
    """Stand-in with the two methods the draw check reads (a storage span)."""

    def __init__(self, ptr, nbytes):
        self.ptr, self.nbytes = ptr, nbytes

    def data_ptr(self):
        return self.ptr

    def numel(self):
        return self.nbytes // 4

    def element_size(self):
        return 4


def test_each_refresh_needs_its_own_randomness():
    """Two refreshes never receive the same (a, e) storage, and a pass with fewer
    draws than refreshes is refused (no GPU: the check only reads storage spans)."""
    from paper_2606_17421_amd.planner import check_refresh_draws
    a0, e0 = _FakeTensor(0x1000, 256), _FakeTensor(0x2000, 64)
    a1, e1 = _FakeTensor(0x3000, 256), _FakeTensor(0x4000, 64)
    check_refresh_draws([(a0, e0), (a1, e1)], 2)
    with pytest.raises(ValueError):
        check_refresh_draws([(a0, e0)], 2)
    with pytest.raises(ValueError):
        check_refresh_draws([(a0, e0), (a0, e1)], 2)                 # a shared
    with pytest.raises(ValueError):
        check_refresh_draws([(a0, e0), (a1, _FakeTensor(0x2020, 64))], 2)   # e overlaps partly
    with pytest.raises(ValueError):
        check_refresh_draws([(a0, e0), (_FakeTensor(0x2000, 16), e1)], 2)   # a inside the first e
