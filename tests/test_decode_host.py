"""Host logic of the decode loop (no GPU): slot allocator, live-length mirror, step plans.

The mirror is checked against an independent definition: by Alg. 1 a slot's live
length is the number of steps it took since it was admitted or last flushed, modulo M
(a step at L = C merges and resets).  The plans are checked for the queue split of
Sec. 4 (append queue first, merge queue second) and for graph keys that encode the
phase."""

import random

import pytest

from paper_2608_15533_amd.scheduler import balanced_order, MODES, DecodeScheduler, SlotError


def test_allocator_hands_out_lowest_free_slot_and_rejects_misuse():
    s = DecodeScheduler(3, 4)
    assert [s.admit() for _ in range(3)] == [0, 1, 2]
    assert s.free_slots == 0
    with pytest.raises(SlotError):
        s.admit()
    s.release(1)
    with pytest.raises(SlotError):
        s.release(1)
    with pytest.raises(SlotError):
        s.release(7)
    assert s.admit() == 1
    with pytest.raises(ValueError):
        DecodeScheduler(2, 0)
    with pytest.raises(ValueError):
        DecodeScheduler(2, 4, mode="bogus")


def test_fused_plan_is_all_active_slots_keyed_by_batch_size():
    s = DecodeScheduler(8, 4, "fused")
    for _ in range(5):
        s.admit()
    s.release(2)
    p = s.plan()
    assert p.order == (0, 1, 3, 4)
    assert (p.n_append, p.n_merge, p.key) == (4, 0, ("fused", 4))
    assert p.row_of(3) == 2


def test_fused_plan_puts_merging_slots_first():
    s = DecodeScheduler(6, 3, "fused", merge_first=True)
    a, b = s.admit(), s.admit()
    s.commit(s.plan())                 # a, b at L = 1
    c = s.admit()                      # c at L = 0
    s.commit(s.plan())                 # a, b at L = 2 = C (full), c at L = 1
    p = s.plan()
    assert p.order == (a, b, c)
    assert p.merge_slots == (a, b) and p.append_slots == (c,)
    assert p.key == ("fused", 3)
    s.commit(p)                        # a, b restart at 0; c reaches L = C
    p = s.plan()
    assert p.merge_slots == (c,) and p.order == (c, a, b)


def test_balanced_plan_orders_rows_by_live_length_longest_first():
    """Balanced row order: merging slots first, then by decreasing live length, ties in
    slot order; the same slots and queues as slot order, only the rows move."""
    s = DecodeScheduler(6, 4, "fused", row_order="balanced")
    slots = [s.admit() for _ in range(6)]
    s.live[:] = [1, 3, 0, 2, 3, 1]
    p = s.plan()
    assert p.order == (1, 4, 3, 0, 5, 2)
    assert p.merge_slots == (1, 4) and p.append_slots == (0, 2, 3, 5)
    assert p.key == ("fused", 6)
    assert balanced_order(slots, s.live) == p.order
    with pytest.raises(ValueError):
        DecodeScheduler(2, 4, "fused", row_order="bogus")


def test_balanced_order_spreads_merges_over_the_xcds():
    """With 32 heads per row the kernel runs row r on XCD r mod 8: at any stagger the
    balanced order gives each XCD an equal share of the merging slots (within one)."""
    import numpy as np
    rng = np.random.default_rng(5)
    M = 16
    off = rng.integers(0, M, size=256)
    for k in range(M):
        live = (off + k) % M
        order = balanced_order(range(256), live)
        per_xcd = np.zeros(8, dtype=int)
        for r, slot in enumerate(order):
            per_xcd[r % 8] += live[slot] == M - 1
        assert per_xcd.max() - per_xcd.min() <= 1, (k, per_xcd)


def test_uniform_batch_alternates_append_and_merge_graph_keys():
    """All slots admitted together share one phase: M-1 append plans, then a merge
    plan -- the paper's two graphs per batch descriptor."""
    M = 4
    s = DecodeScheduler(3, M, "phased")
    for _ in range(3):
        s.admit()
    keys = []
    for _ in range(2 * M):
        p = s.plan()
        keys.append(p.key)
        s.commit(p)
    assert keys == [("phased", 3, 0)] * (M - 1) + [("phased", 0, 3)] \
        + [("phased", 3, 0)] * (M - 1) + [("phased", 0, 3)]


def test_merge_interval_one_always_merges():
    s = DecodeScheduler(2, 1, "phased")
    s.admit()
    s.admit()
    for _ in range(3):
        p = s.plan()
        assert (p.n_append, p.n_merge) == (0, 2)
        s.commit(p)


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("seed", range(5))
def test_mirror_matches_steps_since_admission_mod_M(mode, seed):
    """Random admit / release / flush / step traces; the mirror must equal the number of
    steps since admission or flush, modulo M, and a phased plan must put exactly the
    full slots in the merge queue, after the append queue, each sorted."""
    rng = random.Random(seed)
    B, M = 6, rng.choice([1, 2, 3, 5, 8])
    s = DecodeScheduler(B, M, mode)
    since = {}
    for _ in range(300):
        r = rng.random()
        if r < 0.15 and s.free_slots:
            since[s.admit()] = 0
        elif r < 0.25 and s.active:
            slot = rng.choice(s.active)
            s.release(slot)
            del since[slot]
        elif r < 0.30 and s.active:
            slot = rng.choice(s.active)
            s.flushed(slot)
            since[slot] = 0
        else:
            p = s.plan()
            assert sorted(p.order) == sorted(s.active)
            full = sorted(x for x in s.active if since[x] % M == M - 1)
            assert list(p.merge_slots) == full
            assert list(p.append_slots) == sorted(set(s.active) - set(full))
            if mode == "fused":
                assert p.key == ("fused", len(s.active))
                assert p.order == tuple(sorted(s.active))
            else:
                assert list(p.order) == list(p.append_slots) + full
                assert p.key == (mode, p.n_append, p.n_merge)
            s.commit(p)
            for x in p.order:
                since[x] += 1
        for x in s.active:
            assert s.live[x] == since[x] % M


def test_interleaved_order_is_a_balanced_permutation():
    """The interleaved row order keeps the balanced order's per-XCD shares (each XCD's
    rows are every eighth row of the balanced order) and only permutes their dispatch
    order; any row count works."""
    import numpy as np
    from paper_2608_15533_amd.scheduler import interleaved_order
    rng = np.random.default_rng(3)
    for n in (256, 37, 8, 1):
        live = rng.integers(0, 16, size=n)
        o = interleaved_order(range(n), live)
        assert sorted(o) == list(range(n))
    live = rng.integers(0, 16, size=256)
    o, b = interleaved_order(range(256), live), balanced_order(range(256), live)
    for x in range(8):
        assert sorted(o[x::8]) == sorted(b[x::8])
