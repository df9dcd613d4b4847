"""Pins for the paged-pool oracle on hand-checkable cases."""
import numpy as np

from oracle.paging import paged_restore, paged_save


def test_save_then_restore_round_trip_under_permutation():
    rng = np.random.default_rng(0)
    states = rng.standard_normal((3, 2, 4, 4)).astype(np.float32)      # 6 items
    pool = np.full((10, 16), np.nan, np.float32)
    ids = np.array([7, 2, 9, 0, 5, 3], np.int32)
    pool2, err = paged_save(states, pool, ids)
    assert err == 0
    for n, pid in enumerate(ids):
        r, h = divmod(n, 2)
        assert np.array_equal(pool2[pid], states[r, h].ravel())
    untouched = sorted(set(range(10)) - set(ids.tolist()))
    assert np.all(np.isnan(pool2[untouched]))
    dest = np.full_like(states, 123.0)
    back, err = paged_restore(pool2, ids, dest)
    assert err == 0 and np.array_equal(back, states)


def test_minus_one_skips_save_and_zero_fills_restore():
    states = np.ones((2, 1, 2, 2), np.float32)
    pool = np.full((4, 4), 5.0, np.float32)
    pool2, err = paged_save(states, pool, np.array([-1, 1], np.int32))
    assert err == 0 and np.all(pool2[0] == 5) and np.all(pool2[1] == 1)
    dest = np.full((2, 1, 2, 2), 9.0, np.float32)
    back, err = paged_restore(pool2, np.array([-1, 3], np.int32), dest)
    assert err == 0 and np.all(back[0] == 0) and np.all(back[1] == 5)


def test_out_of_range_ids_are_counted_and_leave_destination():
    states = np.arange(8, dtype=np.float32).reshape(2, 1, 2, 2)
    pool = np.zeros((2, 4), np.float32)
    pool2, err = paged_save(states, pool, np.array([2, -5], np.int32))
    assert err == 2 and np.all(pool2 == 0)
    dest = np.full((2, 1, 2, 2), 7.0, np.float32)
    back, err = paged_restore(pool, np.array([0, 99], np.int32), dest)
    assert err == 1 and np.all(back[0] == 0) and np.all(back[1] == 7)
