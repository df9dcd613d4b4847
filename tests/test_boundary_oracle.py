"""Pins for the lookup-rule oracle against the paper's printed values.

Sources: Table 4 (section 5.2), the CPU-reload boundaries of section 5.5 and
the Figure 2 caption; the checkpoint interval C = 1,792 is Table 1's.
"""
import os

import pytest

from oracle.boundary import nonstrict_lookup, strict_prefix_boundary

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [line.split() for line in f if line.strip() and not line.startswith("#")]


TABLE4 = _rows("table4_boundary_matrix.txt")
SERIAL = _rows("serial_reload_boundaries.txt")


@pytest.mark.parametrize("row", TABLE4, ids=[r[0] for r in TABLE4])
def test_table4_after_repair(row):
    N, B_after, suffix = int(row[0]), int(row[4]), int(row[5])
    B = strict_prefix_boundary(N, 1792, N)
    assert B == B_after and N - B == suffix and N - B >= 1


@pytest.mark.parametrize("row", TABLE4, ids=[r[0] for r in TABLE4])
def test_table4_before_repair(row):
    N, B_before, p_before, first_diff = int(row[0]), int(row[1]), int(row[2]), row[3]
    B, p = nonstrict_lookup(N, 1792, N)
    assert (B, p) == (B_before, p_before)
    # the two diverging rows are exactly those where state and scheduler disagree
    assert (B != p) == (first_diff != "-")


@pytest.mark.parametrize("row", SERIAL, ids=[r[0] for r in SERIAL])
def test_serial_reload_boundaries(row):
    N, C, B_ref, suffix = map(int, row)
    assert strict_prefix_boundary(N, C, N) == B_ref
    assert N - B_ref == suffix


def test_figure2_caption():
    assert nonstrict_lookup(3584, 1792, 3584) == (3584, 3583)
    assert strict_prefix_boundary(3584, 1792, 3584) == 1792


@pytest.mark.parametrize("N,C,B", [(256, 16, 240), (3584, 256, 3328), (32768, 1024, 31744)]
                         + [(512 * i, 256, 512 * i - 256) for i in range(1, 10)])
def test_workload_boundaries(N, C, B):
    assert strict_prefix_boundary(N, C, N) == B


def test_properties_small_grid():
    for C in (1, 2, 3, 5, 16, 64):
        for N in range(1, 200):
            for avail in range(0, 210, 7):
                B = strict_prefix_boundary(N, C, avail)
                assert B % C == 0 and 0 <= B <= N - 1 and B <= avail
                # maximal: the next aligned position is outside the query or unavailable
                assert B + C > N - 1 or B + C > avail


def test_invalid_arguments():
    for args in [(0, 16, 0), (-3, 16, 0), (10, 0, 10), (10, -1, 10), (10, 16, -1)]:
        with pytest.raises(ValueError):
            strict_prefix_boundary(*args)
