"""Pins for the joint attention-KV / recurrent-state boundary and its restore.

The paper's reloads move attention-related entries, checkpointed state and
model-specific tail entries together (section 2.1) and it applies the
principle that reusable attention prefixes must align with recurrent
checkpoints (sections 1 and 6).  What it prints about that structure is the
bytes each rank moved per reload (section 5.2) and the total H2D volume of
the instrumented run (section 5.3, Table 5).  A linear model, a constant per
reload (recurrent state and tail entries) plus a constant per restored token
(the attention KV of that rank), fitted on two of those numbers, must
reproduce the others once B comes from the boundary rule: the pre-fix
N = 5,376 count and the nine-reload total are independent checks of the
strict-prefix boundary and the per-token attention bytes.
"""
import os

import numpy as np
import pytest

from oracle.boundary import hybrid_boundary, nonstrict_lookup, strict_prefix_boundary
from oracle.paging import hybrid_restore

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
C_PAPER = 1792          # Table 1
BLOCK = 16              # KV block tokens used here (divides C)


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [line.split() for line in f if line.strip() and not line.startswith("#")]


def _reload_b(n, rule):
    if rule == "strict":
        b, nb = hybrid_boundary(n, C_PAPER, BLOCK, n, n)
        assert nb * BLOCK == b
        return b
    return nonstrict_lookup(n, C_PAPER, n)[0]


def test_reload_bytes_follow_the_hybrid_boundary():
    rows = _rows("hybrid_reload_bytes.txt")
    per_rank = {(int(r[0]), r[2]): int(r[3]) for r in rows if r[0] != "total"}
    total = [r for r in rows if r[0] == "total"][0]
    # fit on the two repaired counts
    b1, b2 = _reload_b(3584, "strict"), _reload_b(5376, "strict")
    assert (b1, b2) == (1792, 3584)
    y1, y2 = per_rank[(3584, "strict")], per_rank[(5376, "strict")]
    assert (y2 - y1) % (b2 - b1) == 0
    per_token = (y2 - y1) // (b2 - b1)
    const = y1 - per_token * b1
    assert per_token == 8268 and const == 39993344
    model = lambda b: const + per_token * b
    # independent checks: the pre-fix counts (B from the pre-fix rule) ...
    for n in (3584, 5376):
        assert model(_reload_b(n, "prefix")) == per_rank[(n, "prefix")]
    # ... and Table 5's H2D volume over the nine repaired reloads on every rank
    ranks, lengths, volume = int(total[1]), [int(x) for x in total[2:-1]], int(total[-1])
    assert len(lengths) == 9
    assert ranks * sum(model(_reload_b(n, "strict")) for n in lengths) == volume


@pytest.mark.parametrize("seed", range(4))
def test_hybrid_boundary_equals_strict_prefix_of_the_shorter_cache(seed):
    rng = np.random.default_rng(seed)
    for _ in range(300):
        bt = int(rng.choice([1, 2, 4, 16]))
        C = bt * int(rng.integers(1, 6))
        N = int(rng.integers(1, 12 * C))
        kv, st = int(rng.integers(0, 12 * C)), int(rng.integers(0, 12 * C))
        B, nb = hybrid_boundary(N, C, bt, kv, st)
        assert B == strict_prefix_boundary(N, C, min(kv, st))
        assert nb * bt == B and B % C == 0 and B <= N - 1 and B <= kv and B <= st
        nxt = B + C                                   # maximal: the next position fails a condition
        assert nxt > N - 1 or nxt > kv or nxt > st


def test_hybrid_boundary_reproduces_table4_and_rejects_misaligned_blocks():
    for r in _rows("table4_boundary_matrix.txt"):
        n, b_after = int(r[0]), int(r[4])
        assert hybrid_boundary(n, C_PAPER, BLOCK, n, n) == (b_after, b_after // BLOCK)
    # state cached only up to the first checkpoint; KV only 1,000 tokens
    assert hybrid_boundary(5376, C_PAPER, BLOCK, 5376, 1792) == (1792, 112)
    assert hybrid_boundary(5376, C_PAPER, BLOCK, 1000, 5376) == (0, 0)
    with pytest.raises(ValueError):
        hybrid_boundary(5376, C_PAPER, 48, 5376, 5376)      # 1,792 is not a multiple of 48
    with pytest.raises(ValueError):
        hybrid_boundary(0, C_PAPER, BLOCK, 0, 0)


def test_hybrid_restore_oracle_hand_case():
    kv_pool = np.arange(6 * 4, dtype=np.uint8).reshape(6, 4)       # 6 pool blocks of 4 bytes
    cache = np.full((5, 4), 0xEE, np.uint8)
    src = np.array([[3, 0, 5], [1, -1, 9]])
    dst = np.array([[4, 2, 0], [1, 3, 3]])
    state_pool = np.arange(3 * 2, dtype=np.float32).reshape(3, 2) + 1
    states = np.full((4, 2), 7.0, np.float32)
    # sequence 0 restores 2 blocks (B = 2 * bt), sequence 1 three (one skipped, one out of range)
    new_cache, new_states, err = hybrid_restore(kv_pool, cache, src, dst, [8, 12], 4, state_pool,
                                                np.array([2, -1, 0, 5]), states)
    assert err == 2                                   # block id 9 and state page 5
    assert np.array_equal(new_cache[4], kv_pool[3]) and np.array_equal(new_cache[2], kv_pool[0])
    assert np.array_equal(new_cache[1], kv_pool[1])
    assert np.all(new_cache[[0, 3]] == 0xEE)          # block 2 of sequence 0 is past B; the others skipped
    assert np.array_equal(new_states[0], state_pool[2]) and np.all(new_states[1] == 0)
    assert np.array_equal(new_states[2], state_pool[0]) and np.all(new_states[3] == 7.0)
    assert np.all(cache == 0xEE) and np.all(states == 7.0)            # inputs untouched
