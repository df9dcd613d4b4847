"""Checkpoint lookup rules by brute-force enumeration.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Section 2.2 of the paper defines N (prompt length), C (checkpoint interval),
B (the prefix a restored checkpoint represents) and p (the scheduler's
computed-token count).  A state for prefix [0, B) continues from B, so the
repaired lookup restricts the query to the prompt without its last token and
selects the largest aligned checkpoint inside it; in a general cache the
checkpoint must also be available (same section).  Section 3.2 describes the
pre-fix behaviour that Table 4's "before" columns record.

Nothing here evaluates the closed form floor((N - 1) / C) * C: every rule
walks the candidate positions 0, C, 2C, ... explicitly.
"""
from __future__ import annotations


def strict_prefix_boundary(n_tokens: int, interval: int, available: int) -> int:
    """Largest aligned boundary b = j * C with b <= N - 1 and b <= available.

    ``available`` is the length of the contiguous cached prefix (tokens).
    b = 0 means a cold start.  Raises ValueError for N < 1, C < 1 or
    available < 0 (the rule is undefined there).
    """
    if n_tokens < 1 or interval < 1 or available < 0:
        raise ValueError("strict_prefix_boundary needs N >= 1, C >= 1, available >= 0")
    best = 0
    b = 0
    while b <= n_tokens - 1:
        if b <= available:
            best = b
        b += interval
    return best


def nonstrict_lookup(n_tokens: int, interval: int, available: int):
    """The pre-fix behaviour (section 3.2): lookup over all N tokens.

    Returns (B, p): the retained lookup boundary B is the largest aligned
    checkpoint b <= N (and <= available); the complete-prompt branch then
    credits the scheduler with N - 1 when B == N, otherwise p = B.  With
    B == N and p == N - 1 the restored state already holds token N - 1 and
    the scheduler feeds it again.
    """
    if n_tokens < 1 or interval < 1 or available < 0:
        raise ValueError("lookup needs N >= 1, C >= 1, available >= 0")
    best = 0
    b = 0
    while b <= n_tokens:
        if b <= available:
            best = b
        b += interval
    p = n_tokens - 1 if best == n_tokens else best
    return best, p
