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


def hybrid_boundary(n_tokens: int, interval: int, kv_block_tokens: int, kv_cached: int, state_cached: int):
    """Joint boundary of a hybrid cache: attention KV blocks and recurrent
    checkpoints restored at one position B (sections 1 and 6: reusable
    attention prefixes must align with recurrent checkpoints).

    B is the largest b = j * C with b <= N - 1 (the strict prefix of section
    2.2) whose every KV block [0, b) is cached (the first kv_cached tokens
    are, in whole blocks of kv_block_tokens) and whose checkpoint exists
    (checkpoints are cached for every multiple of C up to state_cached).
    Returns (B, number of KV blocks in [0, B)).  Raises ValueError when the
    blocks do not tile the checkpoint interval (no checkpoint position would
    fall on a block boundary) or on negative or zero sizes.
    """
    if n_tokens < 1 or interval < 1 or kv_block_tokens < 1 or kv_cached < 0 or state_cached < 0:
        raise ValueError("hybrid_boundary needs N, C, block >= 1 and cached lengths >= 0")
    if interval % kv_block_tokens != 0:
        raise ValueError("KV blocks must tile the checkpoint interval")
    best = 0
    b = 0
    while b <= n_tokens - 1:
        blocks_cached = all((j + 1) * kv_block_tokens <= kv_cached for j in range(b // kv_block_tokens))
        if blocks_cached and b <= state_cached:
            best = b
        b += interval
    return best, best // kv_block_tokens
