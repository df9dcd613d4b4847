"""Paged state pool as NumPy fancy indexing.

TEST INFRASTRUCTURE ONLY (see the package docstring).

A page holds one head's recurrent state ([dk, dv] fp32); item n of a state
array [n_rows, H, dk, dv] is (row, head) = divmod(n, H).  The paper moves
checkpointed state between tiers as page rows (section 3.1 and Table 5);
here the pool is a [n_pages, page_elems] array and a page table maps items
to pages:

* save:    pool[ids[n]] = states[n] for ids[n] in [0, n_pages); -1 skips;
           any other id is an error (counted, item skipped).
* restore: states[n] = pool[ids[n]] for valid ids; -1 yields a zero state
           (a cold start); any other id is an error (counted, destination
           left untouched).
* hybrid restore: for every sequence, the attention KV blocks of its prefix
           [0, B) (block j of sequence i: cache[dst[i, j]] = kv_pool[src[i, j]])
           and the recurrent state pages of its checkpoint at B, as one
           operation; block ids follow the restore's id rules (-1 skips).
"""
from __future__ import annotations

import numpy as np


def paged_save(states: np.ndarray, pool: np.ndarray, ids: np.ndarray):
    """Returns (new pool, error count).  Inputs are not modified."""
    items = np.ascontiguousarray(states).reshape(len(ids), -1)
    out = pool.copy().reshape(pool.shape[0], -1)
    errors = 0
    for n, pid in enumerate(np.asarray(ids).tolist()):
        if pid == -1:
            continue
        if 0 <= pid < out.shape[0]:
            out[pid] = items[n]
        else:
            errors += 1
    return out.reshape(pool.shape), errors


def paged_restore(pool: np.ndarray, ids: np.ndarray, dest: np.ndarray):
    """Returns (new destination, error count).  Inputs are not modified."""
    flat_pool = np.ascontiguousarray(pool).reshape(pool.shape[0], -1)
    out = dest.copy().reshape(len(ids), -1)
    errors = 0
    for n, pid in enumerate(np.asarray(ids).tolist()):
        if pid == -1:
            out[n] = 0
        elif 0 <= pid < flat_pool.shape[0]:
            out[n] = flat_pool[pid]
        else:
            errors += 1
    return out.reshape(dest.shape), errors


def hybrid_restore(kv_pool, cache, src_ids, dst_ids, boundaries, block_tokens, state_pool, state_ids, states):
    """Returns (new cache, new states, error count).  Inputs are not modified.

    src_ids / dst_ids: [n_seqs, max_blocks]; boundaries: B per sequence (a
    multiple of block_tokens); state_ids: [n_seqs * H] page ids, states:
    [n_seqs * H, page_elems].  A block with src or dst -1 is skipped; an id
    out of range on either side is an error (counted once, block skipped).
    """
    out_cache = cache.copy()
    errors = 0
    n_src, n_dst = kv_pool.shape[0], cache.shape[0]
    for i, b in enumerate(boundaries):
        for j in range(int(b) // block_tokens):
            s, d = int(src_ids[i][j]), int(dst_ids[i][j])
            if s == -1 or d == -1:
                continue
            if 0 <= s < n_src and 0 <= d < n_dst:
                out_cache[d] = kv_pool[s]
            else:
                errors += 1
    new_states, e2 = paged_restore(state_pool, state_ids, states)
    return out_cache, new_states, errors + e2
