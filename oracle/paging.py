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
