"""Paged KV cache addressing -- TEST INFRASTRUCTURE (oracle side).

Only ``tests/`` may import this module; it imports nothing from the GPU package.

A paged cache (the block tables of a paged-attention engine such as vLLM, the engine the paper also runs
on, Section 3.1) keeps every sequence's positions in fixed-size blocks of one shared pool: position p of
sequence b lives in pool row ``block_table[b][p // block_size] * block_size + p % block_size``.  Plain
definitions, run literally:

  * ``pool_row``    -- that row;
  * ``build_pool``  -- a pool [NL, rows, Hkv, D] filled from a sequence-ordered cache by copying every
                       position to its row one by one;
  * ``rows_of``     -- the pool rows of a list of retained positions;
  * ``never_retained_again`` -- the positions of a sequence that no step from j to j + horizon
                       retains (each step's retained set from the oracle's Algorithm 1/2 loops);
  * ``freeable_blocks`` -- the logical blocks made only of such positions (Section 3.2: an evicted
                       entry leaves the cache, so its block can go back to the pool).

Pins (``tests/test_oracle_paged.py``): with the identity table of one sequence the pool row is the
position; a pool built from any table reproduces the sequence-ordered cache at every position read back
through the table; a hand-worked example of the freeable blocks (tiny workload at step 80); a block
freeable at one step stays freeable at every later one; a longer horizon frees nothing more.
"""
from __future__ import annotations

import numpy as np

from oracle import retained


def pool_row(block_table_row, block_size: int, p: int) -> int:
    return int(block_table_row[p // block_size]) * block_size + p % block_size


def build_pool(cache: np.ndarray, lengths, block_table: np.ndarray, block_size: int, n_blocks: int) -> np.ndarray:
    """cache [NL, B, Hkv, L, D] -> pool [NL, n_blocks * block_size, Hkv, D]; positions >= lengths[b] are not copied."""
    NL, B, Hkv, _, D = cache.shape
    pool = np.zeros((NL, n_blocks * block_size, Hkv, D), dtype=cache.dtype)
    for b in range(B):
        for p in range(int(lengths[b])):
            pool[:, pool_row(block_table[b], block_size, p)] = cache[:, b, :, p]
    return pool


def rows_of(idx: np.ndarray, count: np.ndarray, block_table: np.ndarray, block_size: int) -> np.ndarray:
    """The pool rows of idx[b, :count[b]] (padding -1 kept)."""
    out = np.full_like(idx, -1)
    for b in range(idx.shape[0]):
        for r in range(int(count[b])):
            out[b, r] = pool_row(block_table[b], block_size, int(idx[b, r]))
    return out


def default_horizon(seg_row, pol_row) -> int:
    """Later steps to scan: enough for the speech window (one token per step once the delay has passed)
    to reach every speech position, plus a margin."""
    _, l_s, _, _ = (int(x) for x in seg_row)
    return l_s + max(int(pol_row[1]), 1) + 4


def never_retained_again(seg_row, pol_row, horizon: int | None = None) -> np.ndarray:
    """Boolean mask over positions [0, length) of a sequence at step j = seg_row[3]: True where none of
    the retained sets of steps j, j+1, .., j+horizon holds the position (the sequence grows by one output
    token per step; positions past the current length are not part of the mask)."""
    p_pre, l_s, p_mid, j = (int(x) for x in seg_row)
    pol_row = np.asarray(pol_row, dtype=np.int32).reshape(5)
    if horizon is None:
        horizon = default_horizon(seg_row, pol_row)
    length = p_pre + l_s + p_mid + j
    kept = np.zeros(length, dtype=bool)
    # the retained sets of steps j .. j + horizon, one row per step, from one call
    steps = np.arange(j, j + horizon + 1, dtype=np.int32)
    seg = np.stack([np.full_like(steps, p_pre), np.full_like(steps, l_s), np.full_like(steps, p_mid), steps], axis=1)
    idx, cnt = retained(seg, pol_row)
    for r in range(len(steps)):
        rows = idx[r, :int(cnt[r])]
        kept[rows[rows < length]] = True
    return ~kept


def freeable_blocks(seg_row, pol_row, block_size: int, horizon: int | None = None) -> list[int]:
    """Logical blocks k (positions [k*block_size, (k+1)*block_size)) that lie inside the current length
    and hold only positions never retained again, ascending."""
    free = never_retained_again(seg_row, pol_row, horizon)
    return [k for k in range(len(free) // block_size) if free[k * block_size:(k + 1) * block_size].all()]
