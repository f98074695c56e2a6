"""Paged KV cache addressing -- TEST INFRASTRUCTURE (oracle side).

Only ``tests/`` may import this module; it imports nothing from the GPU package.

A paged cache (the block tables of a paged-attention engine such as vLLM, the engine the paper also runs
on, Section 3.1) keeps every sequence's positions in fixed-size blocks of one shared pool: position p of
sequence b lives in pool row ``block_table[b][p // block_size] * block_size + p % block_size``.  Plain
definitions, run literally:

  * ``pool_row``    -- that row;
  * ``build_pool``  -- a pool [NL, rows, Hkv, D] filled from a sequence-ordered cache by copying every
                       position to its row one by one;
  * ``rows_of``     -- the pool rows of a list of retained positions.

Pins (``tests/test_oracle_paged.py``): with the identity table of one sequence the pool row is the
position; a pool built from any table reproduces the sequence-ordered cache at every position read back
through the table.
"""
from __future__ import annotations

import numpy as np


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
