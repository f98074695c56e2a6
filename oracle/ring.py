"""Ring storage of the output tokens -- TEST INFRASTRUCTURE (oracle side).

Only ``tests/`` may import this module; it imports nothing from the GPU package.

Physical eviction (paper, Section 3.2: an entry Algorithm 1 evicts leaves the
KV cache).  The output region of a sequence keeps its output sinks in rows
``out0 .. out0 + n_sink - 1`` and every later output token in a ring of ``cap``
rows after them: token ``i`` (0-based, ``i >= n_sink``) is written to row
``out0 + n_sink + (i - n_sink) mod cap``, overwriting whatever token held that
row.  Prompt and speech rows keep their positions.  These are plain
definitions, run literally:

  * ``ring_row``      -- the row a token is written to;
  * ``append_all``    -- the storage after prefill and the appends of output
                         tokens 0 .. j-1 in generation order (last writer wins);
  * ``storage_rows``  -- the storage rows of a list of retained positions.

Pins (``tests/test_oracle_ring.py``): the ring is the identity while it has not
wrapped, every token Algorithm 1 retains still holds its own K/V row after the
appends whenever the ring fits the window (and some retained token is lost for
every ring smaller than the window), and retained tokens never share a row.
"""
from __future__ import annotations

import numpy as np


def ring_row(i0: int, out0: int, n_sink: int, cap: int) -> int:
    """Storage row of 0-based output token i0 of a sequence whose output region starts at out0."""
    if i0 < n_sink:
        return out0 + i0
    return out0 + n_sink + (i0 - n_sink) % cap


def storage_len(seg_row, n_sink: int, cap: int) -> int:
    """Rows of ring storage one sequence needs: prompts, speech, output sinks and the ring."""
    p_pre, l_s, p_mid, _ = (int(x) for x in seg_row)
    return p_pre + l_s + p_mid + n_sink + cap


def append_all(logical: np.ndarray, seg: np.ndarray, n_sink, cap: int, rows: int) -> np.ndarray:
    """Ring storage after all appends.

    logical: [NL, B, Hkv, L, D] cache in sequence positions (any dtype);
    seg: int [B, 4] (prompt_pre, speech_len, prompt_mid, out_len j): tokens 0 .. j-1 have been appended;
    n_sink: output sinks, one int or one per sequence; cap: ring rows; rows: storage rows per sequence.
    Rows no token was written to hold zeros.
    """
    seg = np.asarray(seg).reshape(-1, 4)
    NL, B, Hkv, L, D = logical.shape
    sinks = np.broadcast_to(np.asarray(n_sink), (B,))
    st = np.zeros((NL, B, Hkv, rows, D), dtype=logical.dtype)
    for b in range(B):
        p_pre, l_s, p_mid, j = (int(x) for x in seg[b])
        out0 = p_pre + l_s + p_mid
        st[:, b, :, :out0] = logical[:, b, :, :out0]  # prefill: prompts and speech in place
        for i0 in range(j):  # generation order: a later token overwrites an earlier one's row
            st[:, b, :, ring_row(i0, out0, int(sinks[b]), cap)] = logical[:, b, :, out0 + i0]
    return st


def storage_rows(idx: np.ndarray, count: np.ndarray, seg: np.ndarray, n_sink, cap: int) -> list[list[int]]:
    """The storage row of every retained position (positions of idx[b, :count[b]], same order)."""
    seg = np.asarray(seg).reshape(-1, 4)
    B = seg.shape[0]
    sinks = np.broadcast_to(np.asarray(n_sink), (B,))
    out = []
    for b in range(B):
        p_pre, l_s, p_mid, _ = (int(x) for x in seg[b])
        out0 = p_pre + l_s + p_mid
        rows = []
        for p in idx[b, :int(count[b])].tolist():
            rows.append(p if p < out0 else ring_row(p - out0, out0, int(sinks[b]), cap))
        out.append(rows)
    return out
