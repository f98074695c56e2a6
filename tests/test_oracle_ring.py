"""Pins of the ring-storage oracle (oracle/ring.py) against Algorithm 1 and plain invariants (CPU only).

Ring storage is physical eviction (Section 3.2): a row is reused by a later output token.  What fixes
it is Algorithm 1 itself -- after the appends of tokens 0 .. j-1, every token the algorithm retains at
step j must still be in storage, in a row of its own -- and the special case of a ring that has not
wrapped, which is the plain sequence layout.
"""
import numpy as np
import pytest

import oracle
from oracle import ring as R

OFF = -1


def ids_cache(seg):
    """A [1, B, 1, L, 1] int64 cache whose entry at position p of sequence b is b * 10^6 + p."""
    seg = np.asarray(seg).reshape(-1, 4)
    L = int((seg[:, 0] + seg[:, 1] + seg[:, 2] + seg[:, 3]).max())
    B = seg.shape[0]
    ids = np.arange(B, dtype=np.int64)[:, None] * 10 ** 6 + np.arange(L, dtype=np.int64)[None, :]
    return ids.reshape(1, B, 1, L, 1)


def random_case(rng, window_on=True):
    p_pre, l_s, p_mid = (int(x) for x in rng.integers(0, 40, size=3))
    n_so = int(rng.integers(0, 6))
    if window_on:
        w_o = int(rng.integers(1, 40))
        cap = w_o + int(rng.integers(0, 10))
        j = int(rng.integers(1, 200))
    else:
        w_o = OFF
        j = int(rng.integers(1, 120))
        cap = max(1, j - n_so) + int(rng.integers(0, 10))
    pol = [OFF, 0, 0, w_o, n_so]
    return [p_pre, l_s, p_mid, j], pol, n_so, cap


def test_ring_row_is_identity_until_the_ring_wraps():
    for out0 in (0, 7, 1000):
        for n_so in (0, 1, 4):
            for cap in (1, 5, 64):
                for i0 in range(n_so + cap):
                    assert R.ring_row(i0, out0, n_so, cap) == out0 + i0
                # the next token reuses the first ring row
                assert R.ring_row(n_so + cap, out0, n_so, cap) == out0 + n_so


def test_unwrapped_ring_storage_equals_the_sequence_layout():
    rng = np.random.default_rng(7)
    for _ in range(50):
        seg, pol, n_so, cap = random_case(rng, window_on=False)
        logical = ids_cache([seg])
        rows = R.storage_len(seg, n_so, cap)
        st = R.append_all(logical, [seg], n_so, cap, rows)
        L = sum(seg)
        assert np.array_equal(st[0, 0, 0, :L, 0], logical[0, 0, 0, :L, 0])


@pytest.mark.parametrize("window_on", [True, False])
def test_every_retained_token_survives_the_appends(window_on):
    """Algorithm 1's retained set at step j is intact in ring storage after tokens 0 .. j-1 were
    appended, and its tokens occupy distinct rows (300 random layouts, policies and ring sizes)."""
    rng = np.random.default_rng(11 if window_on else 12)
    for _ in range(300):
        seg, pol, n_so, cap = random_case(rng, window_on)
        idx, cnt = oracle.retained(np.array([seg]), np.array(pol))
        logical = ids_cache([seg])
        st = R.append_all(logical, [seg], n_so, cap, R.storage_len(seg, n_so, cap))
        rows = R.storage_rows(idx, cnt, [seg], n_so, cap)[0]
        assert len(rows) == int(cnt[0]) == len(set(rows))
        got = st[0, 0, 0, rows, 0]
        want = logical[0, 0, 0, idx[0, :cnt[0]], 0]
        assert np.array_equal(got, want), (seg, pol, cap)


def test_a_ring_smaller_than_the_window_loses_a_retained_token():
    """cap < w is not enough: at some step a token inside Algorithm 1's window has been overwritten."""
    for w_o in (2, 5, 17):
        for n_so in (0, 3):
            for cap in range(1, w_o):
                lost = False
                for j in range(1, n_so + w_o + cap + 3):
                    seg = [4, 6, 0, j]
                    pol = [OFF, 0, 0, w_o, n_so]
                    idx, cnt = oracle.retained(np.array([seg]), np.array(pol))
                    logical = ids_cache([seg])
                    st = R.append_all(logical, [seg], n_so, cap, R.storage_len(seg, n_so, cap))
                    rows = R.storage_rows(idx, cnt, [seg], n_so, cap)[0]
                    if not np.array_equal(st[0, 0, 0, rows, 0], logical[0, 0, 0, idx[0, :cnt[0]], 0]):
                        lost = True
                        break
                assert lost, (w_o, n_so, cap)


def test_keep_all_outputs_needs_a_ring_as_long_as_the_outputs():
    """With output eviction off, the step after the ring is full loses the first ring token."""
    for n_so in (0, 2):
        for cap in (1, 4, 9):
            j = n_so + cap + 1
            seg = [3, 5, 0, j]
            idx, cnt = oracle.retained(np.array([seg]), np.array([OFF, 0, 0, OFF, n_so]))
            logical = ids_cache([seg])
            st = R.append_all(logical, [seg], n_so, cap, R.storage_len(seg, n_so, cap))
            rows = R.storage_rows(idx, cnt, [seg], n_so, cap)[0]
            assert len(set(rows)) < len(rows)
            assert not np.array_equal(st[0, 0, 0, rows, 0], logical[0, 0, 0, idx[0, :cnt[0]], 0])
