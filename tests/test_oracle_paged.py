"""Pins of the paged-cache oracle (oracle/paged.py) against its definition's special cases (CPU only)."""
import numpy as np

from oracle import paged as P


def test_identity_table_gives_the_positions():
    for bs in (1, 4, 16):
        table = np.arange(64)
        for p in range(64 * bs):
            assert P.pool_row(table, bs, p) == p


def test_pool_round_trip_through_any_table():
    """Every position read back through its block table equals the sequence-ordered cache."""
    rng = np.random.default_rng(0)
    for bs in (1, 8, 16):
        B, L = 3, 70
        nb = -(-L // bs)
        perm = rng.permutation(B * nb + 5)[:B * nb].reshape(B, nb)
        cache = rng.integers(1, 1000, size=(2, B, 2, L, 3)).astype(np.int32)
        lengths = [70, 33, 1]
        pool = P.build_pool(cache, lengths, perm, bs, B * nb + 5)
        for b in range(B):
            for p in range(lengths[b]):
                assert np.array_equal(pool[:, P.pool_row(perm[b], bs, p)], cache[:, b, :, p])


def test_rows_of_keeps_padding():
    idx = np.array([[0, 5, 17, -1]], dtype=np.int32)
    rows = P.rows_of(idx, np.array([3]), np.array([[4, 2]]), 16)
    assert rows.tolist() == [[64, 69, 33, -1]]


# Hand-worked (from Algorithms 1 and 2 under the readings: window of w tokens starting at
# l_j = max(0, j - max(d,1) + 1), output window [j - w, j) in 0-based output indices): the tiny workload
# (prompt 32, speech 450, speech window 128, delay 72, output window 32, no sinks) at step j = 80.
# Speech: l_80 = 80 - 72 + 1 = 9, so speech tokens 0..8 (positions 32..40) are behind the window for good.
# Output: output tokens 0..47 (positions 482..529) are older than the window [48, 80).
# Blocks of 4 inside [32, 41): 8, 9; inside [482, 530): 121 .. 131.
TINY_SEG = [32, 450, 0, 80]
TINY_POL = [128, 72, 0, 32, 0]


def test_freeable_blocks_hand_worked():
    assert P.freeable_blocks(TINY_SEG, TINY_POL, 4) == [8, 9] + list(range(121, 132))
    free = P.never_retained_again(TINY_SEG, TINY_POL)
    assert free.nonzero()[0].tolist() == list(range(32, 41)) + list(range(482, 530))


def test_freeable_blocks_special_cases():
    # eviction off: nothing is ever freed
    assert P.freeable_blocks([8, 40, 3, 50], [-1, 0, 0, -1, 0], 1) == []
    # sinks stay: speech sinks 4, output sinks 2 (block size 1 gives the positions)
    got = P.freeable_blocks([2, 30, 1, 20], [8, 5, 4, 6, 2], 1)
    l_j = min(20 - 5 + 1, 30 - 8)
    assert got == list(range(2 + 4, 2 + l_j)) + list(range(33 + 2, 33 + 20 - 6))
    # window clamped at the end of speech: the window stops moving, nothing behind it comes back
    assert P.freeable_blocks([0, 10, 0, 100], [4, 1, 0, -1, 0], 1) == list(range(0, 6))


def test_freeable_blocks_grow_and_horizon_is_enough():
    rng = np.random.default_rng(5)
    for _ in range(40):
        seg = [int(rng.integers(0, 6)), int(rng.integers(1, 60)), int(rng.integers(0, 4)), int(rng.integers(1, 50))]
        pol = [int(rng.choice([-1, rng.integers(1, 20)])), int(rng.integers(0, 12)), int(rng.integers(0, 5)),
               int(rng.choice([-1, rng.integers(1, 15)])), int(rng.integers(0, 4))]
        bs = int(rng.choice([1, 2, 4, 8]))
        a = P.freeable_blocks(seg, pol, bs)
        later = P.freeable_blocks(seg[:3] + [seg[3] + 3], pol, bs)
        assert set(a) <= set(later)
        assert a == P.freeable_blocks(seg, pol, bs, horizon=3 * P.default_horizon(seg, pol))
