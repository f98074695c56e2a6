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
