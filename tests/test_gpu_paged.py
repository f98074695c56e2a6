"""GPU parity of the paged KV cache (murmur_evict_compact_paged + murmur_decode_attn over a block pool).

Every sequence's positions live in blocks of one shared pool placed by a random block table; the index list
the eviction emits is checked bit for bit against the oracle's retained positions mapped through the table
(oracle/paged.py), the pool the benchmark builds against the oracle's position-by-position copy, and the
attention against the oracle's Equation 1 over the sequence-ordered cache.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import paged as OP
from paper_2606_01483_amd import murmur as M
from paper_2606_01483_amd import workloads as W
from paper_2606_01483_amd.decode import PagedBatch
from _tol import REL_TOL, LSE_TOL, lse_err, rel_err_fp32

pytestmark = pytest.mark.gpu
OFF = -1


def announce(msg):
    print(f"\n[case] {msg}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    M.lib()
    yield
    torch.cuda.synchronize()
    assert M.murmur_device_error() == 0


def check_paged(wl, steps, block_size, layout, split_len=0):
    pb = PagedBatch(wl, block_size, layout=layout, out_dtype=M.MURMUR_DTYPE_F32, steps=steps, split_len=split_len,
                    seed=block_size)
    want_pool = OP.build_pool(wl.k, pb.lengths, pb.block_table, block_size, pb.n_blocks)
    got = pb.k[0].view(torch.uint16).cpu().numpy()
    if layout != "flash":
        got = got.transpose(0, 2, 1, 3)
    assert np.array_equal(got, want_pool)
    for i, s in enumerate(steps):
        announce(f"paged {wl.name} step {s} block {block_size} layout {layout} split_len {split_len}")
        pb.idx.fill_(-7)
        pb.step(i)
        torch.cuda.synchronize()
        assert M.murmur_device_error() == 0
        idx, cnt = oracle.retained(wl.seg(s), wl.policy, pb.max_keep)
        assert np.array_equal(pb.count.cpu().numpy(), cnt)
        assert np.array_equal(pb.idx.cpu().numpy(), OP.rows_of(idx, cnt, pb.block_table, block_size))
        ref, ref_lse = oracle.attend(wl.q(s), wl.k, wl.v, idx, cnt, scale=wl.scale, n_threads=16)
        assert rel_err_fp32(pb.out.float().cpu().numpy(), ref) <= REL_TOL
        assert lse_err(pb.lse.cpu().numpy(), ref_lse) <= LSE_TOL


@pytest.mark.parametrize("block_size,layout", [(16, "flash"), (1, "flash"), (64, "head"), (16, "head")])
def test_paged_tiny(block_size, layout):
    check_paged(W.make("c1"), [0, 7, 15], block_size, layout)


@pytest.mark.parametrize("split_len", [0, 512])
def test_paged_300s_chunks_with_eviction(split_len):
    check_paged(W.make("c3", steps=4), [0, 3], 16, "flash", split_len)


def test_paged_28_layers():
    """Several layers in one pool per layer (layer stride), ragged sequences, per-sequence policies."""
    rng = np.random.default_rng(3)
    B = 5
    seg0 = np.stack([rng.integers(0, 40, B), rng.integers(100, 700, B), rng.integers(0, 9, B),
                     rng.integers(1, 300, B)], axis=1).astype(np.int32)
    pol = np.stack([np.array([64, OFF, 200, 33, OFF]), rng.integers(0, 50, B), rng.integers(0, 6, B),
                    np.array([40, 100, OFF, 7, 256]), rng.integers(0, 4, B)], axis=1).astype(np.int32)
    wl = W.build("paged_ragged", 99, 6, seg0, pol, 3, planted=False)
    check_paged(wl, [0, 2], 32, "flash")


def test_paged_block_table_too_short():
    """A retained position past the table's blocks: entry -1 and MURMUR_DEVERR_BLOCK; the attention then
    reports the position (NaN outputs)."""
    announce("paged block table too short")
    wl = W.make("c1")
    pb = PagedBatch(wl, 16, out_dtype=M.MURMUR_DTYPE_F32, steps=[0])
    short = pb.max_blocks - 2  # the last two blocks of the sequence are missing
    M.murmur_evict_compact_paged(pb.seg[0], pb.pol, 1, pb.B, pb.bt, short, pb.bs, pb.idx, pb.max_keep, pb.count)
    torch.cuda.synchronize()
    code = M.murmur_device_error()
    assert code & M.MURMUR_DEVERR_BLOCK
    idx = pb.idx.cpu().numpy()[0, :int(pb.count[0])]
    assert np.any(idx == -1)
    pb.attend(0)
    torch.cuda.synchronize()
    assert M.murmur_device_error() & M.MURMUR_DEVERR_POSITION
    assert np.all(np.isnan(pb.out.float().cpu().numpy()))
