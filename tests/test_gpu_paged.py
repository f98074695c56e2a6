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
from paper_2606_01483_amd.decode import DevicePagedBatch, PagedBatch, RecyclingPagedBatch
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
    """28 layers, one pool per layer (layer stride), ragged sequences, per-sequence policies."""
    rng = np.random.default_rng(3)
    B = 5
    seg0 = np.stack([rng.integers(0, 40, B), rng.integers(100, 700, B), rng.integers(0, 9, B),
                     rng.integers(1, 300, B)], axis=1).astype(np.int32)
    pol = np.stack([np.array([64, OFF, 200, 33, OFF]), rng.integers(0, 50, B), rng.integers(0, 6, B),
                    np.array([40, 100, OFF, 7, 256]), rng.integers(0, 4, B)], axis=1).astype(np.int32)
    wl = W.build("paged_ragged", 99, 28, seg0, pol, 3, planted=False)
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


def test_paged_row_beyond_int32_is_a_device_error():
    """A block-table entry whose pool row does not fit in 32 bits (block number 2^27 with blocks of 16): the
    eviction writes -1 and reports MURMUR_DEVERR_BLOCK instead of wrapping into the pool, and the attention
    reports the position (NaN outputs for that sequence)."""
    announce("paged row beyond 2^31")
    wl = W.make("c1")
    pb = PagedBatch(wl, 16, out_dtype=M.MURMUR_DTYPE_F32, steps=[0])
    bt = pb.block_table.copy()
    bt[0, 0] = 1 << 27  # the prompt's first block: always retained; 2^27 * 16 = 2^31
    pb.bt.copy_(torch.from_numpy(bt))
    pb.step(0)
    torch.cuda.synchronize()
    code = M.murmur_device_error()
    assert code & M.MURMUR_DEVERR_BLOCK and code & M.MURMUR_DEVERR_POSITION
    assert np.all(pb.idx.cpu().numpy()[0, :16] == -1)
    assert np.all(np.isnan(pb.out.float().cpu().numpy()))


def recycling_workload(steps):
    """Three sequences whose speech window (48 tokens, delay 20, 4 sinks) and output window (40, 2 sinks)
    move over the whole decode; the third keeps everything (eviction off), so its blocks are never freed."""
    seg0 = np.array([[16, 200, 4, 10], [30, 170, 0, 25], [8, 60, 2, 5]], dtype=np.int32)
    pol = np.array([[48, 20, 4, 40, 2], [32, 5, 0, 24, 0], [-1, 0, 0, -1, 0]], dtype=np.int32)
    return W.build("paged_recycle", 515, 2, seg0, pol, steps, planted=False, hq=8, hkv=2)


@pytest.mark.parametrize("block_size", [16, 4])
def test_paged_recycling_bounds_the_pool(block_size):
    """A 200-step decode on a pool that cannot hold the whole cache: before each step the blocks that no
    later step retains are freed (filled with NaN) and new positions reuse them.  Every step matches the
    oracle's attention over the sequence-ordered cache with no device error (no freed block is read), and
    the pool never needs more than prompt + speech + sinks + output window, plus two partial blocks per
    freed range, per sequence."""
    steps = 200
    wl = recycling_workload(steps)
    seg_last = wl.seg(steps - 1)
    pol = wl.policy
    # what each sequence may hold at once: prompts, speech, output sinks and window (the whole output when
    # output eviction is off), rounded up to blocks, plus the blocks two freed ranges can leave partly used
    cap = 0
    for b in range(wl.batch):
        p_pre, l_s, p_mid, j = (int(x) for x in seg_last[b])
        outs = j if pol[b, 3] < 0 else int(pol[b, 4]) + int(pol[b, 3])
        cap += -(-(p_pre + l_s + p_mid + outs) // block_size) + 4
    without = int((-(-seg_last.sum(axis=1) // block_size)).sum())
    assert cap < without
    announce(f"paged recycling block {block_size}: pool {cap} blocks, {without} without freeing")
    pb = RecyclingPagedBatch(wl, block_size, cap)
    freed_total = 0
    for s in range(steps):
        blocks = pb.prepare(s)
        freed_total = int(blocks[:, :, 1].sum())
        pb.idx.fill_(-7)
        pb.step(s)
        torch.cuda.synchronize()
        assert M.murmur_device_error() == 0, f"step {s}"
        idx, cnt = oracle.retained(wl.seg(s), wl.policy, pb.max_keep)
        assert np.array_equal(pb.count.cpu().numpy(), cnt)
        assert np.array_equal(pb.idx.cpu().numpy(), OP.rows_of(idx, cnt, pb.table, block_size))
        ref, ref_lse = oracle.attend(wl.q(s), wl.k, wl.v, idx, cnt, scale=wl.scale, n_threads=16)
        assert rel_err_fp32(pb.out.float().cpu().numpy(), ref) <= REL_TOL, f"step {s}"
        assert lse_err(pb.lse.cpu().numpy(), ref_lse) <= LSE_TOL, f"step {s}"
    assert pb.peak_in_use <= cap
    assert freed_total > 0 and pb.peak_in_use < without
    assert not pb.freed[2].any()  # eviction off: nothing of the third sequence is freed


def test_paged_freed_block_is_a_device_error():
    """A retained position whose block the table marks freed (-1): the eviction reports
    MURMUR_DEVERR_BLOCK and writes -1, the attention then gives NaN for that sequence only."""
    wl = recycling_workload(4)
    pb = RecyclingPagedBatch(wl, 16, 200)
    pb.prepare(0)
    pb.table[1, 0] = -1  # the prompt of sequence 1 is always retained
    pb.bt.copy_(torch.from_numpy(pb.table))
    announce("paged freed block read")
    pb.step(0)
    torch.cuda.synchronize()
    code = M.murmur_device_error()
    assert code & M.MURMUR_DEVERR_BLOCK and code & M.MURMUR_DEVERR_POSITION
    assert np.all(pb.idx[1, :16].cpu().numpy() == -1)
    y = pb.out.float().cpu().numpy()
    assert np.all(np.isnan(y[:, 1])) and np.all(np.isfinite(y[:, 0])) and np.all(np.isfinite(y[:, 2]))


def manager_model(seg, pol, bs, table, stack):
    """The device block manager's step, written out: sequences in order push their still-allocated blocks
    that the oracle finds freeable (blocks holding only positions no later step retains, from the oracle's
    literal Algorithm 1/2 loops, ascending: speech blocks before output blocks), then those whose current
    token's block is missing pop from the top of the stack in the same order."""
    for b in range(seg.shape[0]):
        for blk in OP.freeable_blocks(seg[b], pol[b], bs):
            if blk < table.shape[1] and table[b, blk] >= 0:
                stack.append(int(table[b, blk]))
                table[b, blk] = -1
    take = [b for b in range(seg.shape[0]) if table[b, (int(seg[b].sum()) - 1) // bs] < 0]
    for i, b in enumerate(take):
        table[b, (int(seg[b].sum()) - 1) // bs] = stack[len(stack) - 1 - i]
    del stack[len(stack) - len(take):]


def device_state(pb):
    top = int(pb.top.item())
    return pb.bt.cpu().numpy(), pb.stack[:top].cpu().numpy().tolist()


@pytest.mark.parametrize("block_size", [16, 4])
def test_device_block_manager_loop(block_size):
    """200 steps with the block manager on the device (murmur_paged_step: free, allocate, append the current
    K/V), on a pool smaller than the whole cache: every step's attention matches the oracle, the block table
    and free stack equal the manager's rule written out on the host, and every block is either in use or on
    the stack exactly once."""
    steps = 200
    wl = recycling_workload(steps)
    seg_last = wl.seg(steps - 1)
    cap = 0
    for b in range(wl.batch):
        p_pre, l_s, p_mid, j = (int(x) for x in seg_last[b])
        outs = j if wl.policy[b, 3] < 0 else int(wl.policy[b, 4]) + int(wl.policy[b, 3])
        cap += -(-(p_pre + l_s + p_mid + outs) // block_size) + 4
    announce(f"device block manager, block {block_size}, pool {cap} blocks")
    pb = DevicePagedBatch(wl, block_size, cap)
    table, stack = device_state(pb)
    table = table.copy()
    for s in range(steps):
        pb.step(s)
        torch.cuda.synchronize()
        assert M.murmur_device_error() == 0, f"step {s}"
        manager_model(wl.seg(s), wl.policy, block_size, table, stack)
        got_table, got_stack = device_state(pb)
        assert np.array_equal(got_table, table), f"step {s}"
        assert got_stack == stack, f"step {s}"
        used = got_table[got_table >= 0].tolist()
        assert sorted(used + got_stack) == list(range(cap)), f"step {s}"
        idx, cnt = oracle.retained(wl.seg(s), wl.policy, pb.max_keep)
        assert np.array_equal(pb.idx.cpu().numpy(), OP.rows_of(idx, cnt, got_table, block_size))
        ref, ref_lse = oracle.attend(wl.q(s), wl.k, wl.v, idx, cnt, scale=wl.scale, n_threads=16)
        assert rel_err_fp32(pb.out.float().cpu().numpy(), ref) <= REL_TOL, f"step {s}"
        assert lse_err(pb.lse.cpu().numpy(), ref_lse) <= LSE_TOL, f"step {s}"


def test_device_block_manager_graph_replays():
    """Twelve steps (three launches each) captured into one HIP graph, replayed three times from the starting
    state with eager work in between: outputs, pool, block table and free stack equal the eager run."""
    wl = recycling_workload(12)
    pb = DevicePagedBatch(wl, 8, 200)
    start = pb.state()
    for i in range(12):
        pb.step(i)
    torch.cuda.synchronize()
    assert M.murmur_device_error() == 0
    want = (pb.out.clone(), pb.lse.clone()) + pb.state()
    announce("device block manager graph replays")
    pb.restore(start)
    graph = torch.cuda.CUDAGraph()
    cap_stream = torch.cuda.Stream()
    cap_stream.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    with torch.cuda.graph(graph, stream=cap_stream):
        for i in range(12):
            pb.step(i)
    for _ in range(3):
        pb.restore(start)
        pb.out.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = (pb.out, pb.lse) + (pb.k, pb.v, pb.bt, pb.stack, pb.top)
        for g, w in zip(got, want):
            assert torch.equal(g, w)
    assert M.murmur_device_error() == 0


def test_device_block_manager_pool_exhausted():
    """A pool one block short: the sequence that finds the stack empty gets MURMUR_DEVERR_POOL, its table
    entry stays -1 and its attention is NaN (reported as a bad position); the others are unaffected."""
    wl = recycling_workload(40)
    seg0 = wl.seg(0)
    prefill = int(sum(-(-(int(seg0[b].sum()) - 1) // 16) for b in range(wl.batch)))
    pb = DevicePagedBatch(wl, 16, prefill)  # no block left for a new one
    announce("device block manager, pool exhausted")
    hit = None
    for s in range(40):
        pb.step(s)
        torch.cuda.synchronize()
        code = M.murmur_device_error()
        if code:
            hit = (s, code)
            break
    assert hit is not None, "some sequence must need a new block within 40 steps"
    s, code = hit
    assert code & M.MURMUR_DEVERR_POOL
    y = pb.out.float().cpu().numpy()
    bad = [b for b in range(wl.batch) if np.isnan(y[:, b]).all()]
    assert len(bad) >= 1 and all(np.isfinite(y[:, b]).all() for b in range(wl.batch) if b not in bad)


def test_device_block_manager_many_sequences():
    """600 ragged sequences (three chunks of 256 in the manager's workgroup), 30 steps: the table and stack
    equal the host rule at every step, with the K/V append (DevicePagedBatch) and, on a copy of the state,
    without a pool (bookkeeping only); attention parity at the first and last step."""
    rng = np.random.default_rng(606)
    B, steps = 600, 30
    seg0 = np.stack([rng.integers(0, 8, B), rng.integers(20, 90, B), rng.integers(0, 4, B), rng.integers(1, 30, B)],
                    axis=1).astype(np.int32)
    pol = np.stack([np.where(rng.random(B) < 0.2, OFF, rng.integers(4, 24, B)), rng.integers(0, 8, B),
                    rng.integers(0, 4, B), np.where(rng.random(B) < 0.2, OFF, rng.integers(2, 16, B)),
                    rng.integers(0, 3, B)], axis=1).astype(np.int32)
    wl = W.build("paged_many", 607, 1, seg0, pol, steps, planted=False, hq=4, hkv=1)
    bs = 8
    last = wl.seg(steps - 1)
    cap = int((-(-last.sum(axis=1) // bs)).sum())  # room for everything: exhaustion is not the point here
    announce(f"device block manager, {B} sequences")
    pb = DevicePagedBatch(wl, bs, cap)
    table, stack = device_state(pb)
    table = table.copy()
    bt2, stack2, top2 = pb.bt.clone(), pb.stack.clone(), pb.top.clone()
    for s in range(steps):
        M.murmur_paged_step(pb.seg[s], pb.pol, 1, B, bt2, pb.max_blocks, bs, stack2, top2, pb.n_blocks, s == 0)
        pb.step(s)
        torch.cuda.synchronize()
        assert M.murmur_device_error() == 0, f"step {s}"
        manager_model(wl.seg(s), wl.policy, bs, table, stack)
        got_table, got_stack = device_state(pb)
        assert np.array_equal(got_table, table), f"step {s}"
        assert got_stack == stack, f"step {s}"
        assert np.array_equal(bt2.cpu().numpy(), table), f"step {s} (no pool)"
        assert stack2[:int(top2.item())].cpu().numpy().tolist() == stack, f"step {s} (no pool)"
        if s in (0, steps - 1):
            idx, cnt = oracle.retained(wl.seg(s), wl.policy, pb.max_keep)
            ref, ref_lse = oracle.attend(wl.q(s), wl.k, wl.v, idx, cnt, scale=wl.scale, n_threads=16)
            assert rel_err_fp32(pb.out.float().cpu().numpy(), ref) <= REL_TOL, f"step {s}"
            assert lse_err(pb.lse.cpu().numpy(), ref_lse) <= LSE_TOL, f"step {s}"
