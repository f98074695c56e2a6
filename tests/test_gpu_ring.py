"""GPU parity of ring storage (murmur_decode_step_ring) against the fp64 oracle.

Physical eviction (Section 3.2): the output tokens live in a ring of `cap` rows after the output sinks,
and every step appends the current token's K/V to its ring row inside the attention launch.  Each case
starts from the storage the oracle's literal appends give (oracle/ring.py), runs consecutive steps on
the GPU and checks, at every step, the attention against the oracle's attention over the sequence-ordered
cache (Equation 1 over Algorithm 1/2's retained set), the retained-set outputs against the oracle's rows,
and at the end the whole storage, bit for bit, against the oracle's appends.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import ring as OR
from paper_2606_01483_amd import murmur as M
from paper_2606_01483_amd import workloads as W
from paper_2606_01483_amd.decode import RingBatch
from _tol import REL_TOL, LSE_TOL, bf16_excess, lse_err, rel_err_fp32

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


def expand(ranges_row):
    out = []
    for start, length in ranges_row:
        out.extend(range(int(start), int(start) + int(length)))
    return out


def oracle_storage(wl, step0, cap):
    """The oracle's ring storage before step step0 (tokens 0 .. j-2 appended)."""
    seg = wl.seg(step0)
    seg[:, 3] -= 1
    n_so = wl.policy[:, 4]
    rows = max(OR.storage_len(seg[b], n_so[b], cap) for b in range(wl.batch))
    rows = (rows + 7) // 8 * 8
    return OR.append_all(wl.k, seg, n_so, cap, rows), OR.append_all(wl.v, seg, n_so, cap, rows), rows


def run_ring_case(wl, steps, cap, split_len=0, out_dtype=M.MURMUR_DTYPE_F32, threads=16):
    assert steps == list(range(steps[0], steps[0] + len(steps))), "ring steps must be consecutive"
    k_st, v_st, rows = oracle_storage(wl, steps[0], cap)
    rb = RingBatch(wl, cap, out_dtype=out_dtype, split_len=split_len, steps=steps, storage=(k_st, v_st))
    assert rb.rows == rows
    n_so = wl.policy[:, 4]
    for i, s in enumerate(steps):
        seg = wl.seg(s)
        rb.idx.fill_(-7)
        rb.step(i)
        torch.cuda.synchronize()
        assert M.murmur_device_error() == 0, f"device error at step {s}"
        idx, cnt = oracle.retained(seg, wl.policy)
        ref, ref_lse = oracle.attend(wl.q(s), wl.k, wl.v, idx, cnt, scale=wl.scale, n_threads=threads)
        y = rb.out.float().cpu().numpy()
        if out_dtype == M.MURMUR_DTYPE_F32:
            assert rel_err_fp32(y, ref) <= REL_TOL, f"step {s}"
        else:
            assert bf16_excess(y, ref) <= REL_TOL, f"step {s}"
        assert lse_err(rb.lse.cpu().numpy(), ref_lse) <= LSE_TOL, f"step {s}"
        # retained-set outputs, in storage rows
        g_cnt, g_idx, g_rng = rb.count.cpu().numpy(), rb.idx.cpu().numpy(), rb.ranges.cpu().numpy()
        assert np.array_equal(g_cnt, cnt)
        want_rows = OR.storage_rows(idx, cnt, seg, n_so, cap)
        for b in range(wl.batch):
            got = expand(g_rng[b])
            assert sorted(got) == sorted(want_rows[b]), f"step {s} sequence {b}"
            assert g_idx[b, :cnt[b]].tolist() == got
            assert np.all(g_idx[b, cnt[b]:] == -1)
    final_seg = wl.seg(steps[-1])
    want_k = OR.append_all(wl.k, final_seg, n_so, cap, rows)
    want_v = OR.append_all(wl.v, final_seg, n_so, cap, rows)
    assert np.array_equal(rb.k[0].view(torch.uint16).cpu().numpy(), want_k)
    assert np.array_equal(rb.v[0].view(torch.uint16).cpu().numpy(), want_v)
    return rb


def test_ring_tiny_all_steps():
    """Tiny workload, ring of exactly the output window (32): it wraps at every step."""
    announce("ring c1 all 16 steps, cap 32")
    wl = W.make("c1")
    run_ring_case(wl, list(range(16)), 32)


def test_ring_tiny_bf16_out():
    announce("ring c1 bf16 output, cap 40")
    wl = W.make("c1")
    run_ring_case(wl, list(range(8)), 40, out_dtype=M.MURMUR_DTYPE_BF16)


def test_ring_300s_chunks_with_eviction():
    """12 x 300 s chunks with eviction: output window 256 in a ring of 256 rows."""
    announce("ring c3 steps 0-5, cap 256")
    wl = W.make("c3", steps=6)
    run_ring_case(wl, list(range(6)), 256)


def ragged_workload(n_layers, steps, seed=77):
    rng = np.random.default_rng(seed)
    B = 6
    seg0 = np.stack([rng.integers(0, 12, B), rng.integers(20, 160, B), rng.integers(0, 6, B),
                     rng.integers(0, 50, B)], axis=1).astype(np.int32)
    w_o = np.array([5, 17, 32, 1, OFF, 60], dtype=np.int32)
    n_so = np.array([0, 2, 4, 3, 1, 0], dtype=np.int32)
    pol = np.stack([np.array([OFF, 40, 16, 7, 100, 25]), np.array([0, 3, 9, 0, 5, 1]),
                    np.array([0, 0, 4, 2, 0, 30]), w_o, n_so], axis=1).astype(np.int32)
    seg0[4, 3] = 0  # keep-all sequence: j - n_so stays within the ring over the steps
    return W.build("ring_ragged", 4242, n_layers, seg0, pol, steps, planted=False)


@pytest.mark.parametrize("n_layers,split_len", [(2, 0), (2, 64), (2, 512), (12, 512)])
def test_ring_ragged_policies_with_sinks(n_layers, split_len):
    """Six sequences with different layouts, windows (1 .. 60, and off) and sinks, a ring of 64 rows:
    wide-schedule splits (automatic and 64 positions), the LDS-staged kernel in one dispatch round and, with
    12 layers, over more than one round."""
    announce(f"ring ragged NL={n_layers} split_len={split_len}")
    wl = ragged_workload(n_layers, steps=40)
    # consecutive steps: every step appends its token, which later steps read
    run_ring_case(wl, list(range(12)) if n_layers > 2 else list(range(40)), 64, split_len=split_len)


def test_ring_capacity_error():
    """A ring smaller than a sequence's output window: that sequence gets count 0, NaN outputs, the
    capacity error bit and no append; the others are unaffected."""
    announce("ring capacity error")
    wl = ragged_workload(1, steps=4)
    cap = 50  # sequence 5 has an output window of 60
    k_st, v_st, rows = oracle_storage(wl, 0, 64)
    rb = RingBatch(wl, cap, out_dtype=M.MURMUR_DTYPE_F32, steps=[0], storage=(k_st, v_st))
    before = rb.k[0].clone()
    rb.step(0)
    torch.cuda.synchronize()
    code = M.murmur_device_error()
    assert code & M.MURMUR_DEVERR_CAPACITY
    y = rb.out.float().cpu().numpy()
    assert np.all(np.isnan(y[:, 5]))
    assert int(rb.count[5]) == 0
    assert torch.equal(rb.k[0][:, 5], before[:, 5])
    assert np.all(np.isfinite(y[:, :4]))


def test_ring_graph_replays_match_eager():
    """Four ring steps captured in a HIP graph, replayed three times (storage reset to the starting
    state before each replay, eager work in between): outputs and storage equal the eager run."""
    announce("ring graph replays")
    wl = ragged_workload(2, steps=4)
    k_st, v_st, _ = oracle_storage(wl, 0, 64)
    rb = RingBatch(wl, 64, out_dtype=M.MURMUR_DTYPE_F32, steps=[0, 1, 2, 3], storage=(k_st, v_st))
    k0, v0 = rb.k[0].clone(), rb.v[0].clone()
    for i in range(4):
        rb.step(i)
    torch.cuda.synchronize()
    want_out, want_k = rb.out.clone(), rb.k[0].clone()
    graph = torch.cuda.CUDAGraph()
    cap_stream = torch.cuda.Stream()
    cap_stream.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    with torch.cuda.graph(graph, stream=cap_stream):
        for i in range(4):
            rb.step(i)
    for _ in range(3):
        rb.k[0].copy_(k0)
        rb.v[0].copy_(v0)
        rb.out.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(rb.out, want_out)
        assert torch.equal(rb.k[0], want_k)
