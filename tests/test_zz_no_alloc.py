"""GPU: the allocation-free decode step (murmur_decode_step_static) against murmur_decode_step.

Both run the same kernels on the same inputs; the static variant keeps its tickets and split partials in the
library's per-device scratch array instead of a caller's workspace.  Two calls in a row, the second on a
smaller input (fewer sequences and splits, so it meets what the first left in the scratch), each compared
with murmur_decode_step bit for bit (outputs, lse, retained-set outputs) and with the fp64 oracle to the
fp32 bar; then the larger call captured into a HIP graph and replayed, with eager work between replays.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_01483_amd import murmur as M
from paper_2606_01483_amd import workloads as W
from paper_2606_01483_amd.decode import DecodeBatch
from _tol import REL_TOL, LSE_TOL, lse_err, rel_err_fp32

pytestmark = pytest.mark.gpu


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


def static_step(db, i, out, lse, sets, stream=None):
    idx, count, ranges = sets
    M.murmur_decode_step_static(db.seg[i], db.pol, db.pol_mode, db.q[i], db.kv[0], idx, count, ranges, db.max_keep,
                                db.B, db.Hq, db.Hkv, db.D, db.wl.scale, db.split_len, out, db.out_dtype, lse, stream)


def run_pair(wl, step, split_len=0):
    """murmur_decode_step, then murmur_decode_step_static on the same inputs; both results."""
    db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=[step], split_len=split_len)
    assert db.ws_bytes <= M.MURMUR_STATIC_SCRATCH_BYTES
    db.step_fused(0)
    out = torch.full_like(db.out, float("nan"))
    lse = torch.full_like(db.lse, float("nan"))
    sets = tuple(torch.full_like(t, -7) for t in db.sets[0])
    static_step(db, 0, out, lse, sets)
    torch.cuda.synchronize()
    assert M.murmur_device_error() == 0
    return db, out, lse, sets


def check_pair(wl, step, split_len=0):
    db, out, lse, sets = run_pair(wl, step, split_len)
    assert torch.equal(out, db.out) and torch.equal(lse, db.lse)
    for got, want in zip(sets, db.sets[0]):
        assert torch.equal(got, want)
    idx, cnt = oracle.retained(wl.seg(step), wl.policy, db.max_keep)
    assert np.array_equal(sets[0].cpu().numpy(), idx) and np.array_equal(sets[1].cpu().numpy(), cnt)
    ref, ref_lse = oracle.attend(wl.q(step), wl.k, wl.v, idx, cnt, scale=wl.scale, n_threads=16)
    assert rel_err_fp32(out.cpu().numpy(), ref) <= REL_TOL
    assert lse_err(lse.cpu().numpy(), ref_lse) <= LSE_TOL
    return db, out, lse, sets


def test_static_step_matches_workspace_step_twice():
    wl3 = W.make("c3", steps=2)
    announce("decode_step_static, 12 x 300 s chunks (48 groups of 5 splits)")
    check_pair(wl3, 1)
    wl1 = W.make("c1")
    announce("decode_step_static, tiny workload (4 groups of 3 splits), second call")
    check_pair(wl1, 7, split_len=64)


def test_static_step_graph_replays():
    wl = W.make("c3", steps=3)
    db, out, lse, sets = run_pair(wl, 2)
    eager_out, eager_lse = out.clone(), lse.clone()
    announce("decode_step_static captured into a graph")
    stream = torch.cuda.current_stream()
    cap = torch.cuda.Stream()
    cap.wait_stream(stream)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=cap):
        static_step(db, 0, out, lse, sets, stream=cap)
    torch.cuda.synchronize()
    small = DecodeBatch(W.make("c1"), out_dtype=M.MURMUR_DTYPE_F32, steps=[3], split_len=64)
    s_out, s_lse = torch.empty_like(small.out), torch.empty_like(small.lse)
    s_sets = tuple(torch.empty_like(t) for t in small.sets[0])
    for trial in range(3):
        out.fill_(float("nan"))
        lse.fill_(float("nan"))
        static_step(small, 0, s_out, s_lse, s_sets)  # eager use of the same scratch between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager_out) and torch.equal(lse, eager_lse), trial
    assert M.murmur_device_error() == 0
