"""GPU parity of per-layer eviction policies (MURMUR_POL_PER_LAYER) against the fp64 oracle.

The paper finds the speech sparsity that eviction exploits on 24 of its model's 28 layers (Section 1,
Section 2.3), so a decoder may keep some layers dense.  With per-layer policies the fused step computes
each layer's retained set from that layer's policy and writes one evict_compact output set per layer;
the oracle evaluates every layer with its own policy (Algorithm 1 / Algorithm 2 as written) and Equation 1.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import ring as OR
from paper_2606_01483_amd import murmur as M
from paper_2606_01483_amd import workloads as W
from paper_2606_01483_amd.decode import DecodeBatch, RingBatch
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


def expand(ranges_row):
    out = []
    for start, length in ranges_row:
        out.extend(range(int(start), int(start) + int(length)))
    return out


def oracle_layers(wl, step, layers, batch=None):
    """Per layer: the oracle's retained set under that layer's policy and Equation 1 over it."""
    seg = wl.seg(step)
    q = wl.q(step)
    outs, lses, sets = [], [], []
    for layer in layers:
        pol = wl.policy[layer]
        idx, cnt = oracle.retained(seg, pol)
        sl = slice(layer, layer + 1)
        qq, kk, vv, ii, cc = q[sl], wl.k[sl], wl.v[sl], idx, cnt
        if batch is not None:
            qq, kk, vv, ii, cc = qq[:, batch], kk[:, batch], vv[:, batch], idx[batch], cnt[batch]
        o, l = oracle.attend(qq, kk, vv, ii, cc, scale=wl.scale, n_threads=16)
        outs.append(o)
        lses.append(l)
        sets.append((idx, cnt))
    return np.concatenate(outs), np.concatenate(lses), sets


def mixed_workload(n_layers=6, steps=3, seed=31):
    """Four sequences, six layers: dense layers, layers with only speech or only output eviction, and
    layers with both, with different windows, delays and sinks per layer and sequence."""
    rng = np.random.default_rng(seed)
    B = 4
    seg0 = np.stack([rng.integers(8, 40, B), rng.integers(300, 900, B), rng.integers(0, 8, B),
                     rng.integers(50, 400, B)], axis=1).astype(np.int32)
    pol = np.zeros((n_layers, B, 5), dtype=np.int32)
    for layer in range(n_layers):
        for b in range(B):
            kind = (layer + b) % 4
            w_s = OFF if kind in (0, 2) else int(rng.integers(16, 300))
            w_o = OFF if kind in (0, 1) else int(rng.integers(1, 200))
            pol[layer, b] = [w_s, int(rng.integers(0, 300)), int(rng.integers(0, 8)), w_o, int(rng.integers(0, 6))]
    return W.build("mixed_layers", 555, n_layers, seg0, pol, steps, planted=False)


@pytest.mark.parametrize("split_len", [0, 64, 512])
def test_per_layer_policies(split_len):
    """Every layer against the oracle with its own policy; the per-layer retained-set outputs bit for bit."""
    wl = mixed_workload()
    db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=[0, 2], split_len=split_len)
    assert db.per_layer
    for i, s in enumerate([0, 2]):
        announce(f"per-layer policies step {s} split_len {split_len}")
        for t in db.sets[0]:
            t.fill_(-7)
        db.step_fused(i)
        torch.cuda.synchronize()
        ref, ref_lse, sets = oracle_layers(wl, s, range(wl.n_layers))
        y = db.out.float().cpu().numpy()
        assert rel_err_fp32(y, ref) <= REL_TOL
        assert lse_err(db.lse.cpu().numpy(), ref_lse) <= LSE_TOL
        idx, cnt, rng = (t.cpu().numpy() for t in db.sets[0])
        for layer, (ref_idx, ref_cnt) in enumerate(sets):
            rows = slice(layer * wl.batch, (layer + 1) * wl.batch)
            assert np.array_equal(cnt[rows], ref_cnt)
            width = ref_idx.shape[1]
            assert np.array_equal(idx[rows, :width], ref_idx)
            assert np.all(idx[rows, width:] == -1)
            for b in range(wl.batch):
                assert expand(rng[layer * wl.batch + b]) == ref_idx[b, :ref_cnt[b]].tolist()


def test_per_layer_without_per_sequence():
    """MURMUR_POL_PER_LAYER alone: one policy per layer shared by every sequence ([NL][1][5])."""
    announce("per-layer policies shared by the sequences")
    wl0 = mixed_workload()
    pol = np.ascontiguousarray(wl0.policy[:, :1, :])  # [NL, 1, 5]
    wl = W.with_policy(wl0, np.repeat(pol, wl0.batch, axis=1))  # the same policies, per sequence, for the oracle
    db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=[1])
    pol_d = torch.from_numpy(pol).cuda()
    M.murmur_decode_step(db.seg[0], pol_d, M.MURMUR_POL_PER_LAYER, db.q[0], db.kv[0], None, None, None, db.max_keep,
                         db.B, db.Hq, db.Hkv, db.D, wl.scale, 0, db.out, db.out_dtype, db.lse, db.ws, db.ws_bytes)
    torch.cuda.synchronize()
    ref, ref_lse, _ = oracle_layers(wl, 1, range(wl.n_layers))
    assert rel_err_fp32(db.out.float().cpu().numpy(), ref) <= REL_TOL
    assert lse_err(db.lse.cpu().numpy(), ref_lse) <= LSE_TOL


def test_28_layers_four_dense_full():
    """c5 with its first four layers dense, at full size, at the first, middle and last of its 256 steps: every
    layer, sequence and head of the fp32 output and the lse against the oracle (each layer under its own
    policy), and the per-layer retained-set outputs bit for bit."""
    wl = W.make("c5_layers")
    steps = [0, wl.steps // 2, wl.steps - 1]
    db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=steps)
    for i, s in enumerate(steps):
        announce(f"c5_layers step {s}")
        for t in db.sets[0]:
            t.fill_(-7)
        db.out.fill_(float("nan"))
        db.step_fused(i)
        torch.cuda.synchronize()
        ref, ref_lse, sets = oracle_layers(wl, s, range(wl.n_layers))
        y = db.out.cpu().numpy().astype(np.float64)
        e = rel_err_fp32(y, ref)
        print(f"  max rel err {e:.3e}  lse err {lse_err(db.lse.cpu().numpy(), ref_lse):.3e}", flush=True)
        assert e <= REL_TOL
        assert lse_err(db.lse.cpu().numpy(), ref_lse) <= LSE_TOL
        idx, cnt, rng = (t.cpu().numpy() for t in db.sets[0])
        for layer, (ref_idx, ref_cnt) in enumerate(sets):
            rows = slice(layer * wl.batch, (layer + 1) * wl.batch)
            assert np.array_equal(cnt[rows], ref_cnt), layer
            width = ref_idx.shape[1]
            assert np.array_equal(idx[rows, :width], ref_idx), layer
            assert np.all(idx[rows, width:] == -1), layer


def test_ring_with_per_layer_policies():
    """Ring storage with per-layer policies (one output sink count per sequence, a ring that holds the
    longest window of any layer): consecutive steps, storage bit for bit at the end."""
    announce("ring + per-layer policies")
    rng = np.random.default_rng(2)
    B, NL, steps = 3, 4, 12
    seg0 = np.stack([rng.integers(0, 10, B), rng.integers(30, 120, B), rng.integers(0, 4, B),
                     rng.integers(0, 20, B)], axis=1).astype(np.int32)
    n_so = np.array([0, 2, 1], dtype=np.int32)
    pol = np.zeros((NL, B, 5), dtype=np.int32)
    windows = [[5, 9, 16], [OFF, OFF, OFF], [1, 30, 7], [12, 12, 12]]
    for layer in range(NL):
        for b in range(B):
            pol[layer, b] = [OFF if layer == 1 else 20 + 7 * layer, 3, 0, windows[layer][b], n_so[b]]
    wl = W.build("ring_layers", 808, NL, seg0, pol, steps, planted=False)
    cap = 40  # >= every window; keep-all layer 1: j - n_so <= 20 + 12
    seg_before = wl.seg(0)
    seg_before[:, 3] -= 1
    rows = max(OR.storage_len(seg_before[b], n_so[b], cap) for b in range(B))
    rows = (rows + 7) // 8 * 8
    st = (OR.append_all(wl.k, seg_before, n_so, cap, rows), OR.append_all(wl.v, seg_before, n_so, cap, rows))
    rb = RingBatch(wl, cap, out_dtype=M.MURMUR_DTYPE_F32, steps=list(range(steps)), storage=st)
    for s in range(steps):
        rb.step(s)
        torch.cuda.synchronize()
        assert M.murmur_device_error() == 0
        ref, ref_lse, sets = oracle_layers(wl, s, range(NL))
        assert rel_err_fp32(rb.out.float().cpu().numpy(), ref) <= REL_TOL, f"step {s}"
        assert lse_err(rb.lse.cpu().numpy(), ref_lse) <= LSE_TOL
        g_rng = rb.ranges.cpu().numpy()
        for layer, (idx, cnt) in enumerate(sets):
            want = OR.storage_rows(idx, cnt, wl.seg(s), n_so, cap)
            for b in range(B):
                assert sorted(expand(g_rng[layer * B + b])) == sorted(want[b])
    final = wl.seg(steps - 1)
    assert np.array_equal(rb.k[0].view(torch.uint16).cpu().numpy(), OR.append_all(wl.k, final, n_so, cap, rows))
    assert np.array_equal(rb.v[0].view(torch.uint16).cpu().numpy(), OR.append_all(wl.v, final, n_so, cap, rows))
