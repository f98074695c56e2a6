"""GPU parity: the HIP path through the C ABI against the fp64 oracle (paper Section 3.2).

Retained lists must match bit for bit; attention outputs must meet the
criteria in _tol.py.  Every case prints its name before it touches the GPU.
"""
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2606_01483_amd import murmur as M
from paper_2606_01483_amd import workloads as W
from paper_2606_01483_amd.decode import DecodeBatch
from _tol import REL_TOL, LSE_TOL, bf16_excess, lse_err, rel_err_elementwise, rel_err_fp32

pytestmark = pytest.mark.gpu
OFF = -1
THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


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


def gpu_evict(seg, pol, max_keep, per_seq=1):
    B = seg.shape[0]
    seg_d = torch.from_numpy(np.ascontiguousarray(seg, dtype=np.int32)).cuda()
    pol_d = torch.from_numpy(np.ascontiguousarray(pol, dtype=np.int32)).cuda()
    idx = torch.full((B, max_keep), -7, dtype=torch.int32, device="cuda")
    cnt = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    rng = torch.full((B, 6, 2), -7, dtype=torch.int32, device="cuda")
    M.murmur_evict_compact(seg_d, pol_d, per_seq, B, idx, max_keep, cnt, rng)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), cnt.cpu().numpy(), rng.cpu().numpy()


def check_evict(seg, pol):
    ref_idx, ref_cnt = oracle.retained(seg, pol)
    max_keep = ref_idx.shape[1]
    idx, cnt, rng = gpu_evict(seg, pol, max_keep)
    assert np.array_equal(cnt, ref_cnt)
    assert np.array_equal(idx, ref_idx)
    for b in range(seg.shape[0]):
        assert expand(rng[b]) == ref_idx[b, :ref_cnt[b]].tolist()
        assert np.all(rng[b, :, 1] >= 0)


# ---- evict_compact: bit-exact ---------------------------------------------------------------------

@pytest.mark.parametrize("config", W.CONFIGS)
def test_evict_workloads_bitexact(config):
    lay = W.layout(config)
    for step in sorted({0, lay.steps // 2, lay.steps - 1}):
        announce(f"evict {config} step {step}")
        check_evict(lay.seg(step), lay.policy)


def test_evict_edge_layouts_bitexact():
    announce("evict edge layouts")
    rows = [  # (seg, policy)
        ([0, 0, 0, 1], [OFF, 0, 0, OFF, 0]),          # a single position
        ([5, 40, 7, 30], [8, 3, 2, 6, 2]),             # prompt_mid > 0, both sinks
        ([5, 40, 7, 3], [8, 3, 2, 6, 2]),              # j < output window
        ([2, 20, 0, 200], [8, 0, 0, 6, 0]),            # window clamped at the end of speech
        ([2, 20, 0, 9], [4, 0, 10, 6, 0]),             # sinks cover the window
        ([3, 10, 1, 5], [10, 0, 0, 5, 0]),             # windows exactly the region length
        ([3, 0, 4, 12], [5, 2, 1, 3, 20]),             # no speech; output sinks beyond j
        ([0, 64, 0, 64], [1, 1, 0, 1, 0]),             # one-token windows
        ([32, 2250, 0, 1264], [562, 512, 0, 256, 0]),  # the 300 s eviction workload at its last step
    ]
    seg = np.array([r[0] for r in rows], dtype=np.int32)
    pol = np.array([r[1] for r in rows], dtype=np.int32)
    check_evict(seg, pol)


def test_evict_random_layouts_bitexact():
    announce("evict 600 random layouts")
    rng = np.random.default_rng(2024)
    B = 600
    seg = np.stack([rng.integers(0, 40, B), rng.integers(0, 400, B), rng.integers(0, 20, B),
                    rng.integers(1, 500, B)], axis=1).astype(np.int32)
    pol = np.stack([np.where(rng.random(B) < 0.2, OFF, rng.integers(1, 300, B)), rng.integers(0, 300, B),
                    rng.integers(0, 30, B), np.where(rng.random(B) < 0.2, OFF, rng.integers(1, 300, B)),
                    rng.integers(0, 30, B)], axis=1).astype(np.int32)
    check_evict(seg, pol)


def test_evict_overflow_and_policy_errors():
    announce("evict device errors")
    seg = np.array([[4, 10, 0, 3], [4, 10, 0, 3]], dtype=np.int32)
    pol = np.array([[OFF, 0, 0, OFF, 0], [0, 0, 0, OFF, 0]], dtype=np.int32)  # row 1: window 0 is invalid
    idx, cnt, rng = gpu_evict(seg, pol, max_keep=5)
    code = M.murmur_device_error()
    assert code == M.MURMUR_DEVERR_OVERFLOW | M.MURMUR_DEVERR_POLICY
    assert cnt.tolist() == [17, 0]
    assert idx[0].tolist() == [0, 1, 2, 3, 4] and idx[1].tolist() == [-1] * 5
    assert M.murmur_device_error() == 0


# ---- decode_attn against the oracle ------------------------------------------------------------------

def oracle_step(wl, step, layers=None, batch=None):
    seg = wl.seg(step)
    idx, cnt = oracle.retained(seg, wl.policy)
    q, k, v = wl.q(step), wl.k, wl.v
    if layers is not None:
        q, k, v = q[layers], k[layers], v[layers]
    if batch is not None:
        q, k, v, idx, cnt = q[:, batch], k[:, batch], v[:, batch], idx[batch], cnt[batch]
    return oracle.attend(q, k, v, idx, cnt, scale=wl.scale, n_threads=THREADS)


def run_gpu(db, i, replica=0):
    db.step(i, replica)
    torch.cuda.synchronize()
    return db.out.float().cpu().numpy().astype(np.float64), db.lse.cpu().numpy().astype(np.float64)


_cache = {}


def tickets_clear(ws, ws_bytes):
    """The ticket region at the start of the workspace (128 bytes per KiB, rounded up to 256) is all zero."""
    region = (128 * -(-ws_bytes // 1024) + 255) // 256 * 256
    return int(torch.count_nonzero(ws[: region // 4]).item()) == 0


def workload(name):
    if name not in _cache:
        _cache[name] = W.make(name)
    return _cache[name]


def test_attn_tiny_all_steps():
    wl = workload("c1")
    db32 = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32)
    db16 = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_BF16)
    for i in range(wl.steps):
        announce(f"attn c1 step {i}")
        ref, ref_lse = oracle_step(wl, i)
        y32, l32 = run_gpu(db32, i)
        y16, _ = run_gpu(db16, i)
        assert rel_err_fp32(y32, ref) <= REL_TOL
        assert lse_err(l32, ref_lse) <= LSE_TOL
        assert bf16_excess(y16, ref) <= REL_TOL


@pytest.mark.parametrize("config", ["c2", "c3", "c4_dense", "c4_evict"])
def test_attn_workloads(config):
    wl = workload(config)
    steps = sorted({0, wl.steps // 2, wl.steps - 1})
    db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=steps)
    for i, s in enumerate(steps):
        announce(f"attn {config} step {s}")
        ref, ref_lse = oracle_step(wl, s)
        y, l = run_gpu(db, i)
        e = rel_err_fp32(y, ref)
        print(f"  max rel err (row-RMS floored) {e:.3e}, elementwise {rel_err_elementwise(y, ref):.3e}, "
              f"lse err {lse_err(l, ref_lse):.3e}", flush=True)
        assert e <= REL_TOL
        assert lse_err(l, ref_lse) <= LSE_TOL


@pytest.mark.parametrize("preset", list(W.ABLATION_PRESETS))
def test_ablation_presets(preset):
    """Every eviction preset of the paper's ablations (batch 16, 300 s chunks) at the first, a middle and
    the last of 2700 decode steps: retained sets bit for bit (fused step outputs) and attention."""
    if "ablation" not in _cache:
        _cache["ablation"] = W.ablation_workload()
    wl = W.with_policy(_cache["ablation"], W.ABLATION_PRESETS[preset])
    steps = [0, 1349, wl.steps - 1]
    db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=steps)
    for i, s in enumerate(steps):
        announce(f"ablation preset {preset!r} step {s}")
        db.step_fused(i)
        torch.cuda.synchronize()
        idx, cnt = oracle.retained(wl.seg(s), wl.policy, db.max_keep)
        assert np.array_equal(db.count.cpu().numpy(), cnt)
        assert np.array_equal(db.idx.cpu().numpy(), idx)
        ref, ref_lse = oracle.attend(wl.q(s), wl.k, wl.v, idx, cnt, scale=wl.scale, n_threads=THREADS)
        y = db.out.float().cpu().numpy()
        assert rel_err_fp32(y, ref) <= REL_TOL
        assert lse_err(db.lse.cpu().numpy(), ref_lse) <= LSE_TOL


def test_attn_28_layers_full():
    """The 28-layer workload at full size at its first, middle and last step, through both paths
    (murmur_evict_compact + murmur_decode_attn, and the one-launch murmur_decode_step): every layer, sequence
    and head of the fp32 output and the lse against the oracle, element by element; the fused step's index
    lists, counts and range tables bit for bit; the bf16 store path on the whole output at the middle step."""
    wl = workload("c5")
    steps = [0, wl.steps // 2, wl.steps - 1]
    db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=steps)
    db16 = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_BF16, steps=steps[1:2])
    for i, s in enumerate(steps):
        ref, ref_lse = oracle_step(wl, s)
        for path in ("two launches", "fused"):
            announce(f"attn c5 step {s} (28 layers), {path}")
            db.out.fill_(float("nan"))
            db.lse.fill_(float("nan"))
            if path == "fused":
                for t in db.sets[0]:
                    t.fill_(-7)
                db.step_fused(i)
            else:
                db.step(i)
            torch.cuda.synchronize()
            y = db.out.cpu().numpy().astype(np.float64)
            l = db.lse.cpu().numpy().astype(np.float64)
            e = rel_err_fp32(y, ref)
            print(f"  max rel err (row-RMS floored) {e:.3e}, elementwise {rel_err_elementwise(y, ref):.3e}, "
                  f"lse err {lse_err(l, ref_lse):.3e}", flush=True)
            assert e <= REL_TOL and lse_err(l, ref_lse) <= LSE_TOL, (s, path)
            if path == "fused":
                check_retained_outputs(db, wl, s)
        if s == steps[1]:
            announce(f"attn c5 step {s} (28 layers), bf16 store")
            y16, _ = run_gpu(db16, 0)
            assert bf16_excess(y16, ref) <= REL_TOL


def test_split_count_invariance():
    wl = workload("c3")
    ref, ref_lse = oracle_step(wl, 0)
    outs = []
    for split_len in (0, 32, 96, 128, 160, 192, 256, 512, 1024):
        announce(f"attn c3 split_len {split_len}")
        db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, split_len=split_len, steps=[0])
        y, l = run_gpu(db, 0)
        assert rel_err_fp32(y, ref) <= REL_TOL and lse_err(l, ref_lse) <= LSE_TOL
        outs.append(y)
    for split_len in (96, 160, 192):  # index lists too, splits of a whole and a partial pass per wavefront
        announce(f"attn c3 split_len {split_len} index list")
        db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, split_len=split_len, steps=[0], use_ranges=False)
        y, l = run_gpu(db, 0)
        assert rel_err_fp32(y, ref) <= REL_TOL and lse_err(l, ref_lse) <= LSE_TOL
        outs.append(y)
    for y in outs[1:]:
        assert rel_err_fp32(y, outs[0]) <= 1e-4


def test_index_mode_matches_range_mode_and_is_deterministic():
    wl = workload("c3")
    announce("attn c3 index vs range mode")
    a = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=[5], use_ranges=True)
    b = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=[5], use_ranges=False)
    ya, la = run_gpu(a, 0)
    yb, lb = run_gpu(b, 0)
    assert np.array_equal(ya, yb) and np.array_equal(la, lb)
    yc, lc = run_gpu(a, 0)
    assert np.array_equal(ya, yc) and np.array_equal(la, lc)
    # the workspace tickets are back at zero after every call
    assert tickets_clear(a.ws, a.ws_bytes)


def test_workspace_shared_across_shapes():
    """One workspace, zeroed once, serves calls of different shapes and kernels in turn (4, 48 and 384
    (layer, sequence, KV head) groups; 2 to 21 splits per group; wide-schedule and LDS-staged splits, and
    the two-level merge of 17 splits with its per-set tickets), all passing the same ws_bytes: a call with
    more groups than the one before never finds its tickets on partials that call left behind."""
    announce("attn workspace shared across shapes and schedules")
    rng = np.random.default_rng(404)
    B = 24
    seg0 = np.stack([rng.integers(0, 20, B), rng.integers(100, 500, B), rng.integers(0, 8, B),
                     rng.integers(1, 200, B)], axis=1).astype(np.int32)
    pol = np.stack([rng.integers(64, 300, B), rng.integers(0, 50, B), rng.integers(0, 8, B),
                    rng.integers(16, 128, B), rng.integers(0, 8, B)], axis=1).astype(np.int32)
    many = W.build("many", 41, 4, seg0, pol, steps=3, planted=False)
    c3, c4, c4d = workload("c3"), workload("c4_evict"), workload("c4_dense")
    cases = [(c4, 128, 0), (many, 128, 0), (c3, 256, 1), (c4d, 2080, 0), (c4, 256, 1), (many, 0, 1), (c3, 512, 2),
             (c4, 512, 2), (c4d, 2080, 1), (many, 256, 2), (c3, 128, 0), (many, 64, 1), (c4, 128, 2)]
    dbs = {}
    for wl, split_len, _ in cases:
        key = (wl.name, split_len)
        if key not in dbs:
            dbs[key] = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, split_len=split_len, steps=[0, 1, 2])
    ws_bytes = max(db.ws_bytes for db in dbs.values())
    ws = torch.zeros(ws_bytes // 4 + 64, dtype=torch.int32, device="cuda")
    for db in dbs.values():
        db.ws, db.ws_bytes = ws, ws_bytes
    for wl, split_len, i in cases:
        db = dbs[(wl.name, split_len)]
        ref, ref_lse = oracle_step(wl, i)
        y, l = run_gpu(db, i)
        assert rel_err_fp32(y, ref) <= REL_TOL and lse_err(l, ref_lse) <= LSE_TOL, (wl.name, split_len, i)
        assert tickets_clear(ws, ws_bytes), (wl.name, split_len, i)


def test_multi_round_grid_both_modes():
    """4 layers x 24 sequences x 4 KV heads of 500-900 retained positions: 384 whole-group workgroups, more than
    one dispatch round, so the LDS-staged kernel runs with one stage per wavefront (two workgroups per compute
    unit); index lists and range tables, fp32 and bf16 outputs."""
    rng = np.random.default_rng(77)
    B = 24
    seg0 = np.stack([np.full(B, 32), rng.integers(1800, 2250, B), np.zeros(B, dtype=np.int64),
                     rng.integers(300, 1200, B)], axis=1).astype(np.int32)
    pol = np.stack([seg0[:, 1] // 4, np.full(B, 512), np.zeros(B, dtype=np.int64), np.full(B, 256),
                    np.zeros(B, dtype=np.int64)], axis=1).astype(np.int32)
    wl = W.build("rounds", 43, 4, seg0, pol, steps=2, planted=True)
    ref, ref_lse = oracle_step(wl, 1)
    for use_ranges in (True, False):
        announce(f"attn 384 whole groups, one-stage LDS kernel, ranges={use_ranges}")
        db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=[1], use_ranges=use_ranges)
        assert db.split_len == 0
        y, l = run_gpu(db, 0)
        assert rel_err_fp32(y, ref) <= REL_TOL and lse_err(l, ref_lse) <= LSE_TOL, use_ranges
        db16 = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_BF16, steps=[1], use_ranges=use_ranges)
        y16, _ = run_gpu(db16, 0)
        assert bf16_excess(y16, ref) <= REL_TOL, use_ranges


@pytest.mark.parametrize("hq,hkv", [(28, 4), (4, 4), (16, 1), (12, 3)])
def test_attn_edge_shapes(hq, hkv):
    announce(f"attn edge shapes hq={hq} hkv={hkv}")
    seg0 = np.array([[0, 0, 0, 0], [5, 40, 7, 2], [3, 300, 2, 100], [1, 9, 0, 400]], dtype=np.int32)
    pol = np.array([[OFF, 0, 0, OFF, 0], [8, 3, 2, 6, 2], [64, 10, 4, 16, 1], [OFF, 0, 0, 128, 3]], dtype=np.int32)
    wl = W.build("edge", 77, 3, seg0, pol, steps=3, planted=False, hq=hq, hkv=hkv)
    db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32)
    for i in range(wl.steps):
        ref, ref_lse = oracle_step(wl, i)
        y, l = run_gpu(db, i)
        assert rel_err_fp32(y, ref) <= REL_TOL and lse_err(l, ref_lse) <= LSE_TOL


def test_attn_strided_cache_layout():
    """K/V stored [layer][kv head][sequence][pos] with padded rows: only the strides change."""
    announce("attn strided cache layout")
    wl = workload("c3")
    ref, ref_lse = oracle_step(wl, 3)
    NL, B, Hkv, L, D = wl.k.shape
    pad = 136
    def relayout(x):
        t = torch.zeros((NL, Hkv, B, L, pad), dtype=torch.bfloat16, device="cuda")
        t[..., :D] = torch.from_numpy(x).view(torch.bfloat16).cuda().permute(0, 2, 1, 3, 4)
        return t
    kt, vt = relayout(wl.k), relayout(wl.v)
    kv = M.make_kv(kt, vt, NL, L, (kt.stride(0), kt.stride(2), kt.stride(1), kt.stride(3)))
    db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=[3])
    db.evict(0)
    M.murmur_decode_attn(db.q[0], kv, db.idx, db.ranges, db.count, db.max_keep, B, wl.hq, Hkv, D, wl.scale, 0,
                         db.out, M.MURMUR_DTYPE_F32, db.lse, db.ws, db.ws_bytes)
    torch.cuda.synchronize()
    y = db.out.cpu().numpy().astype(np.float64)
    assert rel_err_fp32(y, ref) <= REL_TOL and lse_err(db.lse.cpu().numpy(), ref_lse) <= LSE_TOL


@pytest.mark.parametrize("split_len,max_keep", [(0, None), (96, None), (32, None), (288, 288 * 20), (288, 288 * 130)])
def test_attn_device_errors_give_nan(split_len, max_keep):
    """A position outside the cache (index mode) and a count above max_keep are caught by the kernel's
    own bounds checks: nothing outside the cache is read, the sequence's outputs are NaN and the
    device error word says why.  The NaN of the split that saw the position reaches the output through
    every merge: one split, the wide schedule's merges of 2 and 6 partials, and the LDS-staged schedule's
    two-level merge (20 partials) and one-level merge of many (130 partials)."""
    announce(f"attn device errors, split_len {split_len}, max_keep {max_keep}")
    wl = workload("c1")
    db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=[0], use_ranges=False, split_len=split_len,
                     max_keep=max_keep)
    db.evict(0)
    torch.cuda.synchronize()
    db.idx[0, 3] = wl.max_len + 5
    db.attend(0)
    torch.cuda.synchronize()
    assert M.murmur_device_error() == M.MURMUR_DEVERR_POSITION
    assert torch.isnan(db.out).all().item()
    db.evict(0)
    db.count.fill_(db.max_keep + 1)
    db.attend(0)
    torch.cuda.synchronize()
    err = M.murmur_device_error()
    if max_keep is None:
        assert err == M.MURMUR_DEVERR_COUNT
    else:  # the ranks past the real count then hold -1, which the position check reports as well
        assert err in (M.MURMUR_DEVERR_COUNT, M.MURMUR_DEVERR_COUNT | M.MURMUR_DEVERR_POSITION)
    assert torch.isnan(db.out).all().item()
    assert tickets_clear(db.ws, db.ws_bytes)


def test_graph_replays_match_eager_and_pipelined_schedule():
    """Steps captured into a HIP graph (serial, and pipelined over two streams) replay to the eager result
    every time, with eager work and synchronisation between the replays."""
    announce("attn c3 graph replays (serial and pipelined)")
    wl = workload("c3")
    steps = [0, 1, 2, 3]
    db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=steps, replicas=2)
    reps = [0, 1, 0, 1]
    for i in range(4):
        db.step(i, reps[i])
    torch.cuda.synchronize()
    eager = db.out.clone()
    eager_lse = db.lse.clone()

    stream = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    graphs = {}
    for name, fn in (("serial", lambda: [db.step(i, reps[i]) for i in range(4)]),
                     ("pipelined", lambda: db.pipelined_steps(list(range(4)), reps, torch.cuda.current_stream(),
                                                              side))):
        g = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream()
        cap.wait_stream(stream)
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=cap):
            fn()
        torch.cuda.synchronize()
        graphs[name] = g
    for trial in range(3):
        for name, g in graphs.items():
            db.out.zero_()
            db.lse.zero_()
            db.step(1, 1)  # unrelated eager work between replays
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(db.out, eager), (name, trial)
            assert torch.equal(db.lse, eager_lse), (name, trial)
    # the eagerly pipelined schedule gives the same result too
    db.out.zero_()
    db.pipelined_steps(list(range(4)), reps, stream, side)
    torch.cuda.synchronize()
    assert torch.equal(db.out, eager)


def test_many_ragged_sequences_both_modes():
    """130 ragged sequences over 2 layers with per-sequence policies (empty speech and outputs included), index-list
    and range modes, the automatic split, fixed splits on the wide schedule (96 and 256 positions) and on the
    LDS-staged kernel (512)."""
    announce("attn 130 ragged sequences")
    rng = np.random.default_rng(99)
    B = 130
    seg0 = np.stack([rng.integers(0, 20, B), rng.integers(0, 700, B), rng.integers(0, 8, B),
                     rng.integers(0, 300, B)], axis=1).astype(np.int32)
    pol = np.stack([np.where(rng.random(B) < 0.3, OFF, rng.integers(1, 400, B)), rng.integers(0, 200, B),
                    rng.integers(0, 8, B), np.where(rng.random(B) < 0.3, OFF, rng.integers(1, 200, B)),
                    rng.integers(0, 8, B)], axis=1).astype(np.int32)
    wl = W.build("ragged", 31, 2, seg0, pol, steps=2, planted=False)
    ref, ref_lse = oracle_step(wl, 1)
    for split_len in (0, 96, 256, 512):
        for use_ranges in (True, False):
            db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=[1], split_len=split_len,
                             use_ranges=use_ranges)
            y, l = run_gpu(db, 0)
            assert rel_err_fp32(y, ref) <= REL_TOL and lse_err(l, ref_lse) <= LSE_TOL, (split_len, use_ranges)


def test_max_keep_far_above_the_counts():
    """A max_keep far above the actual counts sizes the grid for splits that hold no retained position; they
    take part in the merge with an empty partial (results right on two calls in a row, tickets back at zero)."""
    wl = workload("c1")
    steps = [0, wl.steps - 1]
    for split_len in (0, 128, 512):
        db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=steps, split_len=split_len, max_keep=8192)
        for i, s in enumerate(steps):
            announce(f"attn c1, max_keep 8192, split_len {split_len}, step {s}")
            ref, ref_lse = oracle_step(wl, s)
            for _ in range(2):
                y, l = run_gpu(db, i)
                assert rel_err_fp32(y, ref) <= REL_TOL and lse_err(l, ref_lse) <= LSE_TOL
        assert tickets_clear(db.ws, db.ws_bytes)


def test_merge_every_partial_count():
    """Every count of partials per group from 2 to 18 (the merge is specialised on the count up to 16 and
    takes batches beyond): c1's 192 retained positions in splits of 96, 64 and 32 positions, with max_keep
    raised so that the splits past the counts hold empty partials."""
    wl = workload("c1")
    s = wl.steps - 1
    ref, ref_lse = oracle_step(wl, s)
    cases = [(96, 192), (64, 192), (64, 256), (64, 320)] + [(32, 32 * n) for n in range(6, 19)]
    for split_len, max_keep in cases:
        n = -(-max_keep // split_len)
        announce(f"attn c1 step {s}, split_len {split_len}, max_keep {max_keep}: {n} partials per group")
        db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=[s], split_len=split_len, max_keep=max_keep)
        assert db.split_len == split_len
        y, l = run_gpu(db, 0)
        assert rel_err_fp32(y, ref) <= REL_TOL and lse_err(l, ref_lse) <= LSE_TOL, (split_len, max_keep)
        assert tickets_clear(db.ws, db.ws_bytes)


def test_two_level_merge_counts():
    """The LDS-staged schedule's merges of 17 to 128 splits in two levels (sets of 8, the last set short or
    whole) and beyond 128 in one: the one-hour dense list in splits of 2080 to 288 positions, the last with
    max_keep raised to 130 splits (the ones past the count empty)."""
    wl = workload("c4_dense")
    s = wl.steps - 1
    ref, ref_lse = oracle_step(wl, s)
    seen = []
    for split_len, max_keep in ((2080, None), (1472, None), (1408, None), (544, None), (288, None), (288, 288 * 130)):
        db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=[s], split_len=split_len, max_keep=max_keep)
        n = -(-db.max_keep // split_len)
        seen.append(n)
        announce(f"attn c4_dense step {s}, split_len {split_len}: {n} partials per group")
        y, l = run_gpu(db, 0)
        assert rel_err_fp32(y, ref) <= REL_TOL and lse_err(l, ref_lse) <= LSE_TOL, (split_len, n)
        assert tickets_clear(db.ws, db.ws_bytes)
    # a short last set (n mod 8 == 1 and otherwise), a whole one, the largest two-level count's region, one level
    assert any(16 < n <= 128 and n % 8 == 1 for n in seen) and any(16 < n <= 128 and n % 8 == 0 for n in seen)
    assert any(16 < n <= 128 and n % 8 not in (0, 1) for n in seen) and any(n > 128 for n in seen)
    # two levels in a grid of more than one dispatch round (the one-stage form): c3's 48 groups in 20 splits
    # of 288 positions (the splits past each sequence's count empty), 960 workgroups
    wl = workload("c3")
    ref, ref_lse = oracle_step(wl, 0)
    db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=[0], split_len=288, max_keep=288 * 20)
    announce("attn c3 step 0, split_len 288, max_keep 5760: 20 partials per group, 960 workgroups")
    y, l = run_gpu(db, 0)
    assert rel_err_fp32(y, ref) <= REL_TOL and lse_err(l, ref_lse) <= LSE_TOL
    assert tickets_clear(db.ws, db.ws_bytes)


# ---- murmur_decode_step: eviction and attention in one launch ------------------------------------

def check_retained_outputs(db, wl, s, buf=0):
    """The fused step's retained-set outputs against the oracle, bit for bit."""
    ref_idx, ref_cnt = oracle.retained(wl.seg(s), wl.policy, max_keep=db.max_keep)
    idx, cnt, rng = (t.cpu().numpy() for t in db.sets[buf])
    assert np.array_equal(cnt, ref_cnt)
    assert np.array_equal(idx, ref_idx)
    for b in range(db.B):
        assert expand(rng[b]) == ref_idx[b, :ref_cnt[b]].tolist()


@pytest.mark.parametrize("config", ["c1", "c2", "c3", "c4_dense", "c4_evict", "c5"])
def test_decode_step_fused(config):
    """murmur_decode_step against the oracle with the automatic split and a fixed one: attention to the fp32
    bar (every layer, sequence and head), the index list, counts and range tables it writes bit-exact."""
    wl = workload(config)
    steps = [0, wl.steps - 1]
    for split_len in (0, 256):
        db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=steps, split_len=split_len)
        for i, s in enumerate(steps):
            announce(f"decode_step {config} step {s} split_len {split_len}")
            ref, ref_lse = oracle_step(wl, s)
            for t in db.sets[0]:
                t.fill_(-7)
            db.out.fill_(float("nan"))
            db.step_fused(i)
            torch.cuda.synchronize()
            y = db.out.float().cpu().numpy().astype(np.float64)
            l = db.lse.cpu().numpy().astype(np.float64)
            assert rel_err_fp32(y, ref) <= REL_TOL and lse_err(l, ref_lse) <= LSE_TOL
            check_retained_outputs(db, wl, s)
        assert tickets_clear(db.ws, db.ws_bytes)


def test_decode_step_fused_ragged_and_without_outputs():
    """130 ragged sequences with per-sequence policies, retained-set outputs written and not."""
    announce("decode_step, 130 ragged sequences")
    rng = np.random.default_rng(123)
    B = 130
    seg0 = np.stack([rng.integers(0, 20, B), rng.integers(0, 700, B), rng.integers(0, 8, B),
                     rng.integers(0, 300, B)], axis=1).astype(np.int32)
    pol = np.stack([np.where(rng.random(B) < 0.3, OFF, rng.integers(1, 400, B)), rng.integers(0, 200, B),
                    rng.integers(0, 8, B), np.where(rng.random(B) < 0.3, OFF, rng.integers(1, 200, B)),
                    rng.integers(0, 8, B)], axis=1).astype(np.int32)
    wl = W.build("ragged", 37, 2, seg0, pol, steps=2, planted=False)
    ref, ref_lse = oracle_step(wl, 1)
    for split_len in (0, 64, 256):
        db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=[1], split_len=split_len)
        for outputs in (True, False):
            db.out.fill_(float("nan"))
            db.step_fused(0, outputs=outputs)
            torch.cuda.synchronize()
            y = db.out.float().cpu().numpy().astype(np.float64)
            l = db.lse.cpu().numpy().astype(np.float64)
            assert rel_err_fp32(y, ref) <= REL_TOL and lse_err(l, ref_lse) <= LSE_TOL, (split_len, outputs)
        check_retained_outputs(db, wl, 1)


def test_decode_step_fused_device_errors():
    """An invalid policy and a count above max_keep: the evict_compact outputs and errors, NaN attention."""
    announce("decode_step device errors")
    wl = workload("c1")
    db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=[0])
    bad_pol = torch.tensor([[0, 0, 0, 0, 0]], dtype=torch.int32, device="cuda")  # out_window 0: invalid
    idx, cnt, rng = db.sets[0]
    M.murmur_decode_step(db.seg[0], bad_pol, 0, db.q[0], db.kv[0], idx, cnt, rng, db.max_keep, db.B, db.Hq, db.Hkv,
                         db.D, wl.scale, 0, db.out, db.out_dtype, db.lse, db.ws, db.ws_bytes)
    torch.cuda.synchronize()
    assert M.murmur_device_error() == M.MURMUR_DEVERR_POLICY | M.MURMUR_DEVERR_COUNT
    assert torch.isnan(db.out).all().item()
    assert cnt.cpu().tolist() == [0] and (idx == -1).all().item() and (rng == 0).all().item()
    true_cnt = int(oracle.retained(wl.seg(0), wl.policy)[1][0])
    small = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=[0], max_keep=true_cnt - 5)
    small.step_fused(0)
    torch.cuda.synchronize()
    assert M.murmur_device_error() == M.MURMUR_DEVERR_OVERFLOW | M.MURMUR_DEVERR_COUNT
    assert torch.isnan(small.out).all().item()
    ref_idx, _ = oracle.retained(wl.seg(0), wl.policy)
    assert small.count.cpu().tolist() == [true_cnt]
    assert np.array_equal(small.idx.cpu().numpy()[0], ref_idx[0, : true_cnt - 5])


def test_decode_step_fused_graph_replays():
    """Fused steps captured into a HIP graph replay to the eager result every time."""
    announce("decode_step graph replays")
    wl = workload("c3")
    steps = [0, 1, 2]
    db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=steps)
    outs = []
    for i in range(len(steps)):
        db.step_fused(i)
        torch.cuda.synchronize()
        outs.append(db.out.clone())
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        db.step_fused(0, stream=s)  # warm-up on the capture stream
        g.capture_begin()
        for i in range(len(steps)):
            db.step_fused(i, stream=s)
        g.capture_end()
    torch.cuda.current_stream().wait_stream(s)
    for _ in range(3):
        db.out.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(db.out, outs[-1])
        db.step_fused(0)
        torch.cuda.synchronize()
        assert torch.equal(db.out, outs[0])
