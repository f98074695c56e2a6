"""Seeded random configurations through every entry point, against the fp64 oracle (GPU).

Each case draws a batch size, layer count, GQA shape, sequence layouts, per-sequence policies, a split length
and an entry point -- index list, range table, fused step, ring storage or paged
pool -- and checks two decode steps: the attention to the fp32 bar and, where the entry point writes them,
the retained sets bit for bit.  The case is printed before it touches the GPU.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import paged as OP
from oracle import ring as OR
from paper_2606_01483_amd import murmur as M
from paper_2606_01483_amd import workloads as W
from paper_2606_01483_amd.decode import DecodeBatch, PagedBatch, RingBatch
from _tol import REL_TOL, LSE_TOL, lse_err, rel_err_fp32

pytestmark = pytest.mark.gpu
OFF = -1
N_CASES = 40
MODES = ("index", "ranges", "fused", "ring", "paged")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    M.lib()
    yield
    torch.cuda.synchronize()
    assert M.murmur_device_error() == 0


def draw_case(k):
    rng = np.random.default_rng(7000 + k)
    B = int(rng.integers(1, 20))
    NL = int(rng.integers(1, 4))
    hkv = int(rng.choice([1, 2, 4]))
    group = int(rng.choice([1, 2, 4, 7, 8, 16]))
    seg0 = np.stack([rng.integers(0, 41, B), rng.integers(0, 1500, B), rng.integers(0, 9, B),
                     rng.integers(0, 600, B)], axis=1).astype(np.int32)
    pol = np.stack([np.where(rng.random(B) < 0.3, OFF, rng.integers(1, 800, B)), rng.integers(0, 600, B),
                    rng.integers(0, 41, B), np.where(rng.random(B) < 0.3, OFF, rng.integers(1, 300, B)),
                    rng.integers(0, 9, B)], axis=1).astype(np.int32)
    mode = MODES[k % len(MODES)]
    choices = [0, 32, 64, 96, 128, 192, 256, 384, 640, 1024]
    if mode != "ring":
        choices.append(512)
    split_len = int(rng.choice(choices))
    unscaled = bool(rng.random() < 0.5)  # queries N(0,1) with scale 1/sqrt(D), else pre-scaled with scale 1
    return dict(B=B, NL=NL, hkv=hkv, group=group, seg0=seg0, pol=pol, mode=mode, split_len=split_len,
                unscaled=unscaled, planted=bool(rng.random() < 0.5), block=int(rng.choice([1, 8, 16, 64])))


def check_attention(wl, s, out, lse, max_keep=None):
    idx, cnt = oracle.retained(wl.seg(s), wl.policy, max_keep)
    ref, ref_lse = oracle.attend(wl.q(s), wl.k, wl.v, idx, cnt, scale=wl.scale, n_threads=16)
    assert rel_err_fp32(out.float().cpu().numpy(), ref) <= REL_TOL
    assert lse_err(lse.cpu().numpy(), ref_lse) <= LSE_TOL
    return idx, cnt


@pytest.mark.parametrize("k", range(N_CASES))
def test_random_configuration(k):
    c = draw_case(k)
    print(f"\n[case] random {k}: mode {c['mode']} B={c['B']} NL={c['NL']} Hkv={c['hkv']} G={c['group']} "
          f"split_len={c['split_len']} unscaled={c['unscaled']} block={c['block']}", flush=True)
    kw = dict(hq=c["hkv"] * c["group"], hkv=c["hkv"])
    if c["unscaled"]:
        kw.update(scale=1.0 / math.sqrt(W.HEAD_DIM), q_scale=1.0)
    wl = W.build(f"random{k}", 9000 + k, c["NL"], c["seg0"], c["pol"], 2, planted=c["planted"] and c["hkv"] > 0,
                 **kw)
    steps = [0, 1]
    mode = c["mode"]
    if mode in ("index", "ranges", "fused"):
        db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, split_len=c["split_len"], use_ranges=mode == "ranges",
                         steps=steps)
        for i, s in enumerate(steps):
            if mode == "fused":
                db.step_fused(i)
            else:
                db.step(i)
            torch.cuda.synchronize()
            idx, cnt = check_attention(wl, s, db.out, db.lse, db.max_keep)
            g_idx, g_cnt, g_rng = (t.cpu().numpy() for t in db.sets[0])
            assert np.array_equal(g_cnt, cnt)
            assert np.array_equal(g_idx, idx)
    elif mode == "ring":
        n_so = wl.policy[:, 4]
        last_j = wl.seg(steps[-1])[:, 3]
        cap = int(max([int(w) for w in wl.policy[:, 3] if w >= 1] + [int(j - n) for j, n in zip(last_j, n_so)] + [1]))
        seg_before = wl.seg(0)
        seg_before[:, 3] -= 1
        rows = max(OR.storage_len(seg_before[b], n_so[b], cap) for b in range(wl.batch))
        rows = (rows + 7) // 8 * 8
        st = (OR.append_all(wl.k, seg_before, n_so, cap, rows), OR.append_all(wl.v, seg_before, n_so, cap, rows))
        rb = RingBatch(wl, cap, out_dtype=M.MURMUR_DTYPE_F32, split_len=c["split_len"], steps=steps, storage=st)
        for i, s in enumerate(steps):
            rb.step(i)
            torch.cuda.synchronize()
            check_attention(wl, s, rb.out, rb.lse)
        final = wl.seg(steps[-1])
        assert np.array_equal(rb.k[0].view(torch.uint16).cpu().numpy(), OR.append_all(wl.k, final, n_so, cap, rows))
    else:
        pb = PagedBatch(wl, c["block"], layout="flash" if k % 2 else "head", out_dtype=M.MURMUR_DTYPE_F32,
                        split_len=c["split_len"], steps=steps, seed=k)
        for i, s in enumerate(steps):
            pb.step(i)
            torch.cuda.synchronize()
            idx, cnt = check_attention(wl, s, pb.out, pb.lse, pb.max_keep)
            assert np.array_equal(pb.idx.cpu().numpy(), OP.rows_of(idx, cnt, pb.block_table, c["block"]))
    assert M.murmur_device_error() == 0
