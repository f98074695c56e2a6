"""GPU parity at the largest sizes: one sequence of 2^22 retained positions (4 GiB each of K and V, every
position kept), through the fused step (range table) and through murmur_evict_compact + the index-list
attention, checked against the fp64 oracle on the KV head whose rows lie furthest into the cache (byte
offsets past 3 GiB).  Also a batch of 4096 one-token sequences (the grid's sequence dimension, several
dispatch rounds)."""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_01483_amd import murmur as M
from paper_2606_01483_amd import workloads as W
from _tol import REL_TOL, LSE_TOL, lse_err, rel_err_fp32

pytestmark = pytest.mark.gpu
OFF = -1


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    M.lib()
    yield
    torch.cuda.synchronize()
    assert M.murmur_device_error() == 0


def announce(msg):
    print(f"\n[case] {msg}", flush=True)


def test_attn_four_million_positions():
    L = 1 << 22
    hq, hkv, D = W.HQ, W.HKV, W.HEAD_DIM
    G = hq // hkv
    announce(f"one sequence of {L} positions, {hkv} KV heads")
    k, v = W.large_cache(L, seed=4242, hkv=hkv)
    kv = M.kv_from_tensors(k, v)
    seg = np.array([[32, L - 64, 0, 32]], dtype=np.int32)  # 32 + (L - 64) + 0 + 32 = L positions
    pol = np.array([OFF, 0, 0, OFF, 0], dtype=np.int32)  # eviction off: every position is retained
    rng = np.random.default_rng(4243)
    q_bits = W.f32_to_bf16_bits(rng.standard_normal((1, 1, hq, D), dtype=np.float32))
    scale = 1.0 / math.sqrt(D)
    dev = torch.device("cuda")
    seg_d = torch.from_numpy(seg).to(dev)
    pol_d = torch.from_numpy(pol).to(dev)
    q = torch.from_numpy(q_bits).view(torch.bfloat16).to(dev)
    idx = torch.full((1, L), -1, dtype=torch.int32, device=dev)
    count = torch.zeros(1, dtype=torch.int32, device=dev)
    ranges = torch.zeros((1, M.N_PIECES, 2), dtype=torch.int32, device=dev)
    ws_bytes = M.murmur_decode_attn_workspace(1, 1, hq, hkv, L, 0)
    ws = torch.zeros(ws_bytes // 4 + 64, dtype=torch.int32, device=dev)
    outs = []
    for path in ("fused", "index"):
        out = torch.full((1, 1, hq, D), float("nan"), dtype=torch.float32, device=dev)
        lse = torch.zeros((1, 1, hq), dtype=torch.float32, device=dev)
        if path == "fused":
            M.murmur_decode_step(seg_d, pol_d, 0, q, kv, idx, count, ranges, L, 1, hq, hkv, D, scale, 0, out,
                                 M.MURMUR_DTYPE_F32, lse, ws, ws_bytes)
        else:
            M.murmur_evict_compact(seg_d, pol_d, 0, 1, idx, L, count, None)
            M.murmur_decode_attn(q, kv, idx, None, count, L, 1, hq, hkv, D, scale, 0, out, M.MURMUR_DTYPE_F32, lse,
                                 ws, ws_bytes)
        torch.cuda.synchronize()
        assert M.murmur_device_error() == 0, path
        assert int(count.item()) == L
        outs.append((out.cpu().numpy(), lse.cpu().numpy()))
    g = hkv - 1  # the KV head whose rows start furthest into the cache
    kh = k[:, :, g:g + 1].view(torch.uint16).cpu().numpy()
    vh = v[:, :, g:g + 1].view(torch.uint16).cpu().numpy()
    del k, v
    o_idx = np.arange(L, dtype=np.int32)[None]
    ref, ref_lse = oracle.attend(q_bits[:, :, g * G:(g + 1) * G], kh, vh, o_idx, np.array([L], dtype=np.int32),
                                 scale=scale, n_threads=16)
    for (out, lse), path in zip(outs, ("fused", "index")):
        assert rel_err_fp32(out[:, :, g * G:(g + 1) * G], ref) <= REL_TOL, path
        assert lse_err(lse[:, :, g * G:(g + 1) * G], ref_lse) <= LSE_TOL, path
    assert np.array_equal(idx[0, :1000].cpu().numpy(), np.arange(1000))


def test_attn_many_short_sequences():
    """4096 sequences of a 2-token prompt, 5 speech tokens and 1 output token (8 positions each; speech window
    3 with delay 0 and output window 1): a grid of 4096 sequences per KV head, several dispatch rounds."""
    B = 4096
    seg0 = np.tile(np.array([[2, 5, 0, 0]], dtype=np.int32), (B, 1))
    pol = np.array([3, 0, 0, 1, 0], dtype=np.int32)
    announce(f"{B} short sequences")
    wl = W.build("many_short", 4096, 1, seg0, pol, 1, planted=False, hq=8, hkv=2)
    from paper_2606_01483_amd.decode import DecodeBatch
    db = DecodeBatch(wl, out_dtype=M.MURMUR_DTYPE_F32, steps=[0])
    db.step_fused(0)
    torch.cuda.synchronize()
    assert M.murmur_device_error() == 0
    idx, cnt = oracle.retained(wl.seg(0), wl.policy, db.max_keep)
    ref, ref_lse = oracle.attend(wl.q(0), wl.k, wl.v, idx, cnt, scale=wl.scale, n_threads=16)
    assert rel_err_fp32(db.out.float().cpu().numpy(), ref) <= REL_TOL
    assert lse_err(db.lse.cpu().numpy(), ref_lse) <= LSE_TOL
    g_idx, g_cnt, _ = (t.cpu().numpy() for t in db.sets[0])
    assert np.array_equal(g_cnt, cnt) and np.array_equal(g_idx, idx)


@pytest.mark.parametrize("s_pos", [(1 << 23) - 8, 1 << 23])
def test_attn_long_row_strides(s_pos):
    """K/V rows 2^23 - 8 and 2^23 elements apart (16 MiB per position; the head rows at the start of each).
    Below 2^23 a pass of 32 consecutive rows addresses them from its first row with 32-bit offsets (up to 31
    rows, about 2^29 bytes); at 2^23 the launch takes 64-bit addresses per row instead.  One sequence of 65
    positions, eviction off, 32-position splits (the last a one-position pass), through the fused step and the
    range-table attention, against the fp64 oracle."""
    L, hq, hkv, D = 65, W.HQ, W.HKV, W.HEAD_DIM
    announce(f"row stride {s_pos} elements, {L} positions")
    rng = np.random.default_rng(4300 + (s_pos & 15))
    k_bits = W.f32_to_bf16_bits(rng.standard_normal((1, 1, hkv, L, D), dtype=np.float32))
    v_bits = W.f32_to_bf16_bits(rng.standard_normal((1, 1, hkv, L, D), dtype=np.float32))
    q_bits = W.f32_to_bf16_bits(rng.standard_normal((1, 1, hq, D), dtype=np.float32))
    scale = 1.0 / math.sqrt(D)
    dev = torch.device("cuda")
    span = (L - 1) * s_pos + hkv * D  # elements from the first row to the end of the last one's head rows
    kv_dev = []
    for bits in (k_bits, v_bits):
        buf = torch.empty(span, dtype=torch.bfloat16, device=dev)  # only the head rows are written and read
        rows = torch.from_numpy(bits[0, 0].transpose(1, 0, 2).copy()).view(torch.bfloat16).to(dev)  # [L, hkv, D]
        buf.as_strided((L, hkv, D), (s_pos, D, 1)).copy_(rows)
        kv_dev.append(buf)
    kv = M.make_kv(kv_dev[0], kv_dev[1], 1, L, (0, 0, D, s_pos))
    seg_d = torch.tensor([[0, L - 1, 0, 1]], dtype=torch.int32, device=dev)  # speech 0..63, output token 64
    pol_d = torch.tensor([OFF, 0, 0, OFF, 0], dtype=torch.int32, device=dev)
    q = torch.from_numpy(q_bits).view(torch.bfloat16).to(dev)
    count = torch.zeros(1, dtype=torch.int32, device=dev)
    ranges = torch.zeros((1, M.N_PIECES, 2), dtype=torch.int32, device=dev)
    ws_bytes = M.murmur_decode_attn_workspace(1, 1, hq, hkv, L, 32)
    ws = torch.zeros(ws_bytes // 4 + 64, dtype=torch.int32, device=dev)
    outs = []
    for path in ("fused", "ranges"):
        out = torch.full((1, 1, hq, D), float("nan"), dtype=torch.float32, device=dev)
        lse = torch.zeros((1, 1, hq), dtype=torch.float32, device=dev)
        if path == "fused":
            M.murmur_decode_step(seg_d, pol_d, 0, q, kv, None, count, ranges, L, 1, hq, hkv, D, scale, 32, out,
                                 M.MURMUR_DTYPE_F32, lse, ws, ws_bytes)
        else:
            M.murmur_decode_attn(q, kv, None, ranges, count, L, 1, hq, hkv, D, scale, 32, out, M.MURMUR_DTYPE_F32,
                                 lse, ws, ws_bytes)
        torch.cuda.synchronize()
        assert M.murmur_device_error() == 0, path
        assert int(count.item()) == L
        outs.append((out.cpu().numpy(), lse.cpu().numpy()))
    del kv_dev
    ref, ref_lse = oracle.attend(q_bits, k_bits, v_bits, np.arange(L, dtype=np.int32)[None],
                                 np.array([L], dtype=np.int32), scale=scale, n_threads=16)
    for (out, lse), path in zip(outs, ("fused", "ranges")):
        assert rel_err_fp32(out, ref) <= REL_TOL, path
        assert lse_err(lse, ref_lse) <= LSE_TOL, path


@pytest.mark.parametrize("s_h", [715827880, 1 << 30])
def test_attn_group_offsets_near_and_past_2_31(s_h):
    """KV heads s_h elements apart, rows contiguous within a head, so the last head's first element lies at
    3 s_h: just below 2^31 elements (the launch lets the wide schedule compute each group's offset with 32-bit
    products) and past it (64-bit products).  One sequence of 65 positions, eviction off, on the wide schedule
    with the automatic split and with 32-position splits, through the fused step and the range-table attention,
    against the fp64 oracle."""
    L, hq, hkv, D = 65, W.HQ, W.HKV, W.HEAD_DIM
    announce(f"KV heads {s_h} elements apart, {L} positions")
    rng = np.random.default_rng(4400 + (s_h & 15))
    k_bits = W.f32_to_bf16_bits(rng.standard_normal((1, 1, hkv, L, D), dtype=np.float32))
    v_bits = W.f32_to_bf16_bits(rng.standard_normal((1, 1, hkv, L, D), dtype=np.float32))
    q_bits = W.f32_to_bf16_bits(rng.standard_normal((1, 1, hq, D), dtype=np.float32))
    scale = 1.0 / math.sqrt(D)
    dev = torch.device("cuda")
    span = (hkv - 1) * s_h + L * D  # elements from the first head's first row to the end of the last head's rows
    kv_dev = []
    for bits in (k_bits, v_bits):
        buf = torch.empty(span, dtype=torch.bfloat16, device=dev)  # only the heads' rows are written and read
        rows = torch.from_numpy(bits[0, 0].copy()).view(torch.bfloat16).to(dev)  # [hkv, L, D]
        buf.as_strided((hkv, L, D), (s_h, D, 1)).copy_(rows)
        kv_dev.append(buf)
    kv = M.make_kv(kv_dev[0], kv_dev[1], 1, L, (0, 0, s_h, D))
    seg_d = torch.tensor([[0, L - 1, 0, 1]], dtype=torch.int32, device=dev)  # speech 0..63, output token 64
    pol_d = torch.tensor([OFF, 0, 0, OFF, 0], dtype=torch.int32, device=dev)
    q = torch.from_numpy(q_bits).view(torch.bfloat16).to(dev)
    count = torch.zeros(1, dtype=torch.int32, device=dev)
    ranges = torch.zeros((1, M.N_PIECES, 2), dtype=torch.int32, device=dev)
    ref, ref_lse = oracle.attend(q_bits, k_bits, v_bits, np.arange(L, dtype=np.int32)[None],
                                 np.array([L], dtype=np.int32), scale=scale, n_threads=16)
    for split_len in (0, 32):
        ws_bytes = M.murmur_decode_attn_workspace(1, 1, hq, hkv, L, split_len)
        ws = torch.zeros(ws_bytes // 4 + 64, dtype=torch.int32, device=dev)
        for path in ("fused", "ranges"):
            out = torch.full((1, 1, hq, D), float("nan"), dtype=torch.float32, device=dev)
            lse = torch.zeros((1, 1, hq), dtype=torch.float32, device=dev)
            if path == "fused":
                M.murmur_decode_step(seg_d, pol_d, 0, q, kv, None, count, ranges, L, 1, hq, hkv, D, scale, split_len,
                                     out, M.MURMUR_DTYPE_F32, lse, ws, ws_bytes)
            else:
                M.murmur_decode_attn(q, kv, None, ranges, count, L, 1, hq, hkv, D, scale, split_len, out,
                                     M.MURMUR_DTYPE_F32, lse, ws, ws_bytes)
            torch.cuda.synchronize()
            assert M.murmur_device_error() == 0, (split_len, path)
            assert int(count.item()) == L
            assert rel_err_fp32(out.cpu().numpy(), ref) <= REL_TOL, (split_len, path)
            assert lse_err(lse.cpu().numpy(), ref_lse) <= LSE_TOL, (split_len, path)
    del kv_dev
