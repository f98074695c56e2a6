"""Host-side checks of the C ABI (no GPU): exported symbols, argument validation, sizing.

Every call here is rejected by the host-side checks, which run before any HIP
call, so nothing reaches a device.  The module is skipped where a GPU is
visible, so that no malformed pointer could ever be launched on one.
"""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

import oracle
from oracle import paged as OP
from oracle import ring as OR
from paper_2606_01483_amd import _build
from paper_2606_01483_amd import murmur as M

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OFF = -1

pytestmark = pytest.mark.skipif(torch.cuda.device_count() > 0, reason="host-only checks run where no GPU is visible")


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not os.path.exists(M.LIB_PATH):
        _build.build()
    M.lib()


def declared_functions():
    text = open(os.path.join(ROOT, "include", "murmur.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(murmur_[a-z_0-9]+)\s*\(", text)))


def test_exports_every_declared_function():
    names = declared_functions()
    assert len(names) == 18
    lib = ctypes.CDLL(M.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_abi_version():
    assert M.murmur_abi_version() == 10


def test_retained_count_host_matches_oracle():
    rng = np.random.default_rng(3)
    B = 300
    seg = np.stack([rng.integers(0, 40, B), rng.integers(0, 400, B), rng.integers(0, 20, B),
                    rng.integers(1, 500, B)], axis=1).astype(np.int32)
    pol = np.stack([np.where(rng.random(B) < 0.2, OFF, rng.integers(1, 300, B)), rng.integers(0, 300, B),
                    rng.integers(0, 30, B), np.where(rng.random(B) < 0.2, OFF, rng.integers(1, 300, B)),
                    rng.integers(0, 30, B)], axis=1).astype(np.int32)
    counts, mx = M.murmur_retained_count_host(seg, pol, 1)
    _, ref = oracle.retained(seg, pol)
    assert np.array_equal(counts, ref) and mx == ref.max()


@pytest.mark.parametrize("seg,pol", [
    ([0, 5, 0, 0], [OFF, 0, 0, OFF, 0]),
    ([0, 5, 0, 3], [0, 0, 0, OFF, 0]),
    ([0, 5, 0, 3], [OFF, 0, 0, 0, 0]),
    ([0, 5, 0, 3], [-2, 0, 0, OFF, 0]),
    ([0, 5, 0, 3], [2, -1, 0, OFF, 0]),
    ([0, 5, 0, 3], [2, 0, -1, OFF, 0]),
    ([0, 5, 0, 3], [2, 0, 0, OFF, -3]),
    ([-1, 5, 0, 3], [OFF, 0, 0, OFF, 0]),
    ([0x7fffffff, 5, 0, 3], [OFF, 0, 0, OFF, 0]),
])
def test_retained_count_host_rejects_invalid(seg, pol):
    with pytest.raises(M.MurmurError) as e:
        M.murmur_retained_count_host(np.array([seg]), np.array(pol))
    assert e.value.code == M.MURMUR_EINVAL
    assert "invalid layout or policy" in M.murmur_last_error()


FAKE = 0x100000  # never dereferenced: every call below fails validation first


def attn_args(**over):
    a = dict(q=FAKE, kv=M.murmur_kv(FAKE, FAKE, 1, 4096, 4096 * 128 * 4, 4096 * 128 * 4, 4096 * 128, 128),
             idx=FAKE, ranges=None, count=FAKE, max_keep=850, B=12, Hq=28, Hkv=4, D=128, scale=1.0, split_len=0,
             out=FAKE, out_dtype=M.MURMUR_DTYPE_BF16, lse=None, ws=FAKE, ws_bytes=1 << 30)
    a.update(over)
    return a


def call_attn(a):
    return M.lib().murmur_decode_attn(a["q"], ctypes.byref(a["kv"]), a["idx"], a["ranges"], a["count"],
                                      a["max_keep"], a["B"], a["Hq"], a["Hkv"], a["D"], a["scale"], a["split_len"],
                                      a["out"], a["out_dtype"], a["lse"], a["ws"], a["ws_bytes"], 0)


@pytest.mark.parametrize("over,code", [
    (dict(q=None), M.MURMUR_EINVAL),
    (dict(out=None), M.MURMUR_EINVAL),
    (dict(ws=None), M.MURMUR_EINVAL),
    (dict(count=None), M.MURMUR_EINVAL),
    (dict(idx=None, ranges=None), M.MURMUR_EINVAL),
    (dict(B=0), M.MURMUR_EINVAL),
    (dict(max_keep=0), M.MURMUR_EINVAL),
    (dict(Hq=30), M.MURMUR_EINVAL),
    (dict(D=64), M.MURMUR_EUNSUPPORTED),
    (dict(Hq=68, Hkv=4), M.MURMUR_EUNSUPPORTED),
    (dict(out_dtype=7), M.MURMUR_EINVAL),
    (dict(scale=float("nan")), M.MURMUR_EINVAL),
    (dict(scale=float("inf")), M.MURMUR_EINVAL),
    (dict(split_len=100), M.MURMUR_EINVAL),
    (dict(split_len=-128), M.MURMUR_EINVAL),
    (dict(split_len=-2), M.MURMUR_EINVAL),
    (dict(max_keep=(1 << 28) + 1), M.MURMUR_EUNSUPPORTED),
    (dict(split_len=-1), M.MURMUR_EINVAL),
    (dict(q=FAKE + 8), M.MURMUR_EINVAL),
    (dict(ws=FAKE + 64), M.MURMUR_EINVAL),
    (dict(lse=FAKE + 2), M.MURMUR_EINVAL),
    (dict(out=FAKE + 8), M.MURMUR_EINVAL),
    (dict(kv=M.murmur_kv(FAKE, FAKE, 1, 4096, 0, 0, 0, 100)), M.MURMUR_EINVAL),   # stride not a multiple of 8
    (dict(kv=M.murmur_kv(FAKE, FAKE, 1, 4096, 0, 0, 0, 64)), M.MURMUR_EINVAL),    # rows overlap
    (dict(kv=M.murmur_kv(FAKE, None, 1, 4096, 0, 0, 0, 128)), M.MURMUR_EINVAL),
    (dict(kv=M.murmur_kv(FAKE, FAKE, 0, 4096, 0, 0, 0, 128)), M.MURMUR_EINVAL),
    (dict(kv=M.murmur_kv(FAKE + 4, FAKE, 1, 4096, 0, 0, 0, 128)), M.MURMUR_EINVAL),
    (dict(ws_bytes=1000), M.MURMUR_ENOSPACE),
])
def test_decode_attn_rejects(over, code):
    assert call_attn(attn_args(**over)) == code
    assert M.murmur_last_error() != ""


def test_evict_compact_rejects():
    lib = M.lib()
    assert lib.murmur_evict_compact(None, FAKE, 0, 12, FAKE, 10, FAKE, None, 0) == M.MURMUR_EINVAL
    assert lib.murmur_evict_compact(FAKE, FAKE, 0, 0, FAKE, 10, FAKE, None, 0) == M.MURMUR_EINVAL
    assert lib.murmur_evict_compact(FAKE, FAKE, 0, 12, FAKE, 0, FAKE, None, 0) == M.MURMUR_EINVAL
    assert lib.murmur_evict_compact(FAKE, FAKE, 2, 12, FAKE, 10, FAKE, None, 0) == M.MURMUR_EINVAL
    assert lib.murmur_evict_compact(FAKE, FAKE, 0, 12, FAKE + 2, 10, FAKE, None, 0) == M.MURMUR_EINVAL


def rnd(x):
    return (x + 255) // 256 * 256


def ticket_region(ws_bytes):
    """Bytes at the start of a workspace that hold the tickets: 128 per KiB of workspace (a 128-byte line per
    ticket), rounded up."""
    return rnd(128 * -(-ws_bytes // 1024))


def split_partials(groups, n_split, G):
    # (m, l) and 128 outputs per (group, split, head)
    return rnd(groups * n_split * G * 2 * 4) + rnd(groups * n_split * G * 128 * 4)


def lds_tickets(groups, n_split):
    """Ticket counters of the LDS-staged schedule: one per group, and one per set of 8 splits when it merges
    17 to 128 splits in two levels."""
    return groups * (1 + -(-n_split // 8)) if 16 < n_split <= 128 else groups


def check_plan(ws, partials, tickets):
    """The workspace holds its ticket region and the partials, with room to spare, and so does any larger one."""
    for w in (ws, ws + 1, ws + 255, ws + 256, ws + 65536, ws + 65536 * 3 + 77, 2 * ws):
        assert ticket_region(w) >= 128 * tickets and ticket_region(w) + partials <= w, w
    assert ws - 256 < max(ticket_region(ws) + partials + 256, rnd(tickets * 1024)) + 256  # and it is the smallest


def test_workspace_sizing():
    ws = M.murmur_decode_attn_workspace(1, 12, 28, 4, 850)
    # 48 groups of 850 positions: 5 splits of 170 positions each, 240 workgroups in one round
    check_plan(ws, split_partials(48, 5, 7), 48)
    assert ws - ticket_region(ws) < split_partials(48, 6, 7)
    # 4 groups of 2592: the estimate balances the per-unit share, in whole passes of 32 rows, against merging
    # many partials; 14 splits of 186 positions take the same 6 passes per workgroup as 16 of 162 with two
    # partials fewer to merge, and fewer than 14 need a seventh pass, so 14 splits
    check_plan(M.murmur_decode_attn_workspace(1, 1, 28, 4, 2592), split_partials(4, 14, 7), 4)
    ws = M.murmur_decode_attn_workspace(1, 1, 28, 4, 2592)
    assert ws - ticket_region(ws) < split_partials(4, 15, 7)
    assert M.murmur_decode_attn_workspace(1, 1, 28, 4, 100) == 256  # one split: nothing to merge
    assert M.murmur_decode_attn_workspace(1, 12, 28, 4, 850, 1024) == 256
    # an explicit split length on a long list
    ws = M.murmur_decode_attn_workspace(1, 1, 28, 4, 35160, 640)
    check_plan(ws, split_partials(4, -(-35160 // 640), 7), lds_tickets(4, -(-35160 // 640)))
    # automatic split of 1100 units over 4 groups: 55 splits of 5 units
    ws = M.murmur_decode_attn_workspace(1, 1, 28, 4, 35160)
    check_plan(ws, split_partials(4, 55, 7), lds_tickets(4, 55))
    assert ws - ticket_region(ws) < split_partials(4, 56, 7)
    # one group of 300 units: too many one-pass splits to merge, so 60 splits of 5 units
    ws = M.murmur_decode_attn_workspace(1, 1, 7, 1, 300 * 128)
    check_plan(ws, split_partials(1, 60, 7), lds_tickets(1, 60))
    assert ws - ticket_region(ws) < split_partials(1, 61, 7)
    # many groups of two splits
    ws = M.murmur_decode_attn_workspace(28, 256, 4, 4, 512, 256)
    check_plan(ws, split_partials(28 * 256 * 4, 2, 1), 28 * 256 * 4)
    with pytest.raises(M.MurmurError):
        M.murmur_decode_attn_workspace(1, 12, 28, 5, 850)
    with pytest.raises(M.MurmurError):
        M.murmur_decode_attn_workspace(1, 12, 28, 4, 850, 48)  # not a multiple of 32
    # splits of 64 and of 192 positions (multiples of one wavefront pass)
    check_plan(M.murmur_decode_attn_workspace(1, 12, 28, 4, 850, 64), split_partials(48, 14, 7), 48)
    check_plan(M.murmur_decode_attn_workspace(1, 12, 28, 4, 850, 192), split_partials(48, 5, 7), 48)
    with pytest.raises(M.MurmurError) as e:
        M.murmur_decode_attn_workspace(1, 12, 28, 4, 850, -1)  # negative split lengths are rejected
    assert e.value.code == M.MURMUR_EINVAL


def test_work_decode_division_is_exact():
    """The wide schedule's division x / d = high word of (x + 1)(ceil(2^32 / d) - 1), for x < 2^16 and
    1 <= d < 2^16 (the launch computes the multiplier, the kernel the product): every x for d up to 1024, and
    for every d the values around each multiple of d (x = kd - 1 and kd, where a short or long product
    would first show) and the largest x."""
    def magic(d):
        return ((1 << 32) + d - 1) // d - 1

    x = np.arange(1 << 16, dtype=np.uint64)
    for d in range(1, 1025):
        assert np.array_equal(((x + 1) * np.uint64(magic(d))) >> np.uint64(32), x // np.uint64(d)), d
    for d in range(1025, 1 << 16):
        k = np.arange(1, (1 << 16) // d + 1, dtype=np.uint64) * np.uint64(d)
        xs = np.concatenate([k - np.uint64(1), k[k < (1 << 16)], np.array([(1 << 16) - 1, 0], dtype=np.uint64)])
        assert magic(d) < (1 << 32)
        assert np.array_equal(((xs + 1) * np.uint64(magic(d))) >> np.uint64(32), xs // np.uint64(d)), d
    assert magic(1) == (1 << 32) - 1


def test_xcd_work_order_is_a_bijection():
    """The wide schedule's workgroup-to-work mapping (the launch packs per - 1 and the number of XCDs that take
    per = ceil(W / 8) items; the kernel maps workgroup w, which the hardware places on XCD w mod 8, to
    x (per - 1) + min(x, tall) + w // 8): a bijection of [0, W) in which every XCD takes one contiguous run,
    for every grid of up to 4096 workgroups."""
    for W in range(1, 4097):
        per = (W + 7) // 8
        per_m1, tall = per - 1, W - 8 * (per - 1)
        assert 1 <= tall <= 8
        work = [(w & 7) * per_m1 + min(w & 7, tall) + (w >> 3) for w in range(W)]
        assert sorted(work) == list(range(W)), W
        for x in range(8):
            run = [work[w] for w in range(x, W, 8)]
            assert run == list(range(run[0], run[0] + len(run))) if run else True, (W, x)


def test_decode_attn_accepts_any_larger_workspace():
    """Host validation (the workspace plan included) passes for the exact size and for larger ones; with no
    GPU the launch itself then fails with MURMUR_EHIP."""
    for split_len in (0, 256):
        ws = M.murmur_decode_attn_workspace(1, 12, 28, 4, 850, split_len)
        for w in (ws, ws + 1, ws + 65536 + 13, 4 * ws):
            assert call_attn(attn_args(split_len=split_len, ws_bytes=w)) == M.MURMUR_EHIP, (split_len, w)
        assert call_attn(attn_args(split_len=split_len, ws_bytes=ws - 1)) == M.MURMUR_ENOSPACE


def test_workspace_init_and_device_error_reject_null():
    lib = M.lib()
    assert lib.murmur_decode_attn_workspace_init(None, 1024, 0) == M.MURMUR_EINVAL
    assert lib.murmur_decode_attn_workspace_init(FAKE + 4, 1024, 0) == M.MURMUR_EINVAL
    assert lib.murmur_device_error(0, None) == M.MURMUR_EINVAL


def call_step(a, seg=FAKE, pol=FAKE, pol_per_seq=0):
    return M.lib().murmur_decode_step(seg, pol, pol_per_seq, a["q"], ctypes.byref(a["kv"]), a["idx"], a["count"],
                                      a["ranges"], a["max_keep"], a["B"], a["Hq"], a["Hkv"], a["D"], a["scale"],
                                      a["split_len"], a["out"], a["out_dtype"], a["lse"], a["ws"], a["ws_bytes"], 0)


@pytest.mark.parametrize("over,step_kw,code", [
    ({}, dict(seg=None), M.MURMUR_EINVAL),
    ({}, dict(pol=None), M.MURMUR_EINVAL),
    ({}, dict(pol_per_seq=4), M.MURMUR_EINVAL),
    ({}, dict(pol_per_seq=-1), M.MURMUR_EINVAL),
    (dict(split_len=-1), dict(pol_per_seq=M.MURMUR_POL_PER_LAYER), M.MURMUR_EINVAL),
    ({}, dict(seg=FAKE + 2), M.MURMUR_EINVAL),
    (dict(idx=FAKE + 1), {}, M.MURMUR_EINVAL),
    (dict(q=None), {}, M.MURMUR_EINVAL),
    (dict(D=64), {}, M.MURMUR_EUNSUPPORTED),
    (dict(split_len=100), {}, M.MURMUR_EINVAL),
    (dict(max_keep=0), {}, M.MURMUR_EINVAL),
    (dict(ws_bytes=1000), {}, M.MURMUR_ENOSPACE),
])
def test_decode_step_rejects(over, step_kw, code):
    assert call_step(attn_args(**over), **step_kw) == code
    assert M.murmur_last_error() != ""


def call_step_static(a, seg=FAKE, pol=FAKE, pol_per_seq=0):
    return M.lib().murmur_decode_step_static(seg, pol, pol_per_seq, a["q"], ctypes.byref(a["kv"]), a["idx"],
                                             a["count"], a["ranges"], a["max_keep"], a["B"], a["Hq"], a["Hkv"],
                                             a["D"], a["scale"], a["split_len"], a["out"], a["out_dtype"], a["lse"], 0)


@pytest.mark.parametrize("over,step_kw,code", [
    ({}, dict(seg=None), M.MURMUR_EINVAL),
    ({}, dict(pol_per_seq=4), M.MURMUR_EINVAL),
    (dict(q=None), {}, M.MURMUR_EINVAL),
    (dict(D=64), {}, M.MURMUR_EUNSUPPORTED),
    (dict(split_len=100), {}, M.MURMUR_EINVAL),
    # 48 groups cut into 27 splits of 32 positions: 4.7 MiB of partials, beyond the 4 MiB scratch
    (dict(split_len=32), {}, M.MURMUR_ENOSPACE),
    # 28 layers x 12 sequences x 4 KV heads = 1344 split groups need more tickets than the scratch holds
    (dict(kv=M.murmur_kv(FAKE, FAKE, 28, 4096, 0, 0, 0, 128), split_len=512, max_keep=1024), {},
     M.MURMUR_ENOSPACE),
])
def test_decode_step_static_rejects(over, step_kw, code):
    """The allocation-free step runs every check before any HIP call, including the scratch limit."""
    assert call_step_static(attn_args(**over), **step_kw) == code
    assert M.murmur_last_error() != ""


def test_decode_step_static_scratch_limit():
    """What fits: the calls whose workspace (same sizes and split_len) is at most MURMUR_STATIC_SCRATCH_BYTES."""
    limit = M.MURMUR_STATIC_SCRATCH_BYTES
    assert M.murmur_decode_attn_workspace(1, 12, 28, 4, 850, 0) <= limit        # 12 x 300 s chunks, eviction
    assert M.murmur_decode_attn_workspace(28, 12, 28, 4, 850, 0) <= limit       # 28 layers
    assert M.murmur_decode_attn_workspace(1, 1, 28, 4, 35160, 0) <= limit       # the hour-long single pass
    assert M.murmur_decode_attn_workspace(1, 12, 28, 4, 850, 32) > limit
    assert M.murmur_decode_attn_workspace(28, 12, 28, 4, 1024, 512) > limit
    # without a GPU a call that passes the checks fails at the first HIP call
    assert call_step_static(attn_args()) == M.MURMUR_EHIP


# ---- ring storage (host layout and argument checks) ----------------------------------------------

def expand(ranges_row):
    out = []
    for start, length in ranges_row:
        out.extend(range(int(start), int(start) + int(length)))
    return out


def test_ring_layout_host_matches_oracle_rows():
    """The six storage pieces hold exactly the oracle's retained tokens, mapped to their ring rows, and
    cur_row is the row the current token is written to (400 random layouts and policies)."""
    rng = np.random.default_rng(21)
    B = 400
    w_o = np.where(rng.random(B) < 0.2, OFF, rng.integers(1, 120, B))
    n_so = rng.integers(0, 8, B)
    j = rng.integers(1, 600, B)
    seg = np.stack([rng.integers(0, 40, B), rng.integers(0, 400, B), rng.integers(0, 20, B), j],
                   axis=1).astype(np.int32)
    pol = np.stack([np.where(rng.random(B) < 0.2, OFF, rng.integers(1, 300, B)), rng.integers(0, 300, B),
                    rng.integers(0, 30, B), w_o, n_so], axis=1).astype(np.int32)
    for cap in (130, 700):
        ok = (w_o <= cap) & ((w_o != OFF) | (j - n_so <= cap))
        seg_ok, pol_ok = seg[ok], pol[ok]
        ranges, cur = M.murmur_ring_layout_host(seg_ok, pol_ok, cap, 1)
        idx, cnt = oracle.retained(seg_ok, pol_ok)
        rows = OR.storage_rows(idx, cnt, seg_ok, pol_ok[:, 4], cap)
        for b in range(seg_ok.shape[0]):
            got = expand(ranges[b])
            assert sorted(got) == sorted(rows[b]) and len(got) == int(cnt[b])
            out0 = int(seg_ok[b, 0] + seg_ok[b, 1] + seg_ok[b, 2])
            assert cur[b] == OR.ring_row(int(seg_ok[b, 3]) - 1, out0, int(pol_ok[b, 4]), cap)
            assert np.all(ranges[b, :, 1] >= 0)


def expand_blocks(blocks_row):
    out = []
    for first, n in blocks_row:
        out.extend(range(int(first), int(first) + int(n)))
    return out


def test_freeable_blocks_host_matches_oracle():
    """The closed form's whole blocks equal the oracle's scan of later steps (300 random layouts, policies
    and block sizes, sinks and windows on and off), the speech part first."""
    rng = np.random.default_rng(31)
    B = 300
    seg = np.stack([rng.integers(0, 9, B), rng.integers(1, 90, B), rng.integers(0, 5, B), rng.integers(1, 80, B)],
                   axis=1).astype(np.int32)
    pol = np.stack([np.where(rng.random(B) < 0.2, OFF, rng.integers(1, 40, B)), rng.integers(0, 20, B),
                    rng.integers(0, 6, B), np.where(rng.random(B) < 0.2, OFF, rng.integers(1, 30, B)),
                    rng.integers(0, 5, B)], axis=1).astype(np.int32)
    for bs in (1, 3, 8):
        got = M.murmur_freeable_blocks_host(seg, pol, bs)
        for b in range(B):
            want = OP.freeable_blocks(seg[b], pol[b], bs)
            assert expand_blocks(got[b]) == want, (b, bs, seg[b], pol[b])


def test_freeable_blocks_host_rejects():
    seg = np.array([[32, 100, 0, 50]], dtype=np.int32)
    with pytest.raises(M.MurmurError):
        M.murmur_freeable_blocks_host(seg, np.array([0, 0, 0, -1, 0], dtype=np.int32), 16)  # window 0
    with pytest.raises(M.MurmurError):
        M.murmur_freeable_blocks_host(seg, np.array([-1, 0, 0, -1, 0], dtype=np.int32), 0)
    lib = M.lib()
    assert lib.murmur_freeable_blocks_host(None, None, 0, 1, 16, None) == M.MURMUR_EINVAL


def test_paged_step_argument_checks():
    """murmur_paged_step rejects bad arguments before any launch; valid ones reach the launch (MURMUR_EHIP
    without a GPU)."""
    lib = M.lib()
    kv = M.make_kv(FAKE, FAKE, 1, 4096, (4096 * 4 * 128, 0, 128, 4 * 128))

    def call(seg=FAKE, pol=FAKE, per_seq=0, B=12, bt=FAKE, max_blocks=8, bs=16, stack=FAKE, top=FAKE, cap=64,
             full=0, pool=None, hkv=4, kn=FAKE, vn=FAKE):
        return lib.murmur_paged_step(seg, pol, per_seq, B, bt, max_blocks, bs, stack, top, cap, full,
                                     ctypes.byref(pool) if pool is not None else None, hkv, kn, vn, None)

    for over in (dict(seg=None), dict(bt=None), dict(stack=None), dict(top=None), dict(B=0), dict(max_blocks=0),
                 dict(cap=0), dict(per_seq=2), dict(bs=12), dict(bs=0), dict(top=FAKE + 2), dict(full=2),
                 dict(pool=kv, kn=None), dict(pool=kv, hkv=0), dict(pool=kv, vn=FAKE + 8)):
        assert call(**over) == M.MURMUR_EINVAL, over
        assert M.murmur_last_error() != ""
    bad_kv = M.make_kv(FAKE, FAKE, 1, 4096, (4096 * 4 * 128, 0, 128, 100))
    assert call(pool=bad_kv) == M.MURMUR_EINVAL
    assert call() == M.MURMUR_EHIP
    assert call(pool=kv) == M.MURMUR_EHIP


def test_ring_layout_host_rejects_rings_too_small():
    seg = np.array([[32, 100, 0, 50]], dtype=np.int32)
    with pytest.raises(M.MurmurError):
        M.murmur_ring_layout_host(seg, np.array([OFF, 0, 0, 64, 0]), 63)  # cap < window
    with pytest.raises(M.MurmurError):
        M.murmur_ring_layout_host(seg, np.array([OFF, 0, 0, OFF, 2]), 47)  # keep-all, 48 ring tokens
    M.murmur_ring_layout_host(seg, np.array([OFF, 0, 0, OFF, 2]), 48)
    with pytest.raises(M.MurmurError):
        M.murmur_ring_layout_host(seg, np.array([OFF, 0, 0, 8, 0]), 0)


def call_ring_step(a, ring, seg=FAKE, pol=FAKE):
    return M.lib().murmur_decode_step_ring(seg, pol, 0, ctypes.byref(ring) if ring is not None else None, a["q"],
                                           ctypes.byref(a["kv"]), a["idx"], a["count"], a["ranges"], a["max_keep"],
                                           a["B"], a["Hq"], a["Hkv"], a["D"], a["scale"], a["split_len"], a["out"],
                                           a["out_dtype"], a["lse"], a["ws"], a["ws_bytes"], 0)


@pytest.mark.parametrize("over,ring,code", [
    ({}, None, M.MURMUR_EINVAL),
    ({}, M.murmur_ring(0, FAKE, FAKE), M.MURMUR_EINVAL),
    ({}, M.murmur_ring(256, None, FAKE), M.MURMUR_EINVAL),
    ({}, M.murmur_ring(256, FAKE + 8, FAKE), M.MURMUR_EINVAL),
    (dict(split_len=-1), M.murmur_ring(256, FAKE, FAKE), M.MURMUR_EINVAL),
    (dict(D=64), M.murmur_ring(256, FAKE, FAKE), M.MURMUR_EUNSUPPORTED),
    (dict(ws_bytes=1000), M.murmur_ring(256, FAKE, FAKE), M.MURMUR_ENOSPACE),
])
def test_decode_step_ring_rejects(over, ring, code):
    assert call_ring_step(attn_args(**over), ring) == code
    assert M.murmur_last_error() != ""


def test_ring_prefill_matches_the_oracle_appends():
    """decode.ring_prefill (the bench's placement of a prefilled state) equals the oracle's literal
    sequence of appends, row for row."""
    from paper_2606_01483_amd.decode import ring_prefill
    rng = np.random.default_rng(5)
    for _ in range(40):
        B = 3
        seg = np.stack([rng.integers(0, 9, B), rng.integers(0, 30, B), rng.integers(0, 5, B),
                        rng.integers(1, 90, B)], axis=1).astype(np.int32)
        n_so = rng.integers(0, 5, B)
        cap = int(rng.integers(1, 40))
        L = int((seg.sum(axis=1)).max())
        cache = rng.integers(1, 60000, size=(2, B, 2, L, 4)).astype(np.uint16)
        rows = max(OR.storage_len(seg[b], n_so[b], cap) for b in range(B))
        assert np.array_equal(ring_prefill(cache, seg, n_so, cap, rows), OR.append_all(cache, seg, n_so, cap, rows))


def test_read_probe_rejects():
    lib = M.lib()
    R, L = M.MURMUR_PROBE_REGISTERS, M.MURMUR_PROBE_LDS
    assert lib.murmur_read_probe(None, 1024, 256, 256, 8, R, FAKE, 0) == M.MURMUR_EINVAL
    assert lib.murmur_read_probe(FAKE, 1000, 256, 256, 8, R, FAKE, 0) == M.MURMUR_EINVAL
    assert lib.murmur_read_probe(FAKE, 0, 256, 256, 8, R, FAKE, 0) == M.MURMUR_EINVAL
    assert lib.murmur_read_probe(FAKE, 1024, 0, 256, 8, R, FAKE, 0) == M.MURMUR_EINVAL
    assert lib.murmur_read_probe(FAKE + 8, 1024, 256, 256, 8, R, FAKE, 0) == M.MURMUR_EINVAL
    for threads in (0, 32, 100, 1088):
        assert lib.murmur_read_probe(FAKE, 1024, 256, threads, 8, R, FAKE, 0) == M.MURMUR_EINVAL
    for depth in (0, 3, 32):
        assert lib.murmur_read_probe(FAKE, 1024, 256, 256, depth, R, FAKE, 0) == M.MURMUR_EINVAL
    assert lib.murmur_read_probe(FAKE, 1024, 256, 256, 8, 2, FAKE, 0) == M.MURMUR_EINVAL
    # direct-to-LDS: (threads / 64) * depth KiB of LDS, at most 64
    assert lib.murmur_read_probe(FAKE, 1024, 256, 1024, 8, L, FAKE, 0) == M.MURMUR_EINVAL
    assert b"LDS" in lib.murmur_last_error()


def test_evict_compact_paged_rejects():
    lib = M.lib()
    good = dict(seg=FAKE, pol=FAKE, per=0, B=12, bt=FAKE, mb=64, bs=16, idx=FAKE, mk=850, cnt=FAKE)

    def call(**over):
        a = dict(good, **over)
        return lib.murmur_evict_compact_paged(a["seg"], a["pol"], a["per"], a["B"], a["bt"], a["mb"], a["bs"],
                                              a["idx"], a["mk"], a["cnt"], None, 0)
    assert call(bt=None) == M.MURMUR_EINVAL
    assert call(bs=12) == M.MURMUR_EINVAL     # not a power of two
    assert call(bs=0) == M.MURMUR_EINVAL
    assert call(mb=0) == M.MURMUR_EINVAL
    assert call(per=2) == M.MURMUR_EINVAL
    assert call(bt=FAKE + 2) == M.MURMUR_EINVAL
    assert call(B=0) == M.MURMUR_EINVAL
