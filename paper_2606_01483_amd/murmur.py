"""ctypes binding of libmurmur.so (include/murmur.h), one Python function per C entry point.

Argument marshalling only: every step of the decode path runs in the HIP
kernels behind the C ABI.  Device buffers are torch tensors (or raw device
addresses); torch supplies memory and streams, nothing else.  The binding never
falls back to another implementation: if libmurmur.so is missing it raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmurmur.so")

MURMUR_OK, MURMUR_EINVAL, MURMUR_EUNSUPPORTED, MURMUR_ENOSPACE, MURMUR_EHIP = 0, -1, -2, -3, -4
MURMUR_DTYPE_BF16, MURMUR_DTYPE_F32 = 1, 2
MURMUR_DEVERR_OVERFLOW, MURMUR_DEVERR_POLICY, MURMUR_DEVERR_POSITION, MURMUR_DEVERR_COUNT = 1, 2, 4, 8
MURMUR_DEVERR_CAPACITY = 16
MURMUR_POL_PER_SEQ, MURMUR_POL_PER_LAYER = 1, 2
MURMUR_DEVERR_BLOCK = 32
MURMUR_DEVERR_POOL = 64
N_PIECES = 6
SPLIT_UNIT = 128

_ERROR_NAMES = {MURMUR_EINVAL: "EINVAL", MURMUR_EUNSUPPORTED: "EUNSUPPORTED", MURMUR_ENOSPACE: "ENOSPACE",
                MURMUR_EHIP: "EHIP"}


class murmur_seg(ctypes.Structure):
    _fields_ = [("prompt_pre", ctypes.c_int32), ("speech_len", ctypes.c_int32), ("prompt_mid", ctypes.c_int32),
                ("out_len", ctypes.c_int32)]


class murmur_policy(ctypes.Structure):
    _fields_ = [("speech_window", ctypes.c_int32), ("speech_delay", ctypes.c_int32),
                ("speech_sink", ctypes.c_int32), ("out_window", ctypes.c_int32), ("out_sink", ctypes.c_int32)]


class murmur_kv(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("n_layers", ctypes.c_int32),
                ("max_len", ctypes.c_int32), ("stride_layer", ctypes.c_int64), ("stride_b", ctypes.c_int64),
                ("stride_h", ctypes.c_int64), ("stride_pos", ctypes.c_int64)]


class murmur_ring(ctypes.Structure):
    _fields_ = [("out_capacity", ctypes.c_int32), ("k_new", ctypes.c_void_p), ("v_new", ctypes.c_void_p)]


class MurmurError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"{_ERROR_NAMES.get(code, code)}: {message}")
        self.code = code


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with paper_2606_01483_amd._build.build() "
                          "(there is no non-HIP fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    i32, i32p, vp, sz = ctypes.c_int32, ctypes.POINTER(ctypes.c_int32), ctypes.c_void_p, ctypes.c_size_t
    lib.murmur_abi_version.restype = ctypes.c_int
    lib.murmur_abi_version.argtypes = []
    lib.murmur_last_error.restype = ctypes.c_char_p
    lib.murmur_last_error.argtypes = []
    lib.murmur_retained_count_host.restype = ctypes.c_int
    lib.murmur_retained_count_host.argtypes = [ctypes.POINTER(murmur_seg), ctypes.POINTER(murmur_policy), i32, i32,
                                               i32p, i32p]
    lib.murmur_evict_compact.restype = ctypes.c_int
    lib.murmur_evict_compact.argtypes = [vp, vp, i32, i32, vp, i32, vp, vp, vp]
    lib.murmur_evict_compact_paged.restype = ctypes.c_int
    lib.murmur_evict_compact_paged.argtypes = [vp, vp, i32, i32, vp, i32, i32, vp, i32, vp, vp, vp]
    lib.murmur_decode_attn_workspace.restype = ctypes.c_int
    lib.murmur_decode_attn_workspace.argtypes = [i32, i32, i32, i32, i32, i32, ctypes.POINTER(sz)]
    lib.murmur_decode_attn_workspace_init.restype = ctypes.c_int
    lib.murmur_decode_attn_workspace_init.argtypes = [vp, sz, vp]
    lib.murmur_decode_attn.restype = ctypes.c_int
    lib.murmur_decode_attn.argtypes = [vp, ctypes.POINTER(murmur_kv), vp, vp, vp, i32, i32, i32, i32, i32,
                                       ctypes.c_float, i32, vp, i32, vp, vp, sz, vp]
    lib.murmur_decode_step.restype = ctypes.c_int
    lib.murmur_decode_step.argtypes = [vp, vp, i32, vp, ctypes.POINTER(murmur_kv), vp, vp, vp, i32, i32, i32, i32, i32,
                                       ctypes.c_float, i32, vp, i32, vp, vp, sz, vp]
    lib.murmur_decode_step_static.restype = ctypes.c_int
    lib.murmur_decode_step_static.argtypes = [vp, vp, i32, vp, ctypes.POINTER(murmur_kv), vp, vp, vp, i32, i32, i32,
                                              i32, i32, ctypes.c_float, i32, vp, i32, vp, vp]
    lib.murmur_ring_layout_host.restype = ctypes.c_int
    lib.murmur_ring_layout_host.argtypes = [ctypes.POINTER(murmur_seg), ctypes.POINTER(murmur_policy), i32, i32, i32,
                                            i32p, i32p]
    lib.murmur_freeable_blocks_host.restype = ctypes.c_int
    lib.murmur_freeable_blocks_host.argtypes = [ctypes.POINTER(murmur_seg), ctypes.POINTER(murmur_policy), i32, i32,
                                                i32, i32p]
    lib.murmur_paged_step.restype = ctypes.c_int
    lib.murmur_paged_step.argtypes = [vp, vp, i32, i32, vp, i32, i32, vp, vp, i32, i32, ctypes.POINTER(murmur_kv), i32,
                                      vp, vp, vp]
    lib.murmur_decode_step_ring.restype = ctypes.c_int
    lib.murmur_decode_step_ring.argtypes = [vp, vp, i32, ctypes.POINTER(murmur_ring), vp, ctypes.POINTER(murmur_kv),
                                            vp, vp, vp, i32, i32, i32, i32, i32, ctypes.c_float, i32, vp, i32, vp,
                                            vp, sz, vp]
    f64p = ctypes.POINTER(ctypes.c_double)
    lib.murmur_plan_chunks.restype = ctypes.c_int
    lib.murmur_plan_chunks.argtypes = [f64p, f64p, i32, ctypes.c_double, ctypes.c_double, ctypes.c_double, i32p,
                                       f64p, f64p, i32p, i32, i32p]
    lib.murmur_chunk_timestamps.restype = ctypes.c_int
    lib.murmur_chunk_timestamps.argtypes = [f64p, i32p, i32, f64p, i32, f64p]
    lib.murmur_read_probe.restype = ctypes.c_int
    lib.murmur_read_probe.argtypes = [vp, sz, i32, i32, i32, i32, vp, vp]
    lib.murmur_device_error.restype = ctypes.c_int
    lib.murmur_device_error.argtypes = [vp, i32p]
    _lib = lib
    return lib


def lib():
    """The loaded ctypes.CDLL (raises ImportError if libmurmur.so is not built)."""
    return _load()


def _check(rc: int) -> None:
    if rc != MURMUR_OK:
        raise MurmurError(rc, _load().murmur_last_error().decode())


def _addr(x) -> int | None:
    """Device address of a torch tensor (or an int address); None stays NULL."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _segs(seg) -> ctypes.Array:
    seg = np.ascontiguousarray(seg, dtype=np.int32).reshape(-1, 4)
    arr = (murmur_seg * seg.shape[0])()
    ctypes.memmove(arr, seg.ctypes.data, seg.nbytes)
    return arr


def _pols(pol) -> ctypes.Array:
    pol = np.ascontiguousarray(pol, dtype=np.int32).reshape(-1, 5)
    arr = (murmur_policy * pol.shape[0])()
    ctypes.memmove(arr, pol.ctypes.data, pol.nbytes)
    return arr


# ---- entry points --------------------------------------------------------------------------------

def murmur_abi_version() -> int:
    return _load().murmur_abi_version()


def murmur_last_error() -> str:
    return _load().murmur_last_error().decode()


def murmur_retained_count_host(seg, pol, pol_per_seq: int | None = None):
    """Host-only retained counts.  seg: int [B,4]; pol: int [5] or [B,5].  Returns (counts [B], max)."""
    seg_np = np.ascontiguousarray(seg, dtype=np.int32).reshape(-1, 4)
    pol_np = np.ascontiguousarray(pol, dtype=np.int32)
    if pol_per_seq is None:
        pol_per_seq = 1 if pol_np.ndim == 2 and pol_np.shape[0] > 1 else 0
    B = seg_np.shape[0]
    counts = np.zeros(B, dtype=np.int32)
    mx = ctypes.c_int32(0)
    _check(_load().murmur_retained_count_host(_segs(seg_np), _pols(pol_np), pol_per_seq, B,
                                              counts.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                              ctypes.byref(mx)))
    return counts, int(mx.value)


def murmur_evict_compact(seg_dev, pol_dev, pol_per_seq: int, B: int, idx_dev, max_keep: int, count_dev,
                         ranges_dev=None, stream=None) -> None:
    """seg_dev: int32 [B,4] device tensor; pol_dev: int32 [1 or B, 5]; idx_dev: int32 [B, max_keep];
    count_dev: int32 [B]; ranges_dev: int32 [B, 6, 2] or None."""
    _check(_load().murmur_evict_compact(_addr(seg_dev), _addr(pol_dev), pol_per_seq, B, _addr(idx_dev), max_keep,
                                        _addr(count_dev), _addr(ranges_dev), _stream(stream)))


def murmur_evict_compact_paged(seg_dev, pol_dev, pol_per_seq: int, B: int, block_table_dev, max_blocks: int,
                               block_size: int, idx_dev, max_keep: int, count_dev, ranges_dev=None,
                               stream=None) -> None:
    """murmur_evict_compact with the index list in rows of a paged pool (block_table_dev int32 [B, max_blocks])."""
    _check(_load().murmur_evict_compact_paged(_addr(seg_dev), _addr(pol_dev), pol_per_seq, B, _addr(block_table_dev),
                                              max_blocks, block_size, _addr(idx_dev), max_keep, _addr(count_dev),
                                              _addr(ranges_dev), _stream(stream)))


def murmur_decode_attn_workspace(n_layers: int, B: int, Hq: int, Hkv: int, max_keep: int, split_len: int = 0) -> int:
    nbytes = ctypes.c_size_t(0)
    _check(_load().murmur_decode_attn_workspace(n_layers, B, Hq, Hkv, max_keep, split_len, ctypes.byref(nbytes)))
    return int(nbytes.value)


def murmur_decode_attn_workspace_init(ws_dev, ws_bytes: int, stream=None) -> None:
    _check(_load().murmur_decode_attn_workspace_init(_addr(ws_dev), ws_bytes, _stream(stream)))


def make_kv(k, v, n_layers: int, max_len: int, strides) -> murmur_kv:
    """murmur_kv from device tensors (or addresses) and element strides (layer, b, head, pos)."""
    return murmur_kv(_addr(k), _addr(v), n_layers, max_len, *[int(s) for s in strides])


def kv_from_tensors(k, v) -> murmur_kv:
    """murmur_kv for bf16 tensors shaped [NL, B, Hkv, max_len, D] with unit head_dim stride."""
    if k.shape != v.shape or k.stride() != v.stride() or k.stride(-1) != 1:
        raise ValueError("k and v must share shape and strides, with a contiguous head dim")
    return make_kv(k, v, k.shape[0], k.shape[3], k.stride()[:4])


def murmur_decode_attn(q_dev, kv: murmur_kv, idx_dev, ranges_dev, count_dev, max_keep: int, B: int, Hq: int,
                       Hkv: int, D: int, scale: float, split_len: int, out_dev, out_dtype: int, lse_dev, ws_dev,
                       ws_bytes: int, stream=None) -> None:
    _check(_load().murmur_decode_attn(_addr(q_dev), ctypes.byref(kv), _addr(idx_dev), _addr(ranges_dev),
                                      _addr(count_dev), max_keep, B, Hq, Hkv, D, float(scale), split_len,
                                      _addr(out_dev), out_dtype, _addr(lse_dev), _addr(ws_dev), ws_bytes,
                                      _stream(stream)))


def murmur_decode_step(seg_dev, pol_dev, pol_per_seq: int, q_dev, kv: murmur_kv, idx_dev, count_dev, ranges_dev,
                       max_keep: int, B: int, Hq: int, Hkv: int, D: int, scale: float, split_len: int, out_dev,
                       out_dtype: int, lse_dev, ws_dev, ws_bytes: int, stream=None) -> None:
    """Eviction and attention of one decode step in one launch; idx/count/ranges outputs are optional."""
    _check(_load().murmur_decode_step(_addr(seg_dev), _addr(pol_dev), pol_per_seq, _addr(q_dev), ctypes.byref(kv),
                                      _addr(idx_dev), _addr(count_dev), _addr(ranges_dev), max_keep, B, Hq, Hkv, D,
                                      float(scale), split_len, _addr(out_dev), out_dtype, _addr(lse_dev),
                                      _addr(ws_dev), ws_bytes, _stream(stream)))


def murmur_decode_step_static(seg_dev, pol_dev, pol_per_seq: int, q_dev, kv: murmur_kv, idx_dev, count_dev,
                              ranges_dev, max_keep: int, B: int, Hq: int, Hkv: int, D: int, scale: float,
                              split_len: int, out_dev, out_dtype: int, lse_dev, stream=None) -> None:
    """murmur_decode_step without a workspace: tickets and partials in the library's per-device scratch."""
    _check(_load().murmur_decode_step_static(_addr(seg_dev), _addr(pol_dev), pol_per_seq, _addr(q_dev),
                                             ctypes.byref(kv), _addr(idx_dev), _addr(count_dev), _addr(ranges_dev),
                                             max_keep, B, Hq, Hkv, D, float(scale), split_len, _addr(out_dev),
                                             out_dtype, _addr(lse_dev), _stream(stream)))


MURMUR_STATIC_SCRATCH_BYTES = 4 << 20


def murmur_ring_layout_host(seg, pol, out_capacity: int, pol_per_seq: int | None = None):
    """Host-only ring-storage layout.  Returns (ranges int32 [B, 6, 2], cur_row int32 [B])."""
    seg_np = np.ascontiguousarray(seg, dtype=np.int32).reshape(-1, 4)
    pol_np = np.ascontiguousarray(pol, dtype=np.int32)
    if pol_per_seq is None:
        pol_per_seq = 1 if pol_np.ndim == 2 and pol_np.shape[0] > 1 else 0
    B = seg_np.shape[0]
    ranges = np.zeros((B, N_PIECES, 2), dtype=np.int32)
    cur = np.zeros(B, dtype=np.int32)
    i32p = ctypes.POINTER(ctypes.c_int32)
    _check(_load().murmur_ring_layout_host(_segs(seg_np), _pols(pol_np), pol_per_seq, B, int(out_capacity),
                                           ranges.ctypes.data_as(i32p), cur.ctypes.data_as(i32p)))
    return ranges, cur


def murmur_freeable_blocks_host(seg, pol, block_size: int, pol_per_seq: int | None = None) -> np.ndarray:
    """Host-only: whole logical blocks no later step retains.  Returns int32 [B, 2, 2]: (first block, number of
    blocks) of the speech part, then of the output part."""
    seg_np = np.ascontiguousarray(seg, dtype=np.int32).reshape(-1, 4)
    pol_np = np.ascontiguousarray(pol, dtype=np.int32)
    if pol_per_seq is None:
        pol_per_seq = 1 if pol_np.ndim == 2 and pol_np.shape[0] > 1 else 0
    B = seg_np.shape[0]
    blocks = np.zeros((B, 2, 2), dtype=np.int32)
    _check(_load().murmur_freeable_blocks_host(_segs(seg_np), _pols(pol_np), pol_per_seq, B, int(block_size),
                                               blocks.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))))
    return blocks


def murmur_paged_step(seg_dev, pol_dev, pol_per_seq: int, B: int, block_table_dev, max_blocks: int, block_size: int,
                      free_stack_dev, free_top_dev, capacity: int, full_scan: bool = False,
                      pool: murmur_kv | None = None, Hkv: int = 0, k_new_dev=None, v_new_dev=None,
                      stream=None) -> None:
    """Device block manager of a paged cache for one decode step (free, allocate, append the current K/V)."""
    _check(_load().murmur_paged_step(_addr(seg_dev), _addr(pol_dev), pol_per_seq, B, _addr(block_table_dev),
                                     max_blocks, block_size, _addr(free_stack_dev), _addr(free_top_dev), capacity,
                                     int(bool(full_scan)), ctypes.byref(pool) if pool is not None else None, Hkv,
                                     _addr(k_new_dev), _addr(v_new_dev), _stream(stream)))


def make_ring(out_capacity: int, k_new, v_new) -> murmur_ring:
    """murmur_ring from the ring size and the current token's K/V (device tensors [NL, B, Hkv, D] or addresses)."""
    return murmur_ring(int(out_capacity), _addr(k_new), _addr(v_new))


def murmur_decode_step_ring(seg_dev, pol_dev, pol_per_seq: int, ring: murmur_ring, q_dev, kv: murmur_kv, idx_dev,
                            count_dev, ranges_dev, max_keep: int, B: int, Hq: int, Hkv: int, D: int, scale: float,
                            split_len: int, out_dev, out_dtype: int, lse_dev, ws_dev, ws_bytes: int,
                            stream=None) -> None:
    """Eviction, attention and the current token's append on ring storage, in one launch."""
    _check(_load().murmur_decode_step_ring(_addr(seg_dev), _addr(pol_dev), pol_per_seq, ctypes.byref(ring),
                                           _addr(q_dev), ctypes.byref(kv), _addr(idx_dev), _addr(count_dev),
                                           _addr(ranges_dev), max_keep, B, Hq, Hkv, D, float(scale), split_len,
                                           _addr(out_dev), out_dtype, _addr(lse_dev), _addr(ws_dev), ws_bytes,
                                           _stream(stream)))


def murmur_plan_chunks(seg_start, seg_end, audio_len: float, max_chunk: float = 300.0,
                       tokens_per_s: float = 7.5):
    """Chunked inference plan (host only).  Returns (chunk_start, chunk_len, speech_tokens, chunk_of_seg)."""
    s0 = np.ascontiguousarray(seg_start, dtype=np.float64)
    s1 = np.ascontiguousarray(seg_end, dtype=np.float64)
    n_seg = int(s0.shape[0])
    f64p, i32p = ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int32)
    n = ctypes.c_int32(0)
    cap = max(1, n_seg + 1)
    while True:
        cs, cl = np.zeros(cap), np.zeros(cap)
        tok, of = np.zeros(cap, dtype=np.int32), np.zeros(max(1, n_seg), dtype=np.int32)
        rc = _load().murmur_plan_chunks(s0.ctypes.data_as(f64p), s1.ctypes.data_as(f64p), n_seg, float(audio_len),
                                        float(max_chunk), float(tokens_per_s), of.ctypes.data_as(i32p),
                                        cs.ctypes.data_as(f64p), cl.ctypes.data_as(f64p), tok.ctypes.data_as(i32p),
                                        cap, ctypes.byref(n))
        if rc == MURMUR_ENOSPACE and n.value > cap:
            cap = n.value
            continue
        _check(rc)
        k = n.value
        return cs[:k], cl[:k], tok[:k], of[:n_seg]


def murmur_chunk_timestamps(t_local, chunk, chunk_len):
    """Equation 4 (host only): absolute timestamps from chunk-relative ones."""
    tl = np.ascontiguousarray(t_local, dtype=np.float64)
    ch = np.ascontiguousarray(chunk, dtype=np.int32)
    cl = np.ascontiguousarray(chunk_len, dtype=np.float64)
    out = np.zeros_like(tl)
    f64p, i32p = ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int32)
    _check(_load().murmur_chunk_timestamps(tl.ctypes.data_as(f64p), ch.ctypes.data_as(i32p), int(tl.shape[0]),
                                           cl.ctypes.data_as(f64p), int(cl.shape[0]), out.ctypes.data_as(f64p)))
    return out


MURMUR_PROBE_REGISTERS = 0
MURMUR_PROBE_LDS = 1


def murmur_read_probe(buf_dev, nbytes: int, n_workgroups: int, sink_dev, threads: int = 256, depth: int = 8,
                      mode: int = MURMUR_PROBE_REGISTERS, stream=None) -> None:
    """Read-only streaming probe over buf_dev[0, nbytes) (measurement of the practical read ceiling):
    n_workgroups workgroups of `threads` threads, `depth` 16-byte loads per thread in flight, into
    registers (MURMUR_PROBE_REGISTERS) or straight to LDS (MURMUR_PROBE_LDS)."""
    _check(_load().murmur_read_probe(_addr(buf_dev), int(nbytes), int(n_workgroups), int(threads), int(depth),
                                     int(mode), _addr(sink_dev), _stream(stream)))


def murmur_device_error(stream=None) -> int:
    code = ctypes.c_int32(0)
    _check(_load().murmur_device_error(_stream(stream), ctypes.byref(code)))
    return int(code.value)
