"""fp64 CPU oracle for Murmur's decode-step attention -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The GPU path never calls it, and it
imports nothing from the GPU package.

The arithmetic lives in ``murmur_oracle.c`` (plain C, fp64, built with gcc);
this module compiles it and marshals numpy arrays through ctypes.

What it computes (paper, Section 3.2):
  * ``retained``: the kept KV positions of every sequence at output step j, from
    Algorithm 1 (output tokens, sinks plus a recent window), Algorithm 2 with
    Equation 2's sinks (speech tokens, a delayed sliding window), and the two
    system prompts, which are always kept;
  * ``attend``: Equation 1's softmax attention of the current token over exactly
    those positions, in fp64, with the log-sum-exp of the logits.

Pins: every function here is checked in ``tests/test_oracle_*.py`` against
values the paper prints (Equation 3's speed-up ratios), closed forms, library
routines (torch scaled-dot-product attention, scipy logsumexp/softmax) and
brute force on tiny inputs.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "murmur_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

SEG_FIELDS = 4  # prompt_pre, speech_len, prompt_mid, out_len (j)
POL_FIELDS = 5  # speech_window, speech_delay, speech_sink, out_window, out_sink


def build(force: bool = False) -> str:
    """Compile murmur_oracle.c into liboracle.so with gcc (no fast-math, no FMA contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
               "-pthread", "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        i32p = ctypes.POINTER(ctypes.c_int32)
        u16p = ctypes.POINTER(ctypes.c_uint16)
        f64p = ctypes.POINTER(ctypes.c_double)
        lib.oracle_retained.argtypes = [i32p, i32p, ctypes.c_int32, ctypes.c_int32, i32p, ctypes.c_int32, i32p]
        lib.oracle_retained.restype = ctypes.c_int
        lib.oracle_attn.argtypes = [u16p, u16p, u16p] + [ctypes.c_int32] * 6 + [i32p, i32p, ctypes.c_int32,
                                                                                 ctypes.c_double, f64p, f64p,
                                                                                 ctypes.c_int32]
        lib.oracle_attn.restype = ctypes.c_int
        lib.oracle_abi_version.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def retained(seg: np.ndarray, pol: np.ndarray, max_keep: int | None = None):
    """Retained positions per sequence.

    seg: int32 [B, 4] rows (prompt_pre, speech_len, prompt_mid, out_len j >= 1).
    pol: int32 [5] (shared) or [B, 5] (per sequence) rows
         (speech_window, speech_delay, speech_sink, out_window, out_sink); -1 window = keep all.
    Returns (idx int32 [B, max_keep] ascending, padded with -1; count int32 [B]).
    With max_keep None the list is sized to the largest count.
    """
    lib = _load()
    seg = np.ascontiguousarray(seg, dtype=np.int32).reshape(-1, SEG_FIELDS)
    pol = np.ascontiguousarray(pol, dtype=np.int32)
    per_seq = 1 if pol.ndim == 2 else 0
    pol = pol.reshape(-1, POL_FIELDS)
    if per_seq and pol.shape[0] != seg.shape[0]:
        raise ValueError("per-sequence policy needs one row per sequence")
    B = seg.shape[0]
    count = np.zeros(B, dtype=np.int32)
    if max_keep is None:
        dummy = np.zeros(1, dtype=np.int32)
        rc = lib.oracle_retained(_ptr(seg, ctypes.c_int32), _ptr(pol, ctypes.c_int32), per_seq, B,
                                 _ptr(dummy, ctypes.c_int32), 0, _ptr(count, ctypes.c_int32))
        if rc == -1:
            raise ValueError("oracle_retained: invalid layout or policy")
        max_keep = max(1, int(count.max()) if B else 1)
    idx = np.full((B, max_keep), -1, dtype=np.int32)
    rc = lib.oracle_retained(_ptr(seg, ctypes.c_int32), _ptr(pol, ctypes.c_int32), per_seq, B,
                             _ptr(idx, ctypes.c_int32), max_keep, _ptr(count, ctypes.c_int32))
    if rc == -1:
        raise ValueError("oracle_retained: invalid layout or policy")
    if rc == -2:
        raise ValueError("oracle_retained: max_keep smaller than a retained count")
    return idx, count


def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, idx: np.ndarray, count: np.ndarray,
           scale: float = 1.0, n_threads: int = 1):
    """Equation 1 over the retained set, fp64.

    q: uint16 bf16 bits [NL, B, Hq, D]; k, v: uint16 bf16 bits [NL, B, Hkv, Lmax, D];
    idx: int32 [B, max_keep]; count: int32 [B].
    Returns (out float64 [NL, B, Hq, D], lse float64 [NL, B, Hq]).
    """
    lib = _load()
    q = np.ascontiguousarray(q, dtype=np.uint16)
    k = np.ascontiguousarray(k, dtype=np.uint16)
    v = np.ascontiguousarray(v, dtype=np.uint16)
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    count = np.ascontiguousarray(count, dtype=np.int32)
    NL, B, Hq, D = q.shape
    _, _, Hkv, Lmax, _ = k.shape
    if k.shape != (NL, B, Hkv, Lmax, D) or v.shape != k.shape:
        raise ValueError("k/v shape mismatch")
    if idx.shape[0] != B or count.shape != (B,):
        raise ValueError("idx/count shape mismatch")
    out = np.zeros((NL, B, Hq, D), dtype=np.float64)
    lse = np.zeros((NL, B, Hq), dtype=np.float64)
    rc = lib.oracle_attn(_ptr(q, ctypes.c_uint16), _ptr(k, ctypes.c_uint16), _ptr(v, ctypes.c_uint16),
                         NL, B, Hq, Hkv, D, Lmax, _ptr(idx, ctypes.c_int32), _ptr(count, ctypes.c_int32),
                         idx.shape[1], float(scale), _ptr(out, ctypes.c_double), _ptr(lse, ctypes.c_double),
                         int(n_threads))
    if rc == -3:
        raise ArithmeticError("oracle_attn: softmax weights did not sum to one")
    if rc != 0:
        raise ValueError("oracle_attn: invalid input")
    return out, lse
