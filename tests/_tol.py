"""Parity criteria for the attention outputs.

fp32 accumulation against the fp64 oracle: 2e-3 maximum row-RMS-floored relative
error, i.e. an element's error is measured relative to max(|ref|, rms of its
128-wide output row), so that near-zero elements of a row are not judged on their
own scale.  A bf16 store adds at most half a bf16 ulp of the reference on top.
The lse gets an absolute-or-relative 1e-5 bound (fp32 logits of |s| <~ 10 carry
~1e-6).  The plain elementwise relative error |y - ref| / max(|ref|, 1e-6) is
reported beside it (rel_err_elementwise); elements far below their row's scale
make it large without any loss of accuracy in the row.
"""
import numpy as np

REL_TOL = 2e-3
LSE_TOL = 1e-5


def rel_err_fp32(y: np.ndarray, ref: np.ndarray) -> float:
    y = np.asarray(y, dtype=np.float64)
    rms = np.sqrt(np.mean(ref * ref, axis=-1, keepdims=True))
    denom = np.maximum(np.abs(ref), rms)
    return float(np.max(np.abs(y - ref) / denom))


ELEM_FLOOR = 1e-6


def rel_err_elementwise(y: np.ndarray, ref: np.ndarray, floor: float = ELEM_FLOOR) -> float:
    """max over elements of |y - ref| / max(|ref|, floor)."""
    y = np.asarray(y, dtype=np.float64)
    return float(np.max(np.abs(y - ref) / np.maximum(np.abs(ref), floor)))


def half_ulp_bf16(ref: np.ndarray) -> np.ndarray:
    a = np.abs(ref).astype(np.float64)
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -126)))
    return 2.0 ** (e - 8)  # bf16 has 8 significant bits: ulp = 2^(e-7), half ulp = 2^(e-8)


def bf16_excess(y: np.ndarray, ref: np.ndarray) -> float:
    """max over elements of (|y - ref| - half_ulp(ref)) / max(|ref|, rms): must be <= REL_TOL."""
    y = np.asarray(y, dtype=np.float64)
    rms = np.sqrt(np.mean(ref * ref, axis=-1, keepdims=True))
    denom = np.maximum(np.abs(ref), rms)
    return float(np.max((np.abs(y - ref) - half_ulp_bf16(ref)) / denom))


def lse_err(y: np.ndarray, ref: np.ndarray) -> float:
    return float(np.max(np.abs(np.asarray(y, dtype=np.float64) - ref) / np.maximum(1.0, np.abs(ref))))
