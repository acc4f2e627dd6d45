"""CPU oracle for AQLM dequantization and matrix products.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package.  The GPU library
never imports, links or calls it, and the two share no code.

The arithmetic lives in ``aqlm_oracle.c`` (plain C, fp64 products, built
without FMA contraction); this module only marshals numpy arrays into it.
What is computed follows Eq. 2 and Fig. 3 of the paper: the weight group
(i, j) is the sum over m of codeword ``codes[i, j, m]`` of codebook m, the
row is multiplied by the per-output scale ``scales[i]`` and rounded to fp16;
products are then taken in fp64.

Parity status: every function here is pinned by ``tests/test_oracle_pins.py``
(brute force from the one-hot form of Eq. 2, closed forms, invariants and an
exhaustive check of the fp16 rounding against numpy).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle_aqlm.so")
_lib = None

_ERRORS = {1: "null pointer", 2: "bad shape", 3: "unsupported (M, B, g)", 4: "code out of range"}


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _build  # noqa: WPS433 - builds the C file with gcc

        _build.build()
    lib = ctypes.CDLL(_LIB_PATH)
    p, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    lib.oracle_f16_to_f32.argtypes = [ctypes.c_uint16]
    lib.oracle_f16_to_f32.restype = ctypes.c_float
    lib.oracle_f32_to_f16.argtypes = [ctypes.c_float]
    lib.oracle_f32_to_f16.restype = ctypes.c_uint16
    lib.oracle_f32_to_f16_array.argtypes = [p, p, i64]
    lib.oracle_f32_to_f16_array.restype = None
    lib.oracle_f16_to_f32_array.argtypes = [p, p, i64]
    lib.oracle_f16_to_f32_array.restype = None
    lib.oracle_dequantize.argtypes = [p, p, p, i64, i64, i32, i32, i32, p]
    lib.oracle_dequantize.restype = ctypes.c_int
    lib.oracle_dequantize_rows.argtypes = [p, p, p, i64, i64, i32, i32, i32, p, i64, p]
    lib.oracle_dequantize_rows.restype = ctypes.c_int
    lib.oracle_matmul_f16.argtypes = [p, i64, i64, p, i64, p]
    lib.oracle_matmul_f16.restype = ctypes.c_int
    lib.oracle_backward.argtypes = [p, p, p, i64, i64, i32, i32, i32, i64, p, p, p, p]
    lib.oracle_backward.restype = ctypes.c_int
    lib.oracle_aq_loss.argtypes = [p, p, p, p, p, i64, i64, i32, i32, i32, p]
    lib.oracle_aq_loss.restype = ctypes.c_int
    lib.oracle_beam_search.argtypes = [p, p, p, p, p, i64, i64, i32, i32, i32, i32, i32, p]
    lib.oracle_beam_search.restype = ctypes.c_int
    lib.oracle_packed_row_bytes.argtypes = [i64, i32, i32, i32]
    lib.oracle_packed_row_bytes.restype = ctypes.c_int64
    lib.oracle_unpack_codes.argtypes = [p, i64, i64, i32, i32, i32, p]
    lib.oracle_unpack_codes.restype = ctypes.c_int
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_set_threads.argtypes = [ctypes.c_int]
    lib.oracle_set_threads.restype = None
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _bits16(a) -> np.ndarray:
    """fp16 array (or its uint16 bit pattern) -> contiguous uint16 bit pattern."""
    a = np.asarray(a)
    if a.dtype == np.float16:
        a = a.view(np.uint16)
    if a.dtype != np.uint16:
        raise TypeError(f"expected float16 or uint16 bit patterns, got {a.dtype}")
    return np.ascontiguousarray(a)


def _check(st: int):
    if st != 0:
        raise ValueError(f"oracle: {_ERRORS.get(st, st)}")


def num_threads() -> int:
    """Threads a parallel region of the oracle runs with."""
    return int(_load().oracle_num_threads())


def set_threads(n: int) -> None:
    """Threads for the oracle's later parallel regions (from this thread)."""
    _load().oracle_set_threads(int(n))


def f32_to_f16_bits(values) -> np.ndarray:
    """Round fp32 values to fp16 (nearest, ties to even); returns uint16 bits."""
    v = np.ascontiguousarray(np.asarray(values, dtype=np.float32))
    out = np.empty(v.shape, dtype=np.uint16)
    _load().oracle_f32_to_f16_array(_ptr(v), _ptr(out), v.size)
    return out


def f16_bits_to_f32(bits) -> np.ndarray:
    b = _bits16(bits)
    out = np.empty(b.shape, dtype=np.float32)
    _load().oracle_f16_to_f32_array(_ptr(b), _ptr(out), b.size)
    return out


def _layer_args(codes, codebooks, scales, g):
    codes = np.ascontiguousarray(codes)
    cb = _bits16(codebooks)
    sc = _bits16(scales)
    if codes.ndim != 3 or cb.ndim != 3:
        raise ValueError("codes must be [d_out, d_in/g, M] and codebooks [M, 2^B, g]")
    d_out, groups, M = codes.shape
    Mc, entries, gc = cb.shape
    if Mc != M or gc != g or sc.shape != (d_out,):
        raise ValueError("inconsistent codes / codebooks / scales shapes")
    B = int(entries).bit_length() - 1
    if (1 << B) != entries:
        raise ValueError("codebook entry count must be a power of two")
    want = np.uint8 if B <= 8 else np.uint16
    if codes.dtype != want:
        raise TypeError(f"codes for B={B} must be {np.dtype(want).name}")
    return codes, cb, sc, d_out, groups * g, M, B


def dequantize(codes, codebooks, scales, g: int = 8) -> np.ndarray:
    """Dequantized weight matrix as fp16 bit patterns, shape [d_out, d_in]."""
    codes, cb, sc, d_out, d_in, M, B = _layer_args(codes, codebooks, scales, g)
    w = np.empty((d_out, d_in), dtype=np.uint16)
    _check(_load().oracle_dequantize(_ptr(codes), _ptr(cb), _ptr(sc), d_out, d_in, M, B, g, _ptr(w)))
    return w


def dequantize_rows(codes, codebooks, scales, rows, g: int = 8) -> np.ndarray:
    """Only the listed rows of the dequantized matrix (fp16 bits, [len(rows), d_in])."""
    codes, cb, sc, d_out, d_in, M, B = _layer_args(codes, codebooks, scales, g)
    r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    w = np.empty((r.size, d_in), dtype=np.uint16)
    _check(_load().oracle_dequantize_rows(_ptr(codes), _ptr(cb), _ptr(sc), d_out, d_in, M, B, g,
                                          _ptr(r), r.size, _ptr(w)))
    return w


def matmul_f16(w_bits, x) -> np.ndarray:
    """fp64 product of an fp16 matrix [d_out, d_in] with fp16 rows x [n, d_in] -> [n, d_out]."""
    w = _bits16(w_bits)
    xb = _bits16(x)
    if xb.ndim == 1:
        xb = xb[None, :]
    d_out, d_in = w.shape
    n = xb.shape[0]
    if xb.shape[1] != d_in:
        raise ValueError("x has the wrong input width")
    y = np.empty((n, d_out), dtype=np.float64)
    _check(_load().oracle_matmul_f16(_ptr(w), d_out, d_in, _ptr(xb), n, _ptr(y)))
    return y


def aqlm_matmul(codes, codebooks, scales, x, g: int = 8) -> np.ndarray:
    """Reference Y[t, i] = sum_c W[i, c] x[t, c] in fp64 with W = dequantize(...); [n, d_out]."""
    return matmul_f16(dequantize(codes, codebooks, scales, g), x)


def backward(codes, codebooks, scales, x, dy, g: int = 8):
    """Gradients through Eq. 2 for y = x W^T and an upstream gradient dy [n, d_out]:
    returns (dcodebooks [M, 2^B, g], dscales [d_out]) in fp64, with
    G = dy^T x, dC_m[e, k] = sum over (i, j) coded e in codebook m of s_i G[i, j g + k]
    and ds_i = sum_c G[i, c] u[i, c] (u the fp32 codeword sums)."""
    codes, cb, sc, d_out, d_in, M, B = _layer_args(codes, codebooks, scales, g)
    xb = _bits16(x)
    db = _bits16(dy)
    if xb.ndim == 1:
        xb = xb[None, :]
    if db.ndim == 1:
        db = db[None, :]
    n = xb.shape[0]
    if xb.shape != (n, d_in) or db.shape != (n, d_out):
        raise ValueError("x must be [n, d_in] and dy [n, d_out]")
    dcb = np.empty((M, 1 << B, g), dtype=np.float64)
    ds = np.empty(d_out, dtype=np.float64)
    _check(_load().oracle_backward(_ptr(codes), _ptr(cb), _ptr(sc), d_out, d_in, M, B, g, n, _ptr(xb), _ptr(db),
                                   _ptr(dcb), _ptr(ds)))
    return dcb, ds


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32))


def aq_loss(w, h, codes, codebooks, scales, g: int = 8) -> np.ndarray:
    """Per-row objective (w_i - what_i) H (w_i - what_i)^T in fp64, what the exact
    (unrounded) reconstruction of Eq. 2 with scales; w [d_out, d_in], H [d_in, d_in]."""
    codes, cb, sc, d_out, d_in, M, B = _layer_args(codes, codebooks, scales, g)
    wf, hf = _f32(w), _f32(h)
    if wf.shape != (d_out, d_in) or hf.shape != (d_in, d_in):
        raise ValueError("w must be [d_out, d_in] and h [d_in, d_in]")
    out = np.empty(d_out, dtype=np.float64)
    _check(_load().oracle_aq_loss(_ptr(wf), _ptr(hf), _ptr(codes), _ptr(cb), _ptr(sc), d_out, d_in, M, B, g,
                                  _ptr(out)))
    return out


def beam_search(w, h, codes, codebooks, scales, beam: int, sweeps: int = 1, g: int = 8):
    """Phase-1 beam search over codes (fp64); returns (new codes, per-row loss).
    See aqlm_oracle.c for the step order and tie rules."""
    codes, cb, sc, d_out, d_in, M, B = _layer_args(codes, codebooks, scales, g)
    wf, hf = _f32(w), _f32(h)
    if wf.shape != (d_out, d_in) or hf.shape != (d_in, d_in):
        raise ValueError("w must be [d_out, d_in] and h [d_in, d_in]")
    out = codes.copy()
    loss = np.empty(d_out, dtype=np.float64)
    _check(_load().oracle_beam_search(_ptr(wf), _ptr(hf), _ptr(out), _ptr(cb), _ptr(sc), d_out, d_in, M, B, g,
                                      int(beam), int(sweeps), _ptr(loss)))
    return out, loss


def unpack_codes(packed, d_out: int, d_in: int, M: int, B: int, g: int = 8) -> np.ndarray:
    """Codes [d_out, d_in/g, M] (uint16) from bit-packed rows (see aqlm_oracle.c)."""
    lib = _load()
    pitch = int(lib.oracle_packed_row_bytes(d_in, M, B, g))
    pk = np.ascontiguousarray(np.asarray(packed, dtype=np.uint8)).reshape(-1)
    if pk.size != d_out * pitch:
        raise ValueError(f"packed codes must hold {d_out} rows of {pitch} bytes")
    out = np.empty((d_out, d_in // g, M), dtype=np.uint16)
    _check(lib.oracle_unpack_codes(_ptr(pk), d_out, d_in, M, B, g, _ptr(out)))
    return out


def dequantize_packed(packed, codebooks, scales, d_in: int, B: int, g: int = 8) -> np.ndarray:
    """Dequantized weights (fp16 bits) of a layer with bit-packed B-bit codes."""
    cb = _bits16(codebooks)
    M = cb.shape[0]
    d_out = np.asarray(scales).shape[0]
    codes = unpack_codes(packed, d_out, d_in, M, B, g)
    if (1 << B) != cb.shape[1]:
        raise ValueError("codebooks must hold 2^B codewords")
    return dequantize(codes if B > 8 else codes.astype(np.uint8), codebooks, scales, g)
