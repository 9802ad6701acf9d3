"""SBVR CPU oracle -- test infrastructure.

Plain, slow, binary64 reference for what the SBVR GEMV path computes
(Bang et al., "SBVR: Summation of BitVector Representation for Efficient LLM
Quantization").  Only the tests, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` may import this package; the HIP library never
does, and this package never imports the HIP library.

The arithmetic lives in ``sbvr_oracle.c`` (plain C11, IEEE binary64, no
contraction).  This module only marshals numpy arrays into it.

Parity notes: the oracle functions are pinned by the ``-m "not gpu"`` tests in
``tests/test_oracle_*.py``; the generator of the synthetic inputs (``synth``)
is "parity unpinned" beyond determinism and moment checks, since it is
synthetic by design.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np

from .build import build as _build, library_path

GROUP = 128  # weights per SBVR group along the GEMV inner dimension (Sec. 4.1)


class _Params(C.Structure):
    _fields_ = [
        ("n_ratio1", C.c_int),
        ("n_ratio2", C.c_int),
        ("n_scale", C.c_int),
        ("n_bias", C.c_int),
        ("normalise", C.c_int),
    ]


@dataclass(frozen=True)
class SearchParams:
    """Sizes of the coefficient search space (Sec. 4.2, Eqs. 5-7).

    The paper defers the values to an appendix that is not available; these
    defaults are the documented reading: |R1| = |R2| = 8, N_scale = 16,
    N_bias = 4, so |S| = 1024 entries.  ``normalise`` selects the
    span-normalised (True) or literal (False) reading of Eq. 4.
    """

    n_ratio1: int = 8
    n_ratio2: int = 8
    n_scale: int = 16
    n_bias: int = 4
    normalise: bool = True

    def c(self) -> _Params:
        return _Params(self.n_ratio1, self.n_ratio2, self.n_scale, self.n_bias, int(self.normalise))

    @property
    def size(self) -> int:
        return (self.n_ratio1 + self.n_ratio2) * self.n_scale * self.n_bias


DEFAULT = SearchParams()

_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        path = library_path()
        if not os.path.exists(path):
            _build()
        lib = C.CDLL(path)
        P = C.POINTER
        dp, fp, u16p, u32p, u8p, ip = (P(C.c_double), P(C.c_float), P(C.c_uint16),
                                        P(C.c_uint32), P(C.c_uint8), P(C.c_int))
        sig = {
            "oracle_fp16_to_double": (C.c_double, [C.c_uint16]),
            "oracle_fp16_from_double": (C.c_uint16, [C.c_double]),
            "oracle_quantile_linear": (C.c_double, [dp, C.c_int, C.c_double]),
            "oracle_candidate_count": (C.c_int, [P(_Params)]),
            "oracle_candidate_sets": (None, [dp, C.c_int, C.c_int, P(_Params), dp, dp, dp]),
            "oracle_entry_coeffs": (C.c_int, [C.c_double, C.c_double, C.c_double, C.c_int, C.c_int, u16p]),
            "oracle_subset_sums": (None, [u16p, C.c_int, dp]),
            "oracle_nearest": (C.c_int, [dp, C.c_int, C.c_double]),
            "oracle_entry_mse": (C.c_double, [dp, C.c_int, u16p, C.c_int]),
            "oracle_encode_group": (C.c_double, [dp, C.c_int, C.c_int, P(_Params), u16p, u8p, ip]),
            "oracle_encode_matrix": (C.c_int, [C.c_int, C.c_int, C.c_int, fp, P(_Params), C.c_int,
                                               u32p, u16p, dp]),
            "oracle_encode_matrix_cached": (C.c_int, [C.c_int, C.c_int, C.c_int, fp, P(_Params), C.c_int,
                                                      C.c_int, u32p, u16p, dp, u8p]),
            "oracle_decompress": (None, [C.c_int, C.c_int, C.c_int, u32p, u16p, dp]),
            "oracle_gemv_dense": (None, [C.c_int, C.c_int, dp, dp, dp]),
            "oracle_sbvr_gemv": (C.c_int, [C.c_int, C.c_int, C.c_int, u32p, u16p, u16p, C.c_int,
                                           ip, C.c_int, C.c_int, dp]),
            "oracle_sbvr_gemv_f64": (C.c_int, [C.c_int, C.c_int, C.c_int, u32p, u16p, dp, C.c_int,
                                               ip, C.c_int, C.c_int, dp]),
            "oracle_act_quantize": (C.c_int, [C.c_int, C.c_int, u16p, P(C.c_int32), fp]),
            "oracle_act_planes": (None, [C.c_int, C.c_int, P(C.c_int32), u8p]),
            "oracle_act_decode": (None, [C.c_int, C.c_int, u8p, fp, dp]),
            "oracle_rtn_sym_mse": (C.c_double, [dp, C.c_int, C.c_int]),
            "oracle_rtn_asym_mse": (C.c_double, [dp, C.c_int, C.c_int]),
        }
        for name, (res, args) in sig.items():
            f = getattr(lib, name)
            f.restype = res
            f.argtypes = args
        _LIB = lib
    return _LIB


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(C.POINTER(ctype))


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


# --------------------------------------------------------------------------
# binary16 helpers
# --------------------------------------------------------------------------

def fp16_to_double(bits: int) -> float:
    return _lib().oracle_fp16_to_double(int(bits) & 0xFFFF)


def fp16_from_double(v: float) -> int:
    """Nearest binary16 (ties to even) of a binary64 value, as bit pattern."""
    return int(_lib().oracle_fp16_from_double(float(v)))


def fp16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    lib = _lib()
    flat = np.asarray(bits, dtype=np.uint16).ravel()
    return np.array([lib.oracle_fp16_to_double(int(b)) for b in flat]).reshape(np.shape(bits))


# --------------------------------------------------------------------------
# Search space, Algorithm 1
# --------------------------------------------------------------------------

def quantile_linear(data, q: float) -> float:
    d = _f64(data)
    return _lib().oracle_quantile_linear(_ptr(d, C.c_double), d.size, float(q))


def candidate_sets(D, K: int, params: SearchParams = DEFAULT):
    """(R, S, B) candidate arrays of Eqs. 5-11 for group data D."""
    d = _f64(D)
    R = np.zeros(params.n_ratio1 + params.n_ratio2)
    S = np.zeros(params.n_scale)
    B = np.zeros(params.n_bias)
    p = params.c()
    _lib().oracle_candidate_sets(_ptr(d, C.c_double), d.size, K, C.byref(p),
                                 _ptr(R, C.c_double), _ptr(S, C.c_double), _ptr(B, C.c_double))
    return R, S, B


def entry_coeffs(r: float, s: float, b: float, K: int, normalise: bool = True):
    """fp16 bit patterns of one entry's coefficient set (Eq. 4) and finiteness."""
    out = np.zeros(K, dtype=np.uint16)
    ok = _lib().oracle_entry_coeffs(float(r), float(s), float(b), K, int(normalise),
                                    _ptr(out, C.c_uint16))
    return out, bool(ok)


def subset_sums(coeff_bits) -> np.ndarray:
    """AllSubsetSums of fp16 coefficient bit patterns; index p = sum bit_i 2^i."""
    c = np.ascontiguousarray(coeff_bits, dtype=np.uint16)
    K = c.size
    out = np.zeros(1 << K)
    _lib().oracle_subset_sums(_ptr(c, C.c_uint16), K, _ptr(out, C.c_double))
    return out


def nearest(sums, x: float) -> int:
    s = _f64(sums)
    K = int(np.log2(s.size))
    return _lib().oracle_nearest(_ptr(s, C.c_double), K, float(x))


def entry_mse(D, coeff_bits) -> float:
    d = _f64(D)
    c = np.ascontiguousarray(coeff_bits, dtype=np.uint16)
    return _lib().oracle_entry_mse(_ptr(d, C.c_double), d.size, _ptr(c, C.c_uint16), c.size)


def encode_group(D, K: int, params: SearchParams = DEFAULT):
    """Algorithm 1 on one group: (coeff bits [K], codes [n], mse, entry index)."""
    d = _f64(D)
    coeffs = np.zeros(K, dtype=np.uint16)
    codes = np.zeros(d.size, dtype=np.uint8)
    entry = C.c_int(0)
    p = params.c()
    mse = _lib().oracle_encode_group(_ptr(d, C.c_double), d.size, K, C.byref(p),
                                     _ptr(coeffs, C.c_uint16), _ptr(codes, C.c_uint8),
                                     C.byref(entry))
    return coeffs, codes, mse, entry.value


def encode_matrix(W: np.ndarray, K: int, params: SearchParams = DEFAULT, nthreads: int = 0,
                  want_mse: bool = False):
    """Encode an fp32 [O][I] matrix into canonical SBVR.

    Returns (planes uint32 [O][G][K][4], coeffs uint16 [O][G][K][, mse [O][G]]).
    """
    W = np.ascontiguousarray(W, dtype=np.float32)
    O, I = W.shape
    G = I // GROUP
    planes = np.zeros((O, G, K, 4), dtype=np.uint32)
    coeffs = np.zeros((O, G, K), dtype=np.uint16)
    mse = np.zeros((O, G)) if want_mse else None
    p = params.c()
    rc = _lib().oracle_encode_matrix(O, I, K, _ptr(W, C.c_float), C.byref(p), int(nthreads),
                                     _ptr(planes, C.c_uint32), _ptr(coeffs, C.c_uint16),
                                     _ptr(mse, C.c_double) if want_mse else None)
    if rc < 0:
        raise ValueError(f"oracle_encode_matrix rejected shape {O}x{I}, K={K}")
    return (planes, coeffs, mse) if want_mse else (planes, coeffs)


ENCODER_CACHE_MAX = 64


def encode_matrix_cached(W: np.ndarray, K: int, slots: int, params: SearchParams = DEFAULT,
                         nthreads: int = 0):
    """The encoder with the cache of Sec. 4.2 (reading R14): per row, the
    coefficient sets of its last `slots` searched groups are tried first and
    the best one is kept when its MSE is below the mean MSE of the row's
    earlier groups.  Returns (planes, coeffs, mse [O][G], hits uint8 [O][G])."""
    W = np.ascontiguousarray(W, dtype=np.float32)
    O, I = W.shape
    G = I // GROUP
    planes = np.zeros((O, G, K, 4), dtype=np.uint32)
    coeffs = np.zeros((O, G, K), dtype=np.uint16)
    mse = np.zeros((O, G))
    hits = np.zeros((O, G), dtype=np.uint8)
    p = params.c()
    rc = _lib().oracle_encode_matrix_cached(O, I, K, _ptr(W, C.c_float), C.byref(p), int(slots), int(nthreads),
                                            _ptr(planes, C.c_uint32), _ptr(coeffs, C.c_uint16),
                                            _ptr(mse, C.c_double), _ptr(hits, C.c_uint8))
    if rc < 0:
        raise ValueError(f"oracle_encode_matrix_cached rejected shape {O}x{I}, K={K}, slots={slots}")
    return planes, coeffs, mse, hits


# --------------------------------------------------------------------------
# Decompression and fp64 GEMV
# --------------------------------------------------------------------------

def decompress(planes: np.ndarray, coeffs: np.ndarray) -> np.ndarray:
    planes = np.ascontiguousarray(planes, dtype=np.uint32)
    coeffs = np.ascontiguousarray(coeffs, dtype=np.uint16)
    O, G, K, _ = planes.shape
    I = G * GROUP
    out = np.zeros((O, I))
    _lib().oracle_decompress(O, I, K, _ptr(planes, C.c_uint32), _ptr(coeffs, C.c_uint16),
                             _ptr(out, C.c_double))
    return out


def gemv_dense(W: np.ndarray, x: np.ndarray) -> np.ndarray:
    W = _f64(W)
    x = _f64(x)
    O, I = W.shape
    y = np.zeros(O)
    _lib().oracle_gemv_dense(O, I, _ptr(W, C.c_double), _ptr(x, C.c_double), _ptr(y, C.c_double))
    return y


def sbvr_gemv(planes: np.ndarray, coeffs: np.ndarray, x_fp16: np.ndarray, rows=None,
              nthreads: int = 0, return_threads: bool = False):
    """y = W_hat x in binary64 for fp16 activations x [I] or [B][I].

    ``rows`` restricts the output to a list of row indices (sampled parity at
    full size); the result is [n_rows] or [B][n_rows].
    """
    planes = np.ascontiguousarray(planes, dtype=np.uint32)
    coeffs = np.ascontiguousarray(coeffs, dtype=np.uint16)
    O, G, K, _ = planes.shape
    I = G * GROUP
    x = np.asarray(x_fp16)
    if x.dtype == np.float16:
        x = x.view(np.uint16)
    squeeze = x.ndim == 1
    x = np.ascontiguousarray(x.reshape(-1, I), dtype=np.uint16)
    B = x.shape[0]
    if rows is None:
        rows_arr, n_rows = None, O
    else:
        rows_arr = np.ascontiguousarray(rows, dtype=np.int32)
        if rows_arr.size and (rows_arr.min() < 0 or rows_arr.max() >= O):
            raise IndexError("row index out of range")
        n_rows = rows_arr.size
    y = np.zeros((B, n_rows))
    nt = _lib().oracle_sbvr_gemv(O, I, K, _ptr(planes, C.c_uint32), _ptr(coeffs, C.c_uint16),
                                 _ptr(x, C.c_uint16), B,
                                 _ptr(rows_arr, C.c_int) if rows_arr is not None else None,
                                 n_rows, int(nthreads), _ptr(y, C.c_double))
    if nt < 0:
        raise ValueError("oracle_sbvr_gemv rejected its arguments")
    y = y[0] if squeeze else y
    return (y, nt) if return_threads else y


# --------------------------------------------------------------------------
# Online activation conversion (Sec. 4.3, Eq. 12) and the W4A8 GEMV reference
# --------------------------------------------------------------------------

ACT_BITS = 8  # l: SBVR-8 activations (Sec. 4.3)


def act_quantize(x_fp16, l: int = ACT_BITS):
    """Codes q (int32 [I]) and per-group scales s (float32 [I/128]) of the
    online conversion (readings R11-R13 in the C source)."""
    x = np.ascontiguousarray(np.asarray(x_fp16, dtype=np.float16).view(np.uint16))
    I = x.size
    q = np.zeros(I, dtype=np.int32)
    s = np.zeros(I // GROUP, dtype=np.float32)
    if _lib().oracle_act_quantize(I, l, _ptr(x, C.c_uint16), _ptr(q, C.c_int32), _ptr(s, C.c_float)) != 0:
        raise ValueError("oracle_act_quantize rejected its arguments")
    return q, s


def act_planes(q, l: int = ACT_BITS) -> np.ndarray:
    """SBVR-l bitvectors [I][l] of codes q in Eq. 12's coefficient order."""
    q = np.ascontiguousarray(q, dtype=np.int32)
    planes = np.zeros((q.size, l), dtype=np.uint8)
    _lib().oracle_act_planes(q.size, l, _ptr(q, C.c_int32), _ptr(planes, C.c_uint8))
    return planes


def act_decode(planes, s, l: int = ACT_BITS) -> np.ndarray:
    """Decoded activations (binary64) from SBVR-l bitvectors and group scales."""
    planes = np.ascontiguousarray(planes, dtype=np.uint8)
    s = np.ascontiguousarray(s, dtype=np.float32)
    out = np.zeros(planes.shape[0])
    _lib().oracle_act_decode(planes.shape[0], l, _ptr(planes, C.c_uint8), _ptr(s, C.c_float),
                             _ptr(out, C.c_double))
    return out


# --------------------------------------------------------------------------
# Coefficient cache + per-group index (Sec. 4.4)
# --------------------------------------------------------------------------

def gather_coefficients(index, table) -> np.ndarray:
    """Per-(row, group, plane) coefficients of the coefficient-cache format
    (Sec. 4.4): the cache holds coefficient sets table[n][0..k-1] and the
    index names the set each group's k bitvectors use, so
    c[o][g][i] = table[index[o][g]][i].  uint16 (binary16 bits) [O][G][k]."""
    index = np.asarray(index)
    table = np.ascontiguousarray(table, dtype=np.uint16)
    if index.size and int(index.max()) >= table.shape[0]:
        raise ValueError("coefficient index past the end of the cache")
    return table[index.astype(np.int64)]


def coefficient_cache(coeffs):
    """(index uint16 [O][G], table uint16 [N][k]): the distinct coefficient sets
    of a per-group coefficient tensor, in order of first appearance (row-major
    over (o, g)), and each group's position in that list.  Lossless; raises if
    there are more than 65536 distinct sets (16-bit index)."""
    coeffs = np.ascontiguousarray(coeffs, dtype=np.uint16)
    O, G, K = coeffs.shape
    seen = {}
    rows = []
    index = np.empty(O * G, dtype=np.uint16)
    for n, c in enumerate(coeffs.reshape(O * G, K)):
        key = c.tobytes()
        pos = seen.get(key)
        if pos is None:
            pos = seen[key] = len(rows)
            if pos > 65535:
                raise ValueError("more than 65536 distinct coefficient sets")
            rows.append(c)
        index[n] = pos
    return index.reshape(O, G), np.array(rows, dtype=np.uint16).reshape(len(rows), K)


def sbvr_gemv_indexed(planes, index, table, x_fp16, rows=None, nthreads: int = 0) -> np.ndarray:
    """y = W_hat x in binary64 for the coefficient-cache format: the
    coefficients are gathered through the index, then the exact GEMV."""
    return sbvr_gemv(planes, gather_coefficients(index, table), x_fp16, rows=rows, nthreads=nthreads)


def sbvr_gemv_w4a8(planes: np.ndarray, coeffs: np.ndarray, x_fp16: np.ndarray, rows=None,
                   nthreads: int = 0) -> np.ndarray:
    """The W4A8 decode GEMV reference: y = W_hat x_hat in binary64, with x_hat
    the SBVR-8 decoded activations of x (conversion, bitvectors, decoding)."""
    planes = np.ascontiguousarray(planes, dtype=np.uint32)
    coeffs = np.ascontiguousarray(coeffs, dtype=np.uint16)
    O, G, K, _ = planes.shape
    I = G * GROUP
    q, s = act_quantize(x_fp16)
    x_hat = np.ascontiguousarray(act_decode(act_planes(q), s))
    if rows is None:
        rows_arr, n_rows = None, O
    else:
        rows_arr = np.ascontiguousarray(rows, dtype=np.int32)
        n_rows = rows_arr.size
    y = np.zeros(n_rows)
    nt = _lib().oracle_sbvr_gemv_f64(O, I, K, _ptr(planes, C.c_uint32), _ptr(coeffs, C.c_uint16),
                                     _ptr(x_hat, C.c_double), 1,
                                     _ptr(rows_arr, C.c_int) if rows_arr is not None else None,
                                     n_rows, int(nthreads), _ptr(y, C.c_double))
    if nt < 0:
        raise ValueError("oracle_sbvr_gemv_f64 rejected its arguments")
    return y


def rtn_sym_mse(D, bits: int) -> float:
    d = _f64(D)
    return _lib().oracle_rtn_sym_mse(_ptr(d, C.c_double), d.size, bits)


def rtn_asym_mse(D, bits: int) -> float:
    d = _f64(D)
    return _lib().oracle_rtn_asym_mse(_ptr(d, C.c_double), d.size, bits)
