"""SBVR GEMV on MI355X: Python binding of the C ABI in include/sbvr.h.

Argument marshalling only: every step of the computation runs in the HIP
kernels of ``_lib/libsbvr.so``.  PyTorch supplies device memory and streams.
If the library is not built, importing this package raises -- there is no
fallback path.

Functions with the C names take raw integers (device pointers, stream
handles) and return the C status code.  The tensor helpers below check
shapes, allocate outputs with torch and raise ``SBVRError`` on a non-zero
status.
"""
from __future__ import annotations

import ctypes as C
import os

from .build import library_path

GROUP = 128

SBVR_OK = 0
SBVR_E_INVALID_ARG = -1
SBVR_E_UNSUPPORTED = -2
SBVR_E_WORKSPACE = -3
SBVR_E_ALIGNMENT = -4
SBVR_E_HIP = -5

EXPORTED = (
    "sbvr_status_string", "sbvr_version", "sbvr_packed_plane_bytes", "sbvr_packed_coeff_bytes",
    "sbvr_workspace_bytes", "sbvr_pack", "sbvr_unpack", "sbvr_gemv", "sbvr_gemm_small_batch",
    "sbvr_decompress", "sbvr_gemv_a8", "sbvr_packed_index_bytes", "sbvr_packed_table_bytes",
    "sbvr_pack_indexed", "sbvr_unpack_indexed", "sbvr_gemv_indexed", "sbvr_gemv_indexed_a8", "sbvr_encode",
    "sbvr_decompress_indexed", "sbvr_gemm_prefill", "sbvr_gemv_grouped", "sbvr_gemv_grouped_a8",
    "sbvr_encode_cached",
)


class SBVRError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {sbvr_status_string(status)} ({status})")
        self.status = status


def _load():
    # PyTorch ships its own HIP runtime (same SONAME as ROCm's).  Loading torch
    # first makes libsbvr.so bind to that runtime, so device pointers and
    # stream handles from torch are valid in the library; loading ROCm's copy
    # first would put two HIP runtimes in the process.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    path = library_path()
    if not os.path.exists(path):
        raise ImportError(
            f"SBVR HIP library not built ({path}); run `python -c 'import __graft_entry__ as g; g.build()'`")
    lib = C.CDLL(path)
    vp, sz, i32 = C.c_void_p, C.c_size_t, C.c_int
    sig = {
        "sbvr_status_string": (C.c_char_p, [i32]),
        "sbvr_version": (i32, []),
        "sbvr_packed_plane_bytes": (sz, [i32, i32, i32]),
        "sbvr_packed_coeff_bytes": (sz, [i32, i32, i32]),
        "sbvr_workspace_bytes": (sz, [i32, i32, i32, i32]),
        "sbvr_pack": (i32, [i32, i32, i32, vp, vp, vp, vp, vp]),
        "sbvr_unpack": (i32, [i32, i32, i32, vp, vp, vp, vp, vp]),
        "sbvr_gemv": (i32, [i32, i32, i32, vp, vp, vp, vp, vp, sz, vp]),
        "sbvr_gemm_small_batch": (i32, [i32, i32, i32, vp, vp, vp, vp, i32, vp, sz, vp]),
        "sbvr_decompress": (i32, [i32, i32, i32, vp, vp, vp, vp]),
        "sbvr_gemv_a8": (i32, [i32, i32, i32, vp, vp, vp, vp, vp, sz, vp]),
        "sbvr_packed_index_bytes": (sz, [i32, i32, i32]),
        "sbvr_packed_table_bytes": (sz, [i32, i32]),
        "sbvr_pack_indexed": (i32, [i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp]),
        "sbvr_unpack_indexed": (i32, [i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp]),
        "sbvr_gemv_indexed": (i32, [i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, sz, vp]),
        "sbvr_gemv_indexed_a8": (i32, [i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, sz, vp]),
        "sbvr_encode": (i32, [i32, i32, i32, vp, i32, i32, i32, i32, i32, vp, vp, vp, vp]),
        "sbvr_encode_cached": (i32, [i32, i32, i32, vp, i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp]),
        "sbvr_decompress_indexed": (i32, [i32, i32, i32, i32, vp, vp, vp, vp, vp]),
        "sbvr_gemm_prefill": (i32, [i32, i32, i32, vp, vp, vp, vp, i32, vp]),
        "sbvr_gemv_grouped": (i32, [i32, vp, i32, i32, vp, vp, vp, vp, vp, sz, vp]),
        "sbvr_gemv_grouped_a8": (i32, [i32, vp, i32, i32, vp, vp, vp, vp, vp, sz, vp]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


_lib = _load()


# --------------------------------------------------------------------------
# C ABI, same names (raw pointers / stream handles as Python ints)
# --------------------------------------------------------------------------

def sbvr_status_string(status: int) -> str:
    return _lib.sbvr_status_string(int(status)).decode()


def sbvr_version() -> int:
    return _lib.sbvr_version()


def sbvr_packed_plane_bytes(O: int, I: int, k: int) -> int:
    return _lib.sbvr_packed_plane_bytes(O, I, k)


def sbvr_packed_coeff_bytes(O: int, I: int, k: int) -> int:
    return _lib.sbvr_packed_coeff_bytes(O, I, k)


def sbvr_workspace_bytes(O: int, I: int, k: int, B: int = 1) -> int:
    return _lib.sbvr_workspace_bytes(O, I, k, B)


def sbvr_pack(O, I, k, planes_canon, coeffs_canon, planes_dev, coeffs_dev, stream=0) -> int:
    return _lib.sbvr_pack(O, I, k, planes_canon, coeffs_canon, planes_dev, coeffs_dev, stream)


def sbvr_unpack(O, I, k, planes_dev, coeffs_dev, planes_canon, coeffs_canon, stream=0) -> int:
    return _lib.sbvr_unpack(O, I, k, planes_dev, coeffs_dev, planes_canon, coeffs_canon, stream)


def sbvr_gemv(O, I, k, planes_dev, coeffs_dev, x, y, workspace=None, ws_bytes=0, stream=0) -> int:
    return _lib.sbvr_gemv(O, I, k, planes_dev, coeffs_dev, x, y, workspace, ws_bytes, stream)


def sbvr_gemm_small_batch(O, I, k, planes_dev, coeffs_dev, X, Y, B, workspace=None, ws_bytes=0,
                          stream=0) -> int:
    return _lib.sbvr_gemm_small_batch(O, I, k, planes_dev, coeffs_dev, X, Y, B, workspace, ws_bytes,
                                      stream)


def sbvr_gemv_a8(O, I, k, planes_dev, coeffs_dev, x, y, workspace=None, ws_bytes=0, stream=0) -> int:
    return _lib.sbvr_gemv_a8(O, I, k, planes_dev, coeffs_dev, x, y, workspace, ws_bytes, stream)


GEMV_GROUP_MAX = 4
ENCODE_CACHE_MAX = 64


def _grouped(fn, n, O, I, k, planes_dev, coeffs_dev, x, y, workspace, ws_bytes, stream) -> int:
    seq = (O, planes_dev, coeffs_dev, x, y)
    if any(len(v) < n for v in seq):
        return SBVR_E_INVALID_ARG
    m = max(n, 1)
    arr_O = (C.c_int * m)(*[int(v) for v in list(O)[:n]])
    ptrs = [(C.c_void_p * m)(*[int(p) for p in list(v)[:n]]) for v in seq[1:]]
    return fn(n, arr_O, I, k, *ptrs, workspace, ws_bytes, stream)


def sbvr_gemv_grouped(n, O, I, k, planes_dev, coeffs_dev, x, y, workspace=None, ws_bytes=0, stream=0) -> int:
    """O, planes_dev, coeffs_dev, x, y: sequences of n ints (out_features and
    device pointers), marshalled into the host arrays the C call reads."""
    return _grouped(_lib.sbvr_gemv_grouped, n, O, I, k, planes_dev, coeffs_dev, x, y, workspace, ws_bytes, stream)


def sbvr_gemv_grouped_a8(n, O, I, k, planes_dev, coeffs_dev, x, y, workspace=None, ws_bytes=0, stream=0) -> int:
    """As sbvr_gemv_grouped, with the W4A8 conversion of sbvr_gemv_a8."""
    return _grouped(_lib.sbvr_gemv_grouped_a8, n, O, I, k, planes_dev, coeffs_dev, x, y, workspace, ws_bytes,
                    stream)


def sbvr_packed_index_bytes(O: int, I: int, k: int) -> int:
    return _lib.sbvr_packed_index_bytes(O, I, k)


def sbvr_packed_table_bytes(n_sets: int, k: int) -> int:
    return _lib.sbvr_packed_table_bytes(n_sets, k)


def sbvr_pack_indexed(O, I, k, n_sets, planes_canon, index_canon, table_canon, planes_dev, index_dev,
                      table_dev, stream=0) -> int:
    return _lib.sbvr_pack_indexed(O, I, k, n_sets, planes_canon, index_canon, table_canon, planes_dev,
                                  index_dev, table_dev, stream)


def sbvr_unpack_indexed(O, I, k, n_sets, planes_dev, index_dev, table_dev, planes_canon, index_canon,
                        table_canon, stream=0) -> int:
    return _lib.sbvr_unpack_indexed(O, I, k, n_sets, planes_dev, index_dev, table_dev, planes_canon,
                                    index_canon, table_canon, stream)


def sbvr_gemv_indexed(O, I, k, n_sets, planes_dev, index_dev, table_dev, x, y, workspace=None, ws_bytes=0,
                      stream=0) -> int:
    return _lib.sbvr_gemv_indexed(O, I, k, n_sets, planes_dev, index_dev, table_dev, x, y, workspace,
                                  ws_bytes, stream)


def sbvr_gemv_indexed_a8(O, I, k, n_sets, planes_dev, index_dev, table_dev, x, y, workspace=None,
                         ws_bytes=0, stream=0) -> int:
    return _lib.sbvr_gemv_indexed_a8(O, I, k, n_sets, planes_dev, index_dev, table_dev, x, y, workspace,
                                     ws_bytes, stream)


def sbvr_encode(O, I, k, W, n_ratio1, n_ratio2, n_scale, n_bias, normalise, planes_canon, coeffs_canon,
                mse=None, stream=0) -> int:
    return _lib.sbvr_encode(O, I, k, W, n_ratio1, n_ratio2, n_scale, n_bias, normalise, planes_canon,
                            coeffs_canon, mse, stream)


def sbvr_encode_cached(O, I, k, W, n_ratio1, n_ratio2, n_scale, n_bias, normalise, cache_slots, planes_canon,
                       coeffs_canon, mse=None, hits=None, stream=0) -> int:
    return _lib.sbvr_encode_cached(O, I, k, W, n_ratio1, n_ratio2, n_scale, n_bias, normalise, cache_slots,
                                   planes_canon, coeffs_canon, mse, hits, stream)


def sbvr_decompress(O, I, k, planes_dev, coeffs_dev, W, stream=0) -> int:
    return _lib.sbvr_decompress(O, I, k, planes_dev, coeffs_dev, W, stream)


def sbvr_decompress_indexed(O, I, k, n_sets, planes_dev, index_dev, table_dev, W, stream=0) -> int:
    return _lib.sbvr_decompress_indexed(O, I, k, n_sets, planes_dev, index_dev, table_dev, W, stream)


def sbvr_gemm_prefill(O, I, k, planes_dev, coeffs_dev, X, Y, T, stream=0) -> int:
    return _lib.sbvr_gemm_prefill(O, I, k, planes_dev, coeffs_dev, X, Y, T, stream)


# --------------------------------------------------------------------------
# torch tensor helpers
# --------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _stream(stream=None) -> int:
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return int(s.cuda_stream)


def _check(status: int, what: str):
    if status != SBVR_OK:
        raise SBVRError(status, what)


class PackedWeight:
    """An O x I SBVR matrix with k planes, resident in device memory in the
    library's device format."""

    def __init__(self, O: int, I: int, k: int, planes_dev, coeffs_dev):
        self.O, self.I, self.k = O, I, k
        self.planes = planes_dev
        self.coeffs = coeffs_dev

    @property
    def nbytes(self) -> int:
        return self.planes.numel() + self.coeffs.numel()

    @staticmethod
    def alloc(O: int, I: int, k: int, device="cuda"):
        torch = _torch()
        pb, cb = sbvr_packed_plane_bytes(O, I, k), sbvr_packed_coeff_bytes(O, I, k)
        if pb == 0 or cb == 0:
            raise SBVRError(SBVR_E_INVALID_ARG, f"shape {O}x{I} k={k}")
        return PackedWeight(O, I, k, torch.empty(pb, dtype=torch.uint8, device=device),
                            torch.empty(cb, dtype=torch.uint8, device=device))


def _out(out, shape, x):
    """The output tensor: a new fp16 tensor on x's device, or the caller's,
    which must be fp16, contiguous, of exactly `shape` and on x's device (the
    kernels write every element of it)."""
    torch = _torch()
    if out is None:
        return torch.empty(shape, dtype=torch.float16, device=x.device)
    assert out.dtype == torch.float16 and out.is_contiguous() and tuple(out.shape) == tuple(shape), \
        f"out must be a contiguous fp16 tensor of shape {tuple(shape)}"
    assert out.device == x.device, "out must be on the activations' device"
    return out


def _check_input(W, x, shape):
    torch = _torch()
    assert x.dtype == torch.float16 and x.is_contiguous() and tuple(x.shape) == tuple(shape), \
        f"activations must be a contiguous fp16 tensor of shape {tuple(shape)}"
    assert x.is_cuda and x.device == W.planes.device, "activations must be on the weights' device"


def pack(planes_canon, coeffs_canon, stream=None) -> PackedWeight:
    """Repack canonical device tensors (int32/uint32 [O][G][k][4], int16/uint16
    [O][G][k]) into a PackedWeight."""
    O, G, k, four = planes_canon.shape
    assert four == 4 and tuple(coeffs_canon.shape) == (O, G, k)
    assert planes_canon.is_contiguous() and coeffs_canon.is_contiguous()
    assert planes_canon.element_size() == 4 and coeffs_canon.element_size() == 2
    assert planes_canon.is_cuda and coeffs_canon.device == planes_canon.device, "canonical tensors must be on the GPU"
    W = PackedWeight.alloc(O, G * GROUP, k, device=planes_canon.device)
    _check(sbvr_pack(O, G * GROUP, k, planes_canon.data_ptr(), coeffs_canon.data_ptr(),
                     W.planes.data_ptr(), W.coeffs.data_ptr(), _stream(stream)), "sbvr_pack")
    return W


def unpack(W: PackedWeight, stream=None):
    """Canonical (planes int32 [O][G][k][4], coeffs int16 [O][G][k]) device tensors."""
    torch = _torch()
    G = W.I // GROUP
    planes = torch.empty((W.O, G, W.k, 4), dtype=torch.int32, device=W.planes.device)
    coeffs = torch.empty((W.O, G, W.k), dtype=torch.int16, device=W.planes.device)
    _check(sbvr_unpack(W.O, W.I, W.k, W.planes.data_ptr(), W.coeffs.data_ptr(), planes.data_ptr(),
                       coeffs.data_ptr(), _stream(stream)), "sbvr_unpack")
    return planes, coeffs


def gemv(W: PackedWeight, x, out=None, stream=None):
    """y = SBVR(W) x for x fp16 [I]; returns fp16 [O]."""
    _check_input(W, x, (W.I,))
    y = _out(out, (W.O,), x)
    _check(sbvr_gemv(W.O, W.I, W.k, W.planes.data_ptr(), W.coeffs.data_ptr(), x.data_ptr(),
                     y.data_ptr(), None, 0, _stream(stream)), "sbvr_gemv")
    return y


def gemv_grouped(Ws, xs, outs=None, stream=None, a8=False):
    """y_i = SBVR(W_i) x_i for up to GEMV_GROUP_MAX matrices with the same I
    and k, as one kernel launch (a8: each as gemv_a8); returns the list of
    fp16 [O_i] outputs."""
    Ws, xs = list(Ws), list(xs)
    assert 1 <= len(Ws) <= GEMV_GROUP_MAX and len(xs) == len(Ws)
    I, k = Ws[0].I, Ws[0].k
    assert all(W.I == I and W.k == k for W in Ws), "members must share I and k"
    for W, x in zip(Ws, xs):
        _check_input(W, x, (W.I,))
    ys = [_out(None if outs is None else outs[i], (W.O,), xs[i]) for i, W in enumerate(Ws)]
    fn, name = (sbvr_gemv_grouped_a8, "sbvr_gemv_grouped_a8") if a8 else (sbvr_gemv_grouped, "sbvr_gemv_grouped")
    _check(fn(len(Ws), [W.O for W in Ws], I, k, [W.planes.data_ptr() for W in Ws], [W.coeffs.data_ptr() for W in Ws],
              [x.data_ptr() for x in xs], [y.data_ptr() for y in ys], None, 0, _stream(stream)), name)
    return ys


def gemm_small_batch(W: PackedWeight, X, out=None, stream=None):
    """Y = X SBVR(W)^T for X fp16 [B][I], 1 <= B <= 8; returns fp16 [B][O]."""
    assert X.dim() == 2
    B = X.shape[0]
    _check_input(W, X, (B, W.I))
    Y = _out(out, (B, W.O), X)
    _check(sbvr_gemm_small_batch(W.O, W.I, W.k, W.planes.data_ptr(), W.coeffs.data_ptr(),
                                 X.data_ptr(), Y.data_ptr(), B, None, 0, _stream(stream)),
           "sbvr_gemm_small_batch")
    return Y


def gemv_a8(W: PackedWeight, x, out=None, stream=None):
    """The W4A8 decode GEMV: x fp16 [I] converted online to SBVR-8 activations
    (per-128-group scale, 8-bit two's-complement codes); returns fp16 [O]."""
    _check_input(W, x, (W.I,))
    y = _out(out, (W.O,), x)
    _check(sbvr_gemv_a8(W.O, W.I, W.k, W.planes.data_ptr(), W.coeffs.data_ptr(), x.data_ptr(),
                        y.data_ptr(), None, 0, _stream(stream)), "sbvr_gemv_a8")
    return y


class IndexedWeight:
    """An O x I SBVR matrix in the coefficient-cache format (planes, index
    blocks, table of n_sets coefficient sets), resident in device memory in
    the library's device format."""

    def __init__(self, O: int, I: int, k: int, n_sets: int, planes, index, table):
        self.O, self.I, self.k, self.n_sets = O, I, k, n_sets
        self.planes, self.index, self.table = planes, index, table

    @property
    def nbytes(self) -> int:
        return self.planes.numel() + self.index.numel() + self.table.numel()


def pack_indexed(planes_canon, index_canon, table_canon, stream=None) -> IndexedWeight:
    """Repack canonical device tensors (int32/uint32 [O][G][k][4], int16/uint16
    [O][G] index, int16/uint16 [n_sets][k] table) into an IndexedWeight."""
    torch = _torch()
    O, G, k, four = planes_canon.shape
    n_sets = table_canon.shape[0]
    assert four == 4 and tuple(index_canon.shape) == (O, G) and tuple(table_canon.shape) == (n_sets, k)
    for t in (planes_canon, index_canon, table_canon):
        assert t.is_contiguous() and t.is_cuda and t.device == planes_canon.device, \
            "canonical tensors must be contiguous and on one GPU"
    assert planes_canon.element_size() == 4 and index_canon.element_size() == 2 and table_canon.element_size() == 2
    I = G * GROUP
    pb, ib, tb = sbvr_packed_plane_bytes(O, I, k), sbvr_packed_index_bytes(O, I, k), sbvr_packed_table_bytes(n_sets, k)
    if pb == 0 or ib == 0 or tb == 0:
        raise SBVRError(SBVR_E_INVALID_ARG, f"shape {O}x{I} k={k} n_sets={n_sets}")
    dev = planes_canon.device
    W = IndexedWeight(O, I, k, n_sets, torch.empty(pb, dtype=torch.uint8, device=dev),
                      torch.empty(ib, dtype=torch.uint8, device=dev), torch.empty(tb, dtype=torch.uint8, device=dev))
    _check(sbvr_pack_indexed(O, I, k, n_sets, planes_canon.data_ptr(), index_canon.data_ptr(), table_canon.data_ptr(),
                             W.planes.data_ptr(), W.index.data_ptr(), W.table.data_ptr(), _stream(stream)),
           "sbvr_pack_indexed")
    return W


def unpack_indexed(W: IndexedWeight, stream=None):
    """Canonical (planes int32 [O][G][k][4], index int16 [O][G], table int16
    [n_sets][k]) device tensors."""
    torch = _torch()
    G = W.I // GROUP
    dev = W.planes.device
    planes = torch.empty((W.O, G, W.k, 4), dtype=torch.int32, device=dev)
    index = torch.empty((W.O, G), dtype=torch.int16, device=dev)
    table = torch.empty((W.n_sets, W.k), dtype=torch.int16, device=dev)
    _check(sbvr_unpack_indexed(W.O, W.I, W.k, W.n_sets, W.planes.data_ptr(), W.index.data_ptr(),
                               W.table.data_ptr(), planes.data_ptr(), index.data_ptr(), table.data_ptr(),
                               _stream(stream)), "sbvr_unpack_indexed")
    return planes, index, table


def gemv_indexed(W: IndexedWeight, x, out=None, a8: bool = False, stream=None):
    """y = SBVR(W) x on the coefficient-cache format, x fp16 [I]; with
    a8=True the activations are converted online to SBVR-8 (W4A8)."""
    _check_input(W, x, (W.I,))
    y = _out(out, (W.O,), x)
    fn, name = (sbvr_gemv_indexed_a8, "sbvr_gemv_indexed_a8") if a8 else (sbvr_gemv_indexed, "sbvr_gemv_indexed")
    _check(fn(W.O, W.I, W.k, W.n_sets, W.planes.data_ptr(), W.index.data_ptr(), W.table.data_ptr(),
              x.data_ptr(), y.data_ptr(), None, 0, _stream(stream)), name)
    return y


def encode(W, k: int, n_ratio1: int = 8, n_ratio2: int = 8, n_scale: int = 16, n_bias: int = 4,
           normalise: bool = True, want_mse: bool = False, stream=None):
    """Encode a float32 [O][I] device matrix into canonical SBVR on the GPU:
    returns (planes int32 [O][G][k][4], coeffs int16 [O][G][k][, mse float64
    [O][G]]) device tensors.  Defaults: the 1024-entry search grid."""
    torch = _torch()
    assert W.dtype == torch.float32 and W.is_contiguous() and W.dim() == 2 and W.is_cuda
    O, I = W.shape
    G = I // GROUP
    planes = torch.empty((O, G, k, 4), dtype=torch.int32, device=W.device)
    coeffs = torch.empty((O, G, k), dtype=torch.int16, device=W.device)
    mse = torch.empty((O, G), dtype=torch.float64, device=W.device) if want_mse else None
    _check(sbvr_encode(O, I, k, W.data_ptr(), n_ratio1, n_ratio2, n_scale, n_bias, int(normalise), planes.data_ptr(),
                       coeffs.data_ptr(), mse.data_ptr() if want_mse else None, _stream(stream)), "sbvr_encode")
    return (planes, coeffs, mse) if want_mse else (planes, coeffs)


def encode_cached(W, k: int, cache_slots: int = ENCODE_CACHE_MAX, n_ratio1: int = 8, n_ratio2: int = 8,
                  n_scale: int = 16, n_bias: int = 4, normalise: bool = True, stream=None):
    """encode() with the encoder cache of Sec. 4.2 (per row, the sets of its
    last cache_slots searched groups tried first): returns (planes, coeffs,
    mse float64 [O][G], hits uint8 [O][G]) device tensors."""
    torch = _torch()
    assert W.dtype == torch.float32 and W.is_contiguous() and W.dim() == 2 and W.is_cuda
    O, I = W.shape
    G = I // GROUP
    planes = torch.empty((O, G, k, 4), dtype=torch.int32, device=W.device)
    coeffs = torch.empty((O, G, k), dtype=torch.int16, device=W.device)
    mse = torch.empty((O, G), dtype=torch.float64, device=W.device)
    hits = torch.empty((O, G), dtype=torch.uint8, device=W.device)
    _check(sbvr_encode_cached(O, I, k, W.data_ptr(), n_ratio1, n_ratio2, n_scale, n_bias, int(normalise),
                              int(cache_slots), planes.data_ptr(), coeffs.data_ptr(), mse.data_ptr(),
                              hits.data_ptr(), _stream(stream)), "sbvr_encode_cached")
    return planes, coeffs, mse, hits


def gemm_prefill(W: PackedWeight, X, out=None, stream=None):
    """Y = X fp16(W_hat)^T for a prompt X fp16 [T][I] (prefill GEMM on the
    SBVR weights, decoded on the fly); returns fp16 [T][O]."""
    assert X.dim() == 2
    T = X.shape[0]
    _check_input(W, X, (T, W.I))
    Y = _out(out, (T, W.O), X)
    _check(sbvr_gemm_prefill(W.O, W.I, W.k, W.planes.data_ptr(), W.coeffs.data_ptr(), X.data_ptr(), Y.data_ptr(), T,
                             _stream(stream)), "sbvr_gemm_prefill")
    return Y


def decompress(W, out=None, stream=None):
    """The decoded matrix as fp16 [O][I] (prefill path), for a PackedWeight or
    an IndexedWeight."""
    torch = _torch()
    M = torch.empty((W.O, W.I), dtype=torch.float16, device=W.planes.device) if out is None else out
    assert M.dtype == torch.float16 and M.is_contiguous() and tuple(M.shape) == (W.O, W.I)
    assert M.device == W.planes.device, "out must be on the weights' device"
    if isinstance(W, IndexedWeight):
        _check(sbvr_decompress_indexed(W.O, W.I, W.k, W.n_sets, W.planes.data_ptr(), W.index.data_ptr(),
                                       W.table.data_ptr(), M.data_ptr(), _stream(stream)), "sbvr_decompress_indexed")
    else:
        _check(sbvr_decompress(W.O, W.I, W.k, W.planes.data_ptr(), W.coeffs.data_ptr(), M.data_ptr(),
                               _stream(stream)), "sbvr_decompress")
    return M


def algorithmic_bytes_indexed(O: int, I: int, k: int, n_sets: int) -> int:
    """Bytes per call in the coefficient-cache format: planes k*O*I/8, one
    2-byte index per (row, group) 2*O*I/128, the coefficient sets 2*k*n_sets,
    activations 2*I and outputs 2*O."""
    return k * O * I // 8 + 2 * O * I // GROUP + 2 * k * n_sets + 2 * I + 2 * O


def algorithmic_bytes(O: int, I: int, k: int, B: int = 1) -> int:
    """Bytes the method must move per call: planes k*O*I/8, fp16 coefficients
    2*k*O*I/128, activations 2*I*B and outputs 2*O*B."""
    return k * O * I // 8 + 2 * k * O * I // GROUP + 2 * I * B + 2 * O * B
