"""C-ABI checks that need no GPU: the library loads, exports every entry point
declared in include/sbvr.h, and rejects bad arguments on the host before any
HIP call (so nothing is launched and no output is touched)."""
import ctypes as C
import os
import re

import pytest

import paper_2509_18172_amd as sb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "sbvr.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sbvr_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 9
    lib = C.CDLL(sb.library_path())
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(sb.EXPORTED) == names


def test_status_strings_and_version():
    assert sb.sbvr_status_string(0) == "SBVR_OK"
    for code, name in [(-1, "SBVR_E_INVALID_ARG"), (-2, "SBVR_E_UNSUPPORTED"), (-3, "SBVR_E_WORKSPACE"),
                       (-4, "SBVR_E_ALIGNMENT"), (-5, "SBVR_E_HIP")]:
        assert sb.sbvr_status_string(code) == name
    assert sb.sbvr_status_string(12345) == "SBVR_E_UNKNOWN"
    assert sb.sbvr_version() >= 100


@pytest.mark.parametrize("O,I,k", [(4096, 4096, 4), (1, 128, 1), (1001, 640, 3), (14336, 4096, 2)])
def test_size_queries(O, I, k):
    G = I // 128
    tr = {1: 16, 2: 8, 3: 4, 4: 4}[k]  # rows per tile: 16 matrix-core rows of (row, plane)
    tiles, gblocks = -(-O // tr), -(-G // 4)
    assert sb.sbvr_packed_plane_bytes(O, I, k) == tiles * gblocks * 4 * tr * k * 16
    assert sb.sbvr_packed_coeff_bytes(O, I, k) == tiles * gblocks * 4 * tr * k * 2
    # never smaller than the canonical tensors
    assert sb.sbvr_packed_plane_bytes(O, I, k) >= O * G * k * 16
    assert sb.sbvr_packed_coeff_bytes(O, I, k) >= O * G * k * 2
    assert sb.sbvr_workspace_bytes(O, I, k, 1) == 0


@pytest.mark.parametrize("O,I,k", [(0, 128, 4), (4, 100, 4), (4, 0, 4), (4, 128, 0), (-1, 128, 2)])
def test_size_queries_reject_bad_shapes(O, I, k):
    assert sb.sbvr_packed_plane_bytes(O, I, k) == 0
    assert sb.sbvr_packed_coeff_bytes(O, I, k) == 0


FAKE = 1 << 20  # 16-byte-aligned, never dereferenced: every call below fails validation


def gemv(O=16, I=256, k=4, p=FAKE, c=FAKE, x=FAKE, y=FAKE, ws=None, wsb=0):
    return sb.sbvr_gemv(O, I, k, p, c, x, y, ws, wsb, 0)


def test_gemv_validation():
    assert gemv(O=0) == sb.SBVR_E_INVALID_ARG
    assert gemv(I=130) == sb.SBVR_E_INVALID_ARG
    assert gemv(I=64) == sb.SBVR_E_INVALID_ARG
    assert gemv(k=0) == sb.SBVR_E_INVALID_ARG
    assert gemv(k=5) == sb.SBVR_E_UNSUPPORTED
    assert gemv(p=None) == sb.SBVR_E_INVALID_ARG
    assert gemv(c=None) == sb.SBVR_E_INVALID_ARG
    assert gemv(x=None) == sb.SBVR_E_INVALID_ARG
    assert gemv(y=None) == sb.SBVR_E_INVALID_ARG
    assert gemv(p=FAKE + 4) == sb.SBVR_E_ALIGNMENT
    assert gemv(c=FAKE + 8) == sb.SBVR_E_ALIGNMENT
    assert gemv(x=FAKE + 2) == sb.SBVR_E_ALIGNMENT
    assert gemv(y=FAKE + 1) == sb.SBVR_E_ALIGNMENT


def test_small_batch_validation():
    f = lambda B, **kw: sb.sbvr_gemm_small_batch(kw.get("O", 16), 256, kw.get("k", 4), FAKE, FAKE,
                                                 kw.get("X", FAKE), FAKE, B, None, 0, 0)
    assert f(0) == sb.SBVR_E_INVALID_ARG
    assert f(9) == sb.SBVR_E_INVALID_ARG
    assert f(-3) == sb.SBVR_E_INVALID_ARG
    assert f(4, X=None) == sb.SBVR_E_INVALID_ARG
    assert f(4, X=FAKE + 8) == sb.SBVR_E_ALIGNMENT
    assert f(4, k=7) == sb.SBVR_E_UNSUPPORTED


@pytest.mark.parametrize("name", ["sbvr_gemv_grouped", "sbvr_gemv_grouped_a8"])
def test_grouped_validation(name):
    """Every member is validated before anything is launched; the first
    failing member's status is returned."""
    f = getattr(sb, name)

    def g(n=2, O=(16, 32), I=256, k=4, P=(FAKE, FAKE), Cf=(FAKE, FAKE), X=(FAKE, FAKE), Y=(FAKE, FAKE)):
        return f(n, list(O), I, k, list(P), list(Cf), list(X), list(Y))
    assert g(n=0) == sb.SBVR_E_INVALID_ARG
    assert g(n=5, O=(16,) * 5, P=(FAKE,) * 5, Cf=(FAKE,) * 5, X=(FAKE,) * 5, Y=(FAKE,) * 5) == sb.SBVR_E_INVALID_ARG
    assert g(O=(16, 0)) == sb.SBVR_E_INVALID_ARG
    assert g(I=130) == sb.SBVR_E_INVALID_ARG
    assert g(k=5) == sb.SBVR_E_UNSUPPORTED
    assert g(P=(FAKE, 0)) == sb.SBVR_E_INVALID_ARG
    assert g(Y=(0, FAKE)) == sb.SBVR_E_INVALID_ARG
    assert g(X=(FAKE, FAKE + 2)) == sb.SBVR_E_ALIGNMENT
    assert g(Cf=(FAKE + 8, FAKE)) == sb.SBVR_E_ALIGNMENT
    # the first failing member decides: member 0 misaligned, member 1 k-independent shape error
    assert g(O=(16, 0), P=(FAKE + 4, FAKE)) == sb.SBVR_E_ALIGNMENT
    # host arrays shorter than n are refused by the binding
    assert f(3, [16, 16], 256, 4, [FAKE] * 3, [FAKE] * 3, [FAKE] * 3, [FAKE] * 3) == sb.SBVR_E_INVALID_ARG


def test_pack_validation():
    P = lambda **kw: sb.sbvr_pack(kw.get("O", 8), kw.get("I", 256), kw.get("k", 3), kw.get("pc", FAKE),
                                  kw.get("cc", FAKE), kw.get("pd", FAKE), kw.get("cd", FAKE), 0)
    U = lambda **kw: sb.sbvr_unpack(kw.get("O", 8), kw.get("I", 256), kw.get("k", 3), kw.get("pd", FAKE),
                                    kw.get("cd", FAKE), kw.get("pc", FAKE), kw.get("cc", FAKE), 0)
    for F in (P, U):
        assert F(O=0) == sb.SBVR_E_INVALID_ARG
        assert F(I=129) == sb.SBVR_E_INVALID_ARG
        assert F(k=6) == sb.SBVR_E_UNSUPPORTED
        assert F(pc=None) == sb.SBVR_E_INVALID_ARG
        assert F(cd=None) == sb.SBVR_E_INVALID_ARG
        assert F(pc=FAKE + 4) == sb.SBVR_E_ALIGNMENT
        assert F(cc=FAKE + 1) == sb.SBVR_E_ALIGNMENT
        assert F(pd=FAKE + 8) == sb.SBVR_E_ALIGNMENT


def test_algorithmic_bytes_formula():
    # 0.5625 B/weight at k=4 plus activations and outputs
    assert sb.algorithmic_bytes(4096, 4096, 4) == 9_453_568
    assert sb.algorithmic_bytes(14336, 4096, 4) == 33_067_008
    assert sb.algorithmic_bytes(28672, 8192, 4) == 132_194_304
    assert sb.algorithmic_bytes(4096, 4096, 4, B=8) == 9_568_256


def test_row_length_limit():
    """One tile's plane bytes over a whole row are capped at 2^26 (32-bit
    byte offsets inside a workgroup stay below the read-zero offset 2^30):
    a single row of 2^31 - 128 elements, or of 2^25 + 512 at k = 4, is
    refused before any pointer is touched; 2^25 at k = 4 and k = 2 (1 KiB
    plane blocks) is accepted by the size queries."""
    for O, I, k in [(1, (1 << 31) - 128, 4), (1, (1 << 25) + 512, 4), (3, (1 << 25) + 512, 2)]:
        assert sb.sbvr_packed_plane_bytes(O, I, k) == 0, (O, I, k)
        assert gemv(O=O, I=I, k=k) == sb.SBVR_E_UNSUPPORTED
        assert sb.sbvr_gemv_a8(O, I, k, FAKE, FAKE, FAKE, FAKE, None, 0, 0) == sb.SBVR_E_UNSUPPORTED
        assert sb.sbvr_decompress(O, I, k, FAKE, FAKE, FAKE, 0) == sb.SBVR_E_UNSUPPORTED
    assert sb.sbvr_packed_plane_bytes(1, 1 << 25, 4) == (1 << 26)
    assert sb.sbvr_packed_plane_bytes(2, 1 << 25, 2) == (1 << 26)  # one 8-row tile


def test_element_count_limit():
    """O * I must stay below 2^31 (the kernels' element offsets are 32-bit):
    the size queries return 0 and every entry point rejects the shape before
    touching any pointer."""
    big = [(32768, 65536), (65536, 32768), (16384, 131072)]
    for O, I in big:
        assert sb.sbvr_packed_plane_bytes(O, I, 4) == 0
        assert sb.sbvr_packed_index_bytes(O, I, 4) == 0
        assert gemv(O=O, I=I) == sb.SBVR_E_UNSUPPORTED
        assert sb.sbvr_gemv_a8(O, I, 4, FAKE, FAKE, FAKE, FAKE, None, 0, 0) == sb.SBVR_E_UNSUPPORTED
        assert sb.sbvr_encode(O, I, 4, FAKE, 8, 8, 16, 4, 1, FAKE, FAKE, None, 0) == sb.SBVR_E_UNSUPPORTED
    # the largest accepted shape
    assert sb.sbvr_packed_plane_bytes(16383, 131072, 4) == (16383 + 3) // 4 * 256 * 4 * 4 * 4 * 16


def test_new_entry_points_validation():
    a8 = lambda **kw: sb.sbvr_gemv_a8(kw.get("O", 16), kw.get("I", 256), kw.get("k", 4), kw.get("p", FAKE),
                                      FAKE, kw.get("x", FAKE), FAKE, None, 0, 0)
    assert a8(O=0) == sb.SBVR_E_INVALID_ARG
    assert a8(k=5) == sb.SBVR_E_UNSUPPORTED
    assert a8(p=None) == sb.SBVR_E_INVALID_ARG
    assert a8(x=FAKE + 2) == sb.SBVR_E_ALIGNMENT
    ix = lambda **kw: sb.sbvr_gemv_indexed(16, kw.get("I", 256), 4, kw.get("N", 10), FAKE, kw.get("i", FAKE),
                                           kw.get("t", FAKE), FAKE, FAKE, None, 0, 0)
    assert ix(N=0) == sb.SBVR_E_INVALID_ARG
    assert ix(N=65537) == sb.SBVR_E_INVALID_ARG
    assert ix(I=200) == sb.SBVR_E_INVALID_ARG
    assert ix(i=None) == sb.SBVR_E_INVALID_ARG
    assert ix(i=FAKE + 2) == sb.SBVR_E_ALIGNMENT
    assert ix(t=FAKE + 8) == sb.SBVR_E_ALIGNMENT
    assert sb.sbvr_gemv_indexed_a8(16, 256, 4, 0, FAKE, FAKE, FAKE, FAKE, FAKE, None, 0, 0) == sb.SBVR_E_INVALID_ARG
    assert sb.sbvr_decompress_indexed(16, 256, 4, 0, FAKE, FAKE, FAKE, FAKE, 0) == sb.SBVR_E_INVALID_ARG
    assert sb.sbvr_decompress_indexed(16, 256, 4, 5, FAKE, FAKE, FAKE, FAKE + 2, 0) == sb.SBVR_E_ALIGNMENT
    pk = lambda **kw: sb.sbvr_pack_indexed(8, 256, 3, kw.get("N", 4), FAKE, kw.get("ic", FAKE), FAKE, FAKE,
                                           kw.get("id", FAKE), FAKE, 0)
    assert pk(N=0) == sb.SBVR_E_INVALID_ARG
    assert pk(ic=FAKE + 1) == sb.SBVR_E_ALIGNMENT
    assert pk(id=FAKE + 2) == sb.SBVR_E_ALIGNMENT
    assert sb.sbvr_packed_table_bytes(3, 4) == 24 and sb.sbvr_packed_table_bytes(3, 9) == 0
    enc = lambda **kw: sb.sbvr_encode(4, 256, kw.get("k", 4), kw.get("W", FAKE), kw.get("n1", 8), 8, 16,
                                      kw.get("nb", 4), kw.get("norm", 1), FAKE, FAKE, kw.get("m", None), 0)
    assert enc(k=0) == sb.SBVR_E_INVALID_ARG
    assert enc(n1=0) == sb.SBVR_E_INVALID_ARG
    assert enc(nb=-1) == sb.SBVR_E_INVALID_ARG
    assert enc(norm=3) == sb.SBVR_E_INVALID_ARG
    assert enc(n1=1100) == sb.SBVR_E_UNSUPPORTED  # (1100 + 8) * 16 * 4 > 65536 entries
    assert enc(W=None) == sb.SBVR_E_INVALID_ARG
    assert enc(W=FAKE + 2) == sb.SBVR_E_ALIGNMENT
    assert enc(m=FAKE + 4) == sb.SBVR_E_ALIGNMENT
    encc = lambda **kw: sb.sbvr_encode_cached(4, 256, kw.get("k", 4), kw.get("W", FAKE), 8, 8, 16, 4, 1,
                                              kw.get("slots", 4), FAKE, FAKE, kw.get("m", None), None, 0)
    assert encc(slots=65) == sb.SBVR_E_INVALID_ARG
    assert encc(slots=-1) == sb.SBVR_E_INVALID_ARG
    assert encc(k=9) == sb.SBVR_E_UNSUPPORTED
    assert encc(W=None) == sb.SBVR_E_INVALID_ARG
    assert encc(W=FAKE + 2) == sb.SBVR_E_ALIGNMENT
    assert encc(m=FAKE + 4) == sb.SBVR_E_ALIGNMENT


def test_read_probe_loads_and_rejects_bad_arguments():
    """The benchmark's streaming-read helper: it loads, and rejects a null
    pointer or a size that is not a multiple of 16 before any launch."""
    from paper_2509_18172_amd.build import probe_path
    probe = C.CDLL(probe_path())
    fn = probe.sbvr_probe_stream_read
    fn.argtypes = [C.c_void_p, C.c_size_t, C.c_int, C.c_void_p, C.c_void_p]
    fn.restype = C.c_int
    buf = (C.c_ubyte * 64)()
    sink = (C.c_uint * 4)()
    assert fn(None, 64, 0, C.addressof(sink), None) == -1
    assert fn(C.addressof(buf), 0, 0, C.addressof(sink), None) == -1
    assert fn(C.addressof(buf), 24, 1, C.addressof(sink), None) == -1
    assert fn(C.addressof(buf), 64, 0, None, None) == -1
