"""Property tests of the HIP path against the oracle over random shapes.

Shapes are drawn with Hypothesis (derandomised, so every run draws the same
examples, and with no example database): O in [1, 3000], I = 128 * [1, 64],
k in 1..4, B in 1..8.  Each example checks, on the same seeded SBVR tensors
(uniform planes, Gaussian binary16 coefficients) and N(0, 1) binary16
activations:
  - sbvr_gemv (B = 1) or sbvr_gemm_small_batch (B > 1) against the oracle's
    binary64 GEMV of the exactly decoded matrix, per vector, within the gate
    max|y - y_ref| / max|y_ref| <= 1e-3;
  - sbvr_gemv_a8 against the oracle's W4A8 result (SBVR-8 activations);
  - sbvr_decompress bit for bit against rounding the oracle's exact decoding;
  - the coefficient-cache format (a random table and index) against the
    oracle's gathered-coefficient GEMV;
  - grouped launches (sbvr_gemv_grouped / _a8) of 1..4 members with random
    row counts and one shared I and k: every member bit for bit its own
    sbvr_gemv / sbvr_gemv_a8 call, and within the gate of the oracle.
The launch shape (one-shot or streaming kernel, tiles and gblocks per
workgroup, ring depth) follows from O and I, so the draws cover ragged row
tiles, ragged gblocks and every kernel variant of these sizes.
"""
import os

import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
hypothesis = pytest.importorskip("hypothesis")
from hypothesis import HealthCheck, given, settings  # noqa: E402
from hypothesis import strategies as st  # noqa: E402

pytestmark = pytest.mark.gpu

TOL = 1e-3
# 40 draws per test by default; SBVR_PROPERTY_EXAMPLES raises it for a wider sweep
EXAMPLES = int(os.environ.get("SBVR_PROPERTY_EXAMPLES", "40"))
SETTINGS = settings(max_examples=EXAMPLES, deadline=None, derandomize=True, database=None,
                    suppress_health_check=[HealthCheck.function_scoped_fixture, HealthCheck.too_slow])


@pytest.fixture(scope="module")
def sb():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2509_18172_amd as m
    return m


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def rel_err(y, y_ref):
    """The gate's measure for one vector: max|y - y_ref| / max|y_ref| (an
    all-zero reference asks for an all-zero result)."""
    y = np.asarray(y, dtype=np.float64)
    den = np.abs(y_ref).max()
    return float(np.abs(y - y_ref).max() / den) if den > 0 else float(np.abs(y).max())


def decoded(planes, coeffs):
    with np.errstate(over="ignore"):
        return oracle.decompress(planes, coeffs)


shapes = st.tuples(st.integers(1, 3000), st.integers(1, 64).map(lambda g: 128 * g), st.integers(1, 4))


@SETTINGS
@given(shape=shapes, B=st.integers(1, 8))
def test_random_shapes_gemv_and_small_batch(sb, shape, B):
    O, I, k = shape
    seed = O * 131 + I + 7 * k + B
    print(f"shape {O}x{I} k={k} B={B}", flush=True)
    planes, coeffs = synth.random_sbvr(O, I, k, seed=seed)
    W = sb.pack(dev(planes.view(np.int32)), dev(coeffs.view(np.int16)))
    X = synth.activations(I, seed=seed + synth.X_SEED_OFFSET, batch=B)
    if B == 1:
        Y = sb.gemv(W, dev(X[0]))[None]
    else:
        Y = sb.gemm_small_batch(W, dev(X))
    torch.cuda.synchronize()
    Y = Y.cpu().numpy().astype(np.float64)
    Y_ref = np.atleast_2d(oracle.sbvr_gemv(planes, coeffs, X))
    for b in range(B):
        assert rel_err(Y[b], Y_ref[b]) <= TOL, (O, I, k, B, b, rel_err(Y[b], Y_ref[b]))


@SETTINGS
@given(shape=shapes)
def test_random_shapes_w4a8_and_decompress(sb, shape):
    O, I, k = shape
    seed = O * 17 + I + k
    print(f"shape {O}x{I} k={k}", flush=True)
    planes, coeffs = synth.random_sbvr(O, I, k, seed=seed)
    W = sb.pack(dev(planes.view(np.int32)), dev(coeffs.view(np.int16)))
    x = synth.activations(I, seed=seed + synth.X_SEED_OFFSET)
    y = sb.gemv_a8(W, dev(x))
    M = sb.decompress(W)
    torch.cuda.synchronize()
    W_hat = decoded(planes, coeffs)
    assert rel_err(y.cpu().numpy(), oracle.sbvr_gemv_w4a8(planes, coeffs, x)) <= TOL
    with np.errstate(over="ignore"):
        want = W_hat.astype(np.float16).view(np.uint16)
    assert np.array_equal(M.cpu().numpy().view(np.uint16), want)


@SETTINGS
@given(shape=shapes, sets_per_ten=st.integers(1, 10))
def test_random_shapes_coefficient_cache(sb, shape, sets_per_ten):
    O, I, k = shape
    G = I // 128
    n_sets = max(1, min(65536, O * G * sets_per_ten // 10))
    seed = O * 29 + I + k + sets_per_ten
    print(f"shape {O}x{I} k={k} sets={n_sets}", flush=True)
    planes, index, table = synth.random_indexed_sbvr(O, I, k, n_sets, seed=seed)
    Wi = sb.pack_indexed(dev(planes.view(np.int32)), dev(index.view(np.int16)), dev(table.view(np.int16)))
    x = synth.activations(I, seed=seed + synth.X_SEED_OFFSET)
    y = sb.gemv_indexed(Wi, dev(x))
    torch.cuda.synchronize()
    assert rel_err(y.cpu().numpy(), oracle.sbvr_gemv_indexed(planes, index, table, x)) <= TOL


@SETTINGS
@given(rows=st.lists(st.integers(1, 3000), min_size=1, max_size=4), g=st.integers(1, 64), k=st.integers(1, 4),
       a8=st.booleans())
def test_random_grouped_launches(sb, rows, g, k, a8):
    I = 128 * g
    seed = sum(rows) * 7 + I + k + int(a8)
    print(f"grouped {rows} x {I} k={k} a8={a8}", flush=True)
    mats = [synth.random_sbvr(O, I, k, seed=seed + 11 * i) for i, O in enumerate(rows)]
    Ws = [sb.pack(dev(p.view(np.int32)), dev(c.view(np.int16))) for p, c in mats]
    xs = [synth.activations(I, seed=seed + i + synth.X_SEED_OFFSET) for i in range(len(rows))]
    xd = [dev(x) for x in xs]
    ys = sb.gemv_grouped(Ws, xd, a8=a8)
    sep = [(sb.gemv_a8 if a8 else sb.gemv)(W, x) for W, x in zip(Ws, xd)]
    torch.cuda.synchronize()
    ref = oracle.sbvr_gemv_w4a8 if a8 else oracle.sbvr_gemv
    for i, (planes, coeffs) in enumerate(mats):
        got = ys[i].cpu().numpy()
        assert np.array_equal(got.view(np.uint16), sep[i].cpu().numpy().view(np.uint16)), (rows, I, k, a8, i)
        assert rel_err(got, ref(planes, coeffs, xs[i])) <= TOL, (rows, I, k, a8, i)
