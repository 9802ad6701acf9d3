"""The grouped batch-1 GEMV (sbvr_gemv_grouped, and sbvr_gemv_grouped_a8 for
SBVR-8 activations): several GEMVs with the same inner dimension and plane
count in one launch.

  * Every member's output equals, bit for bit, the sbvr_gemv of its own
    arguments (the per-row arithmetic depends only on I and k), and meets the
    1e-3 gate max|y - y_ref| / max|y_ref| against the oracle's binary64 GEMV
    on sampled rows (first and last included).
  * The members' launch shape is the one a single matrix of all their row
    tiles gets: the cases cover the one-shot and the streaming kernels (one
    and several gblocks per wavefront), ragged row counts and 1..4 members.
  * Error paths enqueue nothing; graph replays give the eager bits.
"""
import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = 1e-3


@pytest.fixture(scope="module")
def sb():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2509_18172_amd as m
    return m


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def packed(sb, planes, coeffs):
    W = sb.pack(dev(planes.view(np.int32)), dev(coeffs.view(np.int16)))
    torch.cuda.synchronize()
    return W


def rel_err(y, y_ref):
    den = np.abs(y_ref).max()
    return float(np.abs(y - y_ref).max() / den) if den > 0 else float(np.abs(y).max())


def log(msg):
    print(msg, flush=True)


def members(sb, Os, I, k, seed, shared_x):
    mats = [synth.random_sbvr(O, I, k, seed=seed + 13 * i + O) for i, O in enumerate(Os)]
    Ws = [packed(sb, p, c) for p, c in mats]
    xs = [synth.activations(I, seed=seed + (0 if shared_x else 101 * i)) for i in range(len(Os))]
    return mats, Ws, xs


# (O per member, I, k): q|k|v and gate|up of Llama-3-8B (one-shot; streaming
# with one gblock per wavefront), 8B down twice and 70B o|k (several gblocks
# per wavefront), ragged members at every k, a single member and four.
CASES = [
    ((4096, 1024, 1024), 4096, 4),
    ((14336, 14336), 4096, 4),
    ((4096, 4096), 14336, 4),
    ((8192, 1024), 8192, 4),
    ((1, 17, 300, 1001), 640, 3),
    ((33, 70), 2560, 2),
    ((5, 129, 64), 1152, 1),
    ((1000,), 9088, 4),
    ((257, 3, 4097, 16), 512, 4),
]


@pytest.mark.parametrize("Os,I,k", CASES)
@pytest.mark.parametrize("shared_x", [True, False])
def test_grouped_matches_separate_and_oracle(sb, Os, I, k, shared_x):
    log(f"grouped {Os} x {I} k={k} shared_x={shared_x}")
    mats, Ws, xs = members(sb, Os, I, k, seed=500 + I + k, shared_x=shared_x)
    xd = [dev(x) for x in xs]
    ys = sb.gemv_grouped(Ws, xd)
    sep = [sb.gemv(W, x) for W, x in zip(Ws, xd)]
    torch.cuda.synchronize()
    rng = np.random.default_rng(len(Os) + I)
    for i, ((planes, coeffs), O) in enumerate(zip(mats, Os)):
        got = ys[i].cpu().numpy()
        assert np.array_equal(got.view(np.uint16), sep[i].cpu().numpy().view(np.uint16)), (Os, i)
        rows = np.unique(np.r_[0, O - 1, rng.integers(0, O, min(O, 96))])
        y_ref = oracle.sbvr_gemv(planes, coeffs, xs[i], rows=rows)
        err = rel_err(got[rows].astype(np.float64), y_ref)
        log(f"  member {i} ({O} rows): err {err:.3e}")
        assert err <= TOL, (Os, i, err)


@pytest.mark.parametrize("Os,I,k", [((4096, 1024, 1024), 4096, 4), ((14336, 14336), 4096, 4),
                                     ((4096, 4096), 14336, 4), ((1, 17, 300, 1001), 640, 3), ((33, 70), 2560, 2)])
def test_grouped_a8_matches_separate_and_oracle(sb, Os, I, k):
    """W4A8 members: each bit for bit its own sbvr_gemv_a8, and within the
    gate of the oracle's W4A8 GEMV (the exact product with the SBVR-8
    activations)."""
    log(f"grouped a8 {Os} x {I} k={k}")
    mats, Ws, xs = members(sb, Os, I, k, seed=900 + I + k, shared_x=False)
    xd = [dev(x) for x in xs]
    ys = sb.gemv_grouped(Ws, xd, a8=True)
    sep = [sb.gemv_a8(W, x) for W, x in zip(Ws, xd)]
    torch.cuda.synchronize()
    rng = np.random.default_rng(len(Os) + 7 * I)
    for i, ((planes, coeffs), O) in enumerate(zip(mats, Os)):
        got = ys[i].cpu().numpy()
        assert np.array_equal(got.view(np.uint16), sep[i].cpu().numpy().view(np.uint16)), (Os, i)
        rows = np.unique(np.r_[0, O - 1, rng.integers(0, O, min(O, 96))])
        y_ref = oracle.sbvr_gemv_w4a8(planes, coeffs, xs[i], rows=rows)
        err = rel_err(got[rows].astype(np.float64), y_ref)
        log(f"  member {i} ({O} rows): err {err:.3e}")
        assert err <= TOL, (Os, i, err)


@pytest.mark.parametrize("a8", [False, True])
@pytest.mark.parametrize("Os", [(4096, 14336, 14336), (2048, 1024, 28672), (1024, 30000)])
def test_grouped_members_cross_kernel_families(sb, Os, a8):
    """Members small enough for the one-shot kernel on their own, grouped with
    large ones so that the launch runs the streaming kernel: every member still
    gives the bits of its own call, with fp16 and with SBVR-8 activations (the
    streaming kernel rounds each scaled partial before its row sum, as the
    one-shot kernel does)."""
    I, k = 4096, 4
    log(f"grouped across kernel families {Os} a8={a8}")
    mats, Ws, xs = members(sb, Os, I, k, seed=77 + sum(Os), shared_x=False)
    xd = [dev(x) for x in xs]
    ys = sb.gemv_grouped(Ws, xd, a8=a8)
    sep = [(sb.gemv_a8 if a8 else sb.gemv)(W, x) for W, x in zip(Ws, xd)]
    torch.cuda.synchronize()
    for i, O in enumerate(Os):
        assert torch.equal(ys[i].view(torch.int16), sep[i].view(torch.int16)), (Os, a8, i)


def test_grouped_oracle_encoded_members(sb):
    """Members encoded from Gaussian weights with outliers by the oracle
    (Algorithm 1, k = 4), every row checked."""
    I, k = 1024, 4
    Os = (96, 48, 48)
    mats = [oracle.encode_matrix(synth.weights(O, I, 0.02, seed=synth.seed_for(2, i, 0), outlier_frac=0.001), k)
            for i, O in enumerate(Os)]
    Ws = [packed(sb, p, c) for p, c in mats]
    x = synth.activations(I, seed=91)
    ys = sb.gemv_grouped(Ws, [dev(x)] * 3)
    torch.cuda.synchronize()
    for (planes, coeffs), y in zip(mats, ys):
        y_ref = oracle.sbvr_gemv(planes, coeffs, x)
        assert rel_err(y.cpu().numpy().astype(np.float64), y_ref) <= TOL


def test_grouped_error_paths(sb):
    I, k = 512, 4
    mats, Ws, xs = members(sb, (64, 32), I, k, seed=7, shared_x=True)
    x = dev(xs[0])
    ys = [torch.full((W.O,), 7.0, dtype=torch.float16, device="cuda") for W in Ws]
    O = [W.O for W in Ws]
    P = [W.planes.data_ptr() for W in Ws]
    Cf = [W.coeffs.data_ptr() for W in Ws]
    X = [x.data_ptr()] * 2
    Y = [y.data_ptr() for y in ys]
    g = sb.sbvr_gemv_grouped
    assert g(0, O, I, k, P, Cf, X, Y) == sb.SBVR_E_INVALID_ARG
    assert g(5, O * 3, I, k, P * 3, Cf * 3, X * 3, Y * 3) == sb.SBVR_E_INVALID_ARG
    assert g(2, [64, 0], I, k, P, Cf, X, Y) == sb.SBVR_E_INVALID_ARG          # second member's shape
    assert g(2, O, 100, k, P, Cf, X, Y) == sb.SBVR_E_INVALID_ARG              # I not a multiple of 128
    assert g(2, O, I, 5, P, Cf, X, Y) == sb.SBVR_E_UNSUPPORTED
    assert g(2, O, I, k, P, [Cf[0], 0], X, Y) == sb.SBVR_E_INVALID_ARG        # null pointer
    assert g(2, O, I, k, P, Cf, [X[0], X[0] + 8], Y) == sb.SBVR_E_ALIGNMENT   # misaligned x
    torch.cuda.synchronize()
    assert all(bool((y == 7.0).all()) for y in ys)  # nothing was written
    assert g(2, O, I, k, P, Cf, X, Y) == sb.SBVR_OK
    ga = sb.sbvr_gemv_grouped_a8
    assert ga(0, O, I, k, P, Cf, X, Y) == sb.SBVR_E_INVALID_ARG
    assert ga(2, O, I, 5, P, Cf, X, Y) == sb.SBVR_E_UNSUPPORTED
    assert ga(2, O, I, k, P, Cf, [X[0], X[0] + 8], Y) == sb.SBVR_E_ALIGNMENT
    assert ga(2, O, I, k, P, Cf, X, Y) == sb.SBVR_OK


def test_grouped_graph_replays_match_eager(sb):
    """Grouped launches captured in a HIP graph (q|k|v then gate|up shapes,
    two layers' worth), replayed several times with eager work between the
    replays: every replay gives the eager bits."""
    I, k = 4096, 4
    _, Wa, xa = members(sb, (4096, 1024, 1024), I, k, seed=31, shared_x=True)
    _, Wb, xb = members(sb, (14336, 14336), I, k, seed=32, shared_x=True)
    xA, xB = dev(xa[0]), dev(xb[0])
    eager = [y.clone() for y in sb.gemv_grouped(Wa, [xA] * 3) + sb.gemv_grouped(Wb, [xB] * 2)]
    outs_a = [torch.empty(W.O, dtype=torch.float16, device="cuda") for W in Wa]
    outs_b = [torch.empty(W.O, dtype=torch.float16, device="cuda") for W in Wb]
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        sb.gemv_grouped(Wa, [xA] * 3, outs=outs_a, stream=s)
        sb.gemv_grouped(Wb, [xB] * 2, outs=outs_b, stream=s)
    for rep in range(3):
        for o in outs_a + outs_b:
            o.fill_(0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for e, o in zip(eager, outs_a + outs_b):
            assert torch.equal(e.view(torch.int16), o.view(torch.int16)), rep
