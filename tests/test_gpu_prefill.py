"""The prefill GEMM on SBVR weights (sbvr_gemm_prefill) against the oracle.

  * Per token, the oracle's exact result y_ref = W_hat x (binary64, exactly
    decoded weights) with the gate max|y - y_ref| / max|y_ref| <= 1e-3.
  * The weights the kernel multiplies are pinned bit for bit: with unit
    vectors as tokens, Y[t][o] is one product 1 * w, exact, so it must equal
    the correctly rounded binary16 weight (numpy's rounding of the oracle's
    exact decoding -- the matrix sbvr_decompress writes).
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


def log(msg):
    print(msg, flush=True)


def packed(sb, planes, coeffs):
    W = sb.pack(dev(planes.view(np.int32)), dev(coeffs.view(np.int16)))
    torch.cuda.synchronize()
    return W


def run(sb, W, X):
    Y = sb.gemm_prefill(W, dev(X))
    torch.cuda.synchronize()
    return Y.cpu().numpy().astype(np.float64)


def rel_err(y, y_ref):
    den = np.abs(y_ref).max()
    return float(np.abs(y - y_ref).max() / den) if den > 0 else float(np.abs(y).max())


def fp16_weights(planes, coeffs, rows=None):
    with np.errstate(over="ignore"):
        Wh = oracle.decompress(planes if rows is None else planes[rows], coeffs if rows is None else coeffs[rows])
        return Wh.astype(np.float16).astype(np.float64)


def check(Y, X, planes, coeffs, rows=None, what=""):
    """Per token: the exact-weight gate."""
    y_ref = oracle.sbvr_gemv(planes, coeffs, X, rows=rows)
    Yr = Y if rows is None else Y[:, rows]
    worst = max(rel_err(Yr[t], y_ref[t]) for t in range(X.shape[0]))
    log(f"prefill {what}: worst per-token err vs exact weights {worst:.3e}")
    assert worst <= TOL, (what, worst)


def check_unit_tokens(sb, W, planes, coeffs, cols, what=""):
    """Tokens e_j for the columns `cols`: Y[t][o] must be fp16(w_hat[o][j_t])."""
    I = planes.shape[1] * 128
    X = np.zeros((len(cols), I), dtype=np.float16)
    X[np.arange(len(cols)), cols] = 1.0
    Y = sb.gemm_prefill(W, dev(X))
    torch.cuda.synchronize()
    want = fp16_weights(planes, coeffs)[:, cols].T
    got = Y.cpu().numpy().astype(np.float64)
    assert np.array_equal(got, want), (what, int((got != want).sum()))


@pytest.mark.parametrize("T", [1, 16, 64, 512])
def test_prefill_oracle_encoded(sb, T):
    """An oracle-encoded 1024 x 4096 matrix (N(0, 0.02^2) with outliers,
    Algorithm 1, k = 4), prompts of 1, 16, 64 and 512 tokens."""
    O, I = 1024, 4096
    W = synth.weights(O, I, 0.02, seed=synth.seed_for(1, 0, 1), outlier_frac=0.001)
    planes, coeffs = oracle.encode_matrix(W, 4)
    X = synth.activations(I, seed=700 + T, batch=T)
    check(run(sb, packed(sb, planes, coeffs), X), X, planes, coeffs, what=f"encoded {O}x{I} T={T}")


@pytest.mark.parametrize("O,I,k,T", [(1, 128, 4, 1), (1001, 640, 3, 37), (70, 896, 2, 130), (33, 2560, 1, 17),
                                     (257, 4096, 4, 65), (64, 256, 4, 16), (129, 1152, 2, 3)])
def test_prefill_ragged(sb, O, I, k, T):
    """Row counts that are not a multiple of the 64-row workgroup (nor of the
    device tile), token counts that are not a multiple of 16, ragged last
    gblocks, k = 1..4, one group per K-slice and more."""
    planes, coeffs = synth.random_sbvr(O, I, k, seed=O + 3 * I + k)
    W = packed(sb, planes, coeffs)
    X = synth.activations(I, seed=O + T, batch=T)
    check(run(sb, W, X), X, planes, coeffs, what=f"ragged {O}x{I} k={k} T={T}")
    # every column of the first and the last group, as unit tokens
    cols = np.r_[np.arange(128), np.arange(I - 128, I)] if I > 128 else np.arange(128)
    check_unit_tokens(sb, W, planes, coeffs, cols, what=f"ragged {O}x{I} k={k}")


@pytest.mark.parametrize("O,I", [(14336, 4096), (4096, 14336), (4096, 4096), (1024, 4096), (8192, 8192)])
@pytest.mark.parametrize("T", [64, 128, 256, 512])
def test_prefill_full_size_sampled(sb, O, I, T):
    """Llama-3-8B projection shapes (and the 70B q/o shape) at the
    benchmark's prompt lengths, on sampled rows (first and last included) and
    every token; 256 tokens runs the long-prompt kernel with 8 activation
    chunks per thread (4096 rows: 64-token tiles over four K-slices; 14336
    rows: 128-token tiles over two)."""
    planes, coeffs = synth.random_sbvr(O, I, 4, seed=O + 7 * I)
    X = synth.activations(I, seed=T + O, batch=T)
    rows = np.unique(np.r_[0, O - 1, np.random.default_rng(T).integers(0, O, 62)])
    check(run(sb, packed(sb, planes, coeffs), X), X, planes, coeffs, rows=rows, what=f"full {O}x{I} T={T}")


# The long-prompt kernel (32 x 32 instructions; it runs from 96 tokens where
# its grid has >= 192 workgroups): one case per launch shape the rule picks
# -- (column tiles, token tiles, K-slices) = (1,1,1), (1,1,2), (1,1,4),
# (1,2,1), (1,2,2), (1,4,1), (1,2,4) and (1,4,2) (8 activation chunks per
# thread), (2,1,4), (2,2,2), then (1,4,1) with 240 workgroups and (2,1,2) --
# with ragged row and token counts and k = 1..4.
LONG_CASES = [(1500, 128, 1, 1000), (6144, 256, 2, 100), (1500, 512, 3, 256), (8192, 128, 4, 333),
              (6144, 256, 1, 200), (6144, 128, 3, 1000), (6144, 512, 2, 100), (8192, 256, 4, 333),
              (3000, 512, 1, 256), (12288, 256, 2, 300), (12288, 128, 2, 640), (12288, 256, 3, 160)]


@pytest.mark.parametrize("O,I,k,T", LONG_CASES)
def test_prefill_long_prompt_shapes(sb, O, I, k, T):
    """Sampled rows, every token, against the product the prefill path
    defines, X times the binary16-rounded weights (binary64); and against the
    exact weights where a row has at least 512 terms.  (With a single group
    the rounding of the weights and of the output alone reach the gate: for
    8192 x 128, k = 4, T = 333 the binary64 product of the rounded weights,
    rounded to binary16, is 1.016e-3 from the exact-weight result.)"""
    planes, coeffs = synth.random_sbvr(O, I, k, seed=O + 5 * I + k + T)
    W = packed(sb, planes, coeffs)
    X = synth.activations(I, seed=O + T + 1, batch=T)
    rows = np.unique(np.r_[0, O - 1, np.random.default_rng(O + T).integers(0, O, 62)])
    Y = run(sb, W, X)
    y16 = X.astype(np.float64) @ fp16_weights(planes, coeffs, rows).T
    worst = max(rel_err(Y[t, rows], y16[t]) for t in range(T))
    log(f"prefill long {O}x{I} k={k} T={T}: worst per-token err vs binary16 weights {worst:.3e}")
    assert worst <= TOL, worst
    if I >= 512:
        check(Y, X, planes, coeffs, rows=rows, what=f"long {O}x{I} k={k} T={T}")


def test_prefill_long_prompt_weights_bit_exact(sb):
    """The long-prompt kernel multiplies the correctly rounded binary16
    weights: unit tokens for the first 128 columns (T = 128, one K-slice
    shape) and for all 512 (T = 512, another), ordinary and wide coefficient
    spans (the binary64 table path); and all 512 columns of a 12288-row
    matrix (the 1 x 4 x 1 shape)."""
    O12, I12 = 12288, 512
    planes, coeffs = synth.random_sbvr(O12, I12, 4, seed=76)
    check_unit_tokens(sb, packed(sb, planes, coeffs), planes, coeffs, np.arange(I12), what="long 1x4 T=512")
    O, I, k = 4096, 512, 4
    planes, coeffs = synth.random_sbvr(O, I, k, seed=77)
    W = packed(sb, planes, coeffs)
    check_unit_tokens(sb, W, planes, coeffs, np.arange(128), what="long T=128")
    check_unit_tokens(sb, W, planes, coeffs, np.arange(I), what="long T=512")
    c = coeffs.view(np.float16).copy()
    c[::2, :, 3] = np.float16(3e-6) * np.sign(c[::2, :, 3]).astype(np.float16)
    c[1::4, :, 0] = np.float16(1500.0)
    coeffs = c.view(np.uint16)
    W = packed(sb, planes, coeffs)
    check_unit_tokens(sb, W, planes, coeffs, np.arange(I), what="long wide span")
    X = synth.activations(I, seed=78, batch=512, scale=0.05)
    rows = np.unique(np.r_[0, O - 1, np.random.default_rng(79).integers(0, O, 62)])
    check(run(sb, W, X), X, planes, coeffs, rows=rows, what="long wide span")


def test_prefill_wide_coefficient_span(sb):
    """Coefficient sets spanning more than 12 binades (their subset sums are
    not exact in binary32, so the table falls back to binary64 sums), next to
    ordinary ones; the weights must still be the correctly rounded ones."""
    O, I, k, T = 96, 512, 4, 20
    planes, coeffs = synth.random_sbvr(O, I, k, seed=41)
    c = coeffs.view(np.float16).copy()
    c[::2, :, 3] = np.float16(3e-6) * np.sign(c[::2, :, 3]).astype(np.float16)  # a subnormal term beside ~1e-2
    c[1::4, :, 0] = np.float16(1500.0)
    coeffs = c.view(np.uint16)
    X = synth.activations(I, seed=43, batch=T, scale=0.05)
    W = packed(sb, planes, coeffs)
    check(run(sb, W, X), X, planes, coeffs, what="wide coefficient span")
    check_unit_tokens(sb, W, planes, coeffs, np.arange(I), what="wide coefficient span")


def test_prefill_matches_decompress_and_is_deterministic(sb):
    """The fused kernel multiplies the same binary16 weights sbvr_decompress
    writes (compared with a binary64 GEMM on the decompressed matrix), and
    repeated calls give identical bits."""
    O, I, T = 300, 1024, 48
    planes, coeffs = synth.random_sbvr(O, I, 4, seed=12)
    W = packed(sb, planes, coeffs)
    X = synth.activations(I, seed=13, batch=T)
    M = sb.decompress(W).cpu().numpy().astype(np.float64)
    assert np.array_equal(M, fp16_weights(planes, coeffs))
    Y1 = sb.gemm_prefill(W, dev(X))
    Y2 = sb.gemm_prefill(W, dev(X))
    torch.cuda.synchronize()
    assert torch.equal(Y1.view(torch.int16), Y2.view(torch.int16))
    check(Y1.cpu().numpy().astype(np.float64), X, planes, coeffs, what="vs decompress")


def test_prefill_error_paths(sb):
    O, I = 64, 256
    planes, coeffs = synth.random_sbvr(O, I, 4, seed=5)
    W = packed(sb, planes, coeffs)
    X = dev(synth.activations(I, seed=6, batch=4))
    Y = torch.full((4, O), 7.0, dtype=torch.float16, device="cuda")
    p, c = W.planes.data_ptr(), W.coeffs.data_ptr()
    assert sb.sbvr_gemm_prefill(O, I, 4, p, c, X.data_ptr(), Y.data_ptr(), 0, 0) == sb.SBVR_E_INVALID_ARG
    assert sb.sbvr_gemm_prefill(O, I, 4, p, c, X.data_ptr() + 8, Y.data_ptr(), 4, 0) == sb.SBVR_E_ALIGNMENT
    assert sb.sbvr_gemm_prefill(O, 100, 4, p, c, X.data_ptr(), Y.data_ptr(), 4, 0) == sb.SBVR_E_INVALID_ARG
    assert sb.sbvr_gemm_prefill(O, I, 5, p, c, X.data_ptr(), Y.data_ptr(), 4, 0) == sb.SBVR_E_UNSUPPORTED
    # token counts past 2^22 are refused before anything is read
    assert sb.sbvr_gemm_prefill(O, I, 4, p, c, X.data_ptr(), Y.data_ptr(), (1 << 22) + 1, 0) == sb.SBVR_E_UNSUPPORTED
    torch.cuda.synchronize()
    assert bool((Y == 7.0).all())  # nothing was written


def test_prefill_graph_replays_match_eager(sb):
    """Both prefill kernels (a 64-token and a 512-token prompt) captured in a
    HIP graph, replayed three times with eager work in between: every replay
    gives the eager bits."""
    O, I = 4096, 1024
    planes, coeffs = synth.random_sbvr(O, I, 4, seed=91)
    W = packed(sb, planes, coeffs)
    Xs = [dev(synth.activations(I, seed=92 + T, batch=T)) for T in (64, 512)]
    eager = [sb.gemm_prefill(W, X).clone() for X in Xs]
    outs = [torch.empty((X.shape[0], O), dtype=torch.float16, device="cuda") for X in Xs]
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for X, Y in zip(Xs, outs):
            sb.gemm_prefill(W, X, out=Y, stream=s)
    for rep in range(3):
        for Y in outs:
            Y.fill_(0)
        sb.gemm_prefill(W, Xs[0])  # eager work between the replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for e, Y in zip(eager, outs):
            assert torch.equal(e.view(torch.int16), Y.view(torch.int16)), rep


# Property test over random shapes and prompt lengths (Hypothesis,
# derandomised: every run draws the same examples, no example database):
# both prefill kernels and whatever long-prompt launch shape the rule picks.
hypothesis = pytest.importorskip("hypothesis")
from hypothesis import HealthCheck, given, settings  # noqa: E402
from hypothesis import strategies as st  # noqa: E402


@settings(max_examples=24, deadline=None, derandomize=True, database=None,
          suppress_health_check=[HealthCheck.function_scoped_fixture, HealthCheck.too_slow])
@given(O=st.integers(64, 12288), G=st.integers(1, 12), k=st.integers(1, 4), T=st.integers(1, 700),
       seed=st.integers(0, 2 ** 16))
def test_prefill_random_shapes(sb, O, G, k, T, seed):
    """Sampled rows (first and last included), every token: within the gate of
    the binary64 product with the rounded binary16 weights, and of the exact
    weights where a row has at least 512 terms.  Output vectors of at least 64
    rows: the gate normalises by the vector's largest entry, and for a single
    row it becomes the relative error of one binary32-accumulated dot product,
    which cancellation can push past 1e-3 (a 1 x 128 matrix, k = 1, gave
    1.2e-2 on one of 577 tokens whose sum was 0.03 % of its terms'
    magnitudes)."""
    I = 128 * G
    planes, coeffs = synth.random_sbvr(O, I, k, seed=seed)
    X = synth.activations(I, seed=seed + 1, batch=T)
    Y = run(sb, packed(sb, planes, coeffs), X)
    rows = np.unique(np.r_[0, O - 1, np.random.default_rng(seed).integers(0, O, 40)])
    y16 = X.astype(np.float64) @ fp16_weights(planes, coeffs, rows).T
    worst = max(rel_err(Y[t, rows], y16[t]) for t in range(T))
    log(f"prefill random {O}x{I} k={k} T={T}: worst per-token err vs binary16 weights {worst:.3e}")
    assert worst <= TOL, worst
    if I >= 512:
        check(Y, X, planes, coeffs, rows=rows, what=f"random {O}x{I} k={k} T={T}")
