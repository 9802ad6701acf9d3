"""GPU parity of the HIP SBVR path against the CPU oracle, through the C ABI.

Gate (per activation vector): max_o |y - y_ref| / max_o |y_ref| <= 1e-3, with
y_ref the binary64 GEMV of the exactly decompressed matrix.  Repacking is
checked bit for bit.  Inputs are seeded: Gaussian weights encoded by the
oracle (Algorithm 1) where encoding is fast enough, and directly drawn SBVR
tensors (uniform planes, Gaussian fp16 coefficients) at the full Llama-3-8B
and 70B projection shapes, which are the launch configurations the bench
times.
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


def canon_to_dev(planes, coeffs):
    return dev(planes.view(np.int32)), dev(coeffs.view(np.int16))


def packed(sb, planes, coeffs):
    p, c = canon_to_dev(planes, coeffs)
    W = sb.pack(p, c)
    torch.cuda.synchronize()
    return W


def rel_err(y, y_ref):
    y = np.asarray(y, dtype=np.float64)
    den = np.abs(y_ref).max()
    return float(np.abs(y - y_ref).max() / den) if den > 0 else float(np.abs(y).max())


def run_gemv(sb, W, x16):
    y = sb.gemv(W, dev(x16))
    torch.cuda.synchronize()
    return y.cpu().numpy().astype(np.float64)


def run_gemm(sb, W, X16):
    Y = sb.gemm_small_batch(W, dev(X16))
    torch.cuda.synchronize()
    return Y.cpu().numpy().astype(np.float64)


def log(msg):
    print(msg, flush=True)


# --------------------------------------------------------------------------
# Repacking: bit-exact round trip
# --------------------------------------------------------------------------

@pytest.mark.parametrize("O,I,k", [(1, 128, 4), (5, 640, 3), (17, 384, 2), (1000, 1024, 1),
                                   (4096, 4096, 4), (1024, 14336, 4), (9, 896, 4)])
def test_pack_unpack_round_trip(sb, O, I, k):
    planes, coeffs = synth.random_sbvr(O, I, k, seed=O * 31 + I + k)
    W = packed(sb, planes, coeffs)
    p2, c2 = sb.unpack(W)
    torch.cuda.synchronize()
    assert np.array_equal(p2.cpu().numpy().view(np.uint32), planes)
    assert np.array_equal(c2.cpu().numpy().view(np.uint16), coeffs)
    assert W.planes.numel() == sb.sbvr_packed_plane_bytes(O, I, k)


# --------------------------------------------------------------------------
# configs: oracle-encoded Gaussian weights
# --------------------------------------------------------------------------

def test_cfg1_single_gemv_seed0(sb):
    """1024 x 1024, k = 4, seed 0: W ~ N(0, 0.02^2) encoded by Algorithm 1."""
    W = synth.weights(1024, 1024, 0.02, seed=0)
    planes, coeffs = oracle.encode_matrix(W, 4)
    x = synth.activations(1024, seed=synth.X_SEED_OFFSET)
    Wd = packed(sb, planes, coeffs)
    p2, c2 = sb.unpack(Wd)
    assert np.array_equal(p2.cpu().numpy().view(np.uint32), planes)
    y = run_gemv(sb, Wd, x)
    y_ref = oracle.sbvr_gemv(planes, coeffs, x)
    err = rel_err(y, y_ref)
    log(f"cfg1 1024x1024 k=4 err={err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("k", [4, 3, 2])
@pytest.mark.parametrize("I", [4096, 14336])
def test_encoded_llama8b_rows_with_outliers(sb, k, I):
    """Rows of the Llama-3-8B shapes, N(0, 0.02^2) + 0.1% outliers at +-8 sigma."""
    O = 48
    W = synth.weights(O, I, 0.02, seed=synth.seed_for(2, 0, 4 if I == 4096 else 6), outlier_frac=0.001)
    planes, coeffs = oracle.encode_matrix(W, k)
    x = synth.activations(I, seed=synth.seed_for(2, 0, 4) + synth.X_SEED_OFFSET)
    y = run_gemv(sb, packed(sb, planes, coeffs), x)
    err = rel_err(y, oracle.sbvr_gemv(planes, coeffs, x))
    log(f"encoded {O}x{I} k={k} err={err:.3e}")
    assert err <= TOL


# --------------------------------------------------------------------------
# Full-size shapes in the bench's launch configuration
# --------------------------------------------------------------------------

SHAPES_8B = sorted(set(synth.LLAMA8B.values()))
SHAPES_70B = sorted(set(synth.LLAMA70B.values()))


@pytest.mark.parametrize("O,I", SHAPES_8B + SHAPES_70B)
def test_full_size_k4(sb, O, I):
    planes, coeffs = synth.random_sbvr(O, I, 4, seed=O + 7 * I)
    x = synth.activations(I, seed=O + I + synth.X_SEED_OFFSET)
    y = run_gemv(sb, packed(sb, planes, coeffs), x)
    y_ref = oracle.sbvr_gemv(planes, coeffs, x)
    err = rel_err(y, y_ref)
    log(f"full {O}x{I} k=4 err={err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("k", [2, 3])
@pytest.mark.parametrize("O,I", SHAPES_8B)
def test_full_size_low_bit(sb, O, I, k):
    planes, coeffs = synth.random_sbvr(O, I, k, seed=O + 7 * I + k)
    x = synth.activations(I, seed=O + I + k + synth.X_SEED_OFFSET)
    y = run_gemv(sb, packed(sb, planes, coeffs), x)
    err = rel_err(y, oracle.sbvr_gemv(planes, coeffs, x))
    log(f"full {O}x{I} k={k} err={err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("B", [1, 2, 3, 4, 5, 6, 8])
@pytest.mark.parametrize("O,I", SHAPES_8B)
def test_small_batch_full_size(sb, O, I, B):
    planes, coeffs = synth.random_sbvr(O, I, 4, seed=O + 3 * I)
    X = synth.activations(I, seed=B + O + synth.X_SEED_OFFSET, batch=B)
    W = packed(sb, planes, coeffs)
    Y = run_gemm(sb, W, X)
    Y_ref = oracle.sbvr_gemv(planes, coeffs, X)
    errs = [rel_err(Y[b], Y_ref[b]) for b in range(B)]
    log(f"small batch {O}x{I} B={B} worst err={max(errs):.3e}")
    assert max(errs) <= TOL
    # each vector agrees with the batch-1 kernel to the same bar
    y0 = run_gemv(sb, W, X[0])
    assert rel_err(Y[0], y0.astype(np.float64)) <= TOL


@pytest.mark.parametrize("B", [2, 3, 4, 8])
@pytest.mark.parametrize("O,I", SHAPES_70B)
def test_small_batch_70b_full_size(sb, O, I, B):
    """Llama-3-70B shapes at B = 2, 3, 4 and 8 (every wavefront takes several
    gblocks; B <= 4 runs the depth-4 ring): the 28672-row shapes need more
    LDS per workgroup than a launch may request unless tiles per workgroup
    are capped."""
    planes, coeffs = synth.random_sbvr(O, I, 4, seed=O + 5 * I + B)
    X = synth.activations(I, seed=B + 3 * O + synth.X_SEED_OFFSET, batch=B)
    Y = run_gemm(sb, packed(sb, planes, coeffs), X)
    Y_ref = oracle.sbvr_gemv(planes, coeffs, X)
    errs = [rel_err(Y[b], Y_ref[b]) for b in range(B)]
    log(f"small batch 70b {O}x{I} B={B} worst err={max(errs):.3e}")
    assert max(errs) <= TOL


@pytest.mark.parametrize("k", [1, 2, 3])
def test_small_batch_low_bit(sb, k):
    O, I = 520, 1920
    planes, coeffs = synth.random_sbvr(O, I, k, seed=k)
    X = synth.activations(I, seed=k + 9, batch=6)
    Y = run_gemm(sb, packed(sb, planes, coeffs), X)
    Y_ref = oracle.sbvr_gemv(planes, coeffs, X)
    assert max(rel_err(Y[b], Y_ref[b]) for b in range(6)) <= TOL


# --------------------------------------------------------------------------
# Structured inputs with closed-form answers
# --------------------------------------------------------------------------

def fp16_ulp(v):
    """Spacing above |v| in binary16 (at the largest finite value, the
    spacing below it, 32)."""
    v = np.abs(np.asarray(v, dtype=np.float16))
    with np.errstate(over="ignore"):
        u = (np.nextafter(v, np.float16(np.inf)) - v).astype(np.float64)
    return np.where(np.isinf(u), 32.0, u)


def test_unit_vector_picks_a_column(sb):
    O, I = 256, 1024
    planes, coeffs = synth.random_sbvr(O, I, 4, seed=4)
    What = oracle.decompress(planes, coeffs)
    W = packed(sb, planes, coeffs)
    for j in (0, 1, 31, 32, 127, 128, 500, 1023):
        x = np.zeros(I, dtype=np.float16)
        x[j] = 1.0
        y = run_gemv(sb, W, x)
        col = What[:, j]
        assert np.all(np.abs(y - col.astype(np.float16)) <= fp16_ulp(col)), j


def test_zero_planes_give_positive_zero(sb):
    O, I = 64, 512
    planes = np.zeros((O, I // 128, 4, 4), dtype=np.uint32)
    coeffs = synth.random_sbvr(O, I, 4, seed=1)[1]
    y = sb.gemv(packed(sb, planes, coeffs), dev(synth.activations(I, seed=2)))
    torch.cuda.synchronize()
    assert np.all(y.cpu().numpy().view(np.uint16) == 0)


def test_all_ones_planes(sb):
    O, I = 64, 1024
    planes = np.full((O, I // 128, 3, 4), 0xFFFFFFFF, dtype=np.uint32)
    coeffs = synth.random_sbvr(O, I, 3, seed=5)[1]
    x = synth.activations(I, seed=6)
    y = run_gemv(sb, packed(sb, planes, coeffs), x)
    cf = coeffs.view(np.float16).astype(np.float64).sum(axis=2)           # [O][G]
    xs = x.astype(np.float64).reshape(-1, 128).sum(axis=1)                 # [G]
    assert rel_err(y, cf @ xs) <= TOL


@pytest.mark.parametrize("k", [2, 3, 4])
def test_power_of_two_coefficients_are_integer_codes(sb, k):
    """c_i = 2^i * delta makes every weight an unsigned k-bit integer code times
    delta, so y = delta * (Q x) with Q computed in integer arithmetic."""
    O, I = 200, 2048
    planes = synth.random_sbvr(O, I, k, seed=10 + k)[0]
    delta = 2.0 ** -9
    coeffs = np.broadcast_to(np.array([np.float16(delta * 2 ** i) for i in range(k)]).view(np.uint16),
                             (O, I // 128, k)).copy()
    bits = np.unpackbits(planes.view(np.uint8), bitorder="little").reshape(O, I // 128, k, 128)
    Q = (bits.astype(np.int64) << np.arange(k)[None, None, :, None]).sum(axis=2).reshape(O, I)
    x = synth.activations(I, seed=20 + k)
    y_ref = delta * (Q.astype(np.float64) @ x.astype(np.float64))
    y = run_gemv(sb, packed(sb, planes, coeffs), x)
    assert rel_err(y, y_ref) <= TOL


def test_twos_complement_coefficients(sb):
    """Eq. 12-style coefficients {-8, 1, 2, 4} * s: signed 4-bit integer codes."""
    O, I = 96, 1024
    planes = synth.random_sbvr(O, I, 4, seed=33)[0]
    s = 2.0 ** -6
    coeffs = np.broadcast_to(np.array([np.float16(v * s) for v in (-8, 1, 2, 4)]).view(np.uint16),
                             (O, I // 128, 4)).copy()
    # plane order (i = 0..3) pairs with (-8, 1, 2, 4)
    bits = np.unpackbits(planes.view(np.uint8), bitorder="little").reshape(O, I // 128, 4, 128)
    Q = (bits.astype(np.int64) * np.array([-8, 1, 2, 4])[None, None, :, None]).sum(axis=2).reshape(O, I)
    x = synth.activations(I, seed=34)
    y = run_gemv(sb, packed(sb, planes, coeffs), x)
    assert rel_err(y, s * (Q.astype(np.float64) @ x.astype(np.float64))) <= TOL


def test_linearity_and_determinism(sb):
    O, I = 4096, 4096
    planes, coeffs = synth.random_sbvr(O, I, 4, seed=77)
    W = packed(sb, planes, coeffs)
    x1 = synth.activations(I, seed=1).astype(np.float32)
    x2 = synth.activations(I, seed=2).astype(np.float32)
    x12 = (x1 + x2).astype(np.float16)
    y1 = run_gemv(sb, W, x1.astype(np.float16))
    y2 = run_gemv(sb, W, x2.astype(np.float16))
    y12 = run_gemv(sb, W, x12)
    ref12 = oracle.sbvr_gemv(planes, coeffs, x12)
    assert rel_err(y12, ref12) <= TOL
    assert rel_err(y1 + y2, ref12) <= 5 * TOL  # x1+x2 itself rounds to fp16
    again = run_gemv(sb, W, x12)
    assert np.array_equal(again, y12)  # fixed reduction order -> bit-identical reruns


# --------------------------------------------------------------------------
# Edge cases
# --------------------------------------------------------------------------

@pytest.mark.parametrize("O,I,k", [(1, 128, 4), (3, 128, 1), (1001, 640, 3), (7, 896, 4),
                                   (4097, 1152, 2), (130, 4224, 4), (2, 30720, 4),
                                   # few gblocks per row: the one-shot kernel's tiles per
                                   # workgroup follow the wavefront count (T = 2 in all three)
                                   (8192, 1024, 4), (8191, 896, 3), (2048, 4096, 4),
                                   # streaming at k = 4 with 8 gblocks per row (256 workgroups,
                                   # depth-4 ring): 3073 tiles, the last gblock holds 3 groups
                                   # and the last workgroup 5 tiles
                                   (12291, 3968, 4)])
def test_ragged_shapes(sb, O, I, k):
    planes, coeffs = synth.random_sbvr(O, I, k, seed=O + I + k)
    x = synth.activations(I, seed=O * 3 + 1)
    W = packed(sb, planes, coeffs)
    y_ref = oracle.sbvr_gemv(planes, coeffs, x)
    assert rel_err(run_gemv(sb, W, x), y_ref) <= TOL
    X = synth.activations(I, seed=O * 5 + 2, batch=3)
    Y = run_gemm(sb, W, X)
    Y_ref = oracle.sbvr_gemv(planes, coeffs, X)
    assert max(rel_err(Y[b], Y_ref[b]) for b in range(3)) <= TOL


@pytest.mark.parametrize("O,I,k", [
    # 18 gblocks per row (the last with 3 groups): the streaming kernel's 16
    # wavefronts take 2 or 1 gblocks, the small-batch kernel's 8 take 3 or 2
    (1000, 9088, 4),
    # 17 gblocks: one wavefront takes 2, fifteen take 1 (most uneven)
    (300, 8320, 2),
    # 29 gblocks, the last holding one group, k = 3
    (517, 14464, 3)])
def test_long_rows_uneven_gblock_assignment(sb, O, I, k):
    """Rows longer than 16 gblocks, whose gblock count does not divide over
    the wavefronts: batch 1, W4A8 (k = 4) and small batch B = 2, 5, 8 against
    the oracle, repeated calls bit-identical."""
    planes, coeffs = synth.random_sbvr(O, I, k, seed=O * 7 + I + k)
    W = packed(sb, planes, coeffs)
    x = synth.activations(I, seed=O + 11)
    y = run_gemv(sb, W, x)
    assert rel_err(y, oracle.sbvr_gemv(planes, coeffs, x)) <= TOL
    assert np.array_equal(y, run_gemv(sb, W, x))
    if k == 4:
        assert rel_err(run_gemv_a8(sb, W, x), oracle.sbvr_gemv_w4a8(planes, coeffs, x)) <= TOL
    for B in (2, 5, 8):
        X = synth.activations(I, seed=O + B, batch=B)
        Y = run_gemm(sb, W, X)
        Y_ref = oracle.sbvr_gemv(planes, coeffs, X)
        assert max(rel_err(Y[b], Y_ref[b]) for b in range(B)) <= TOL, B
        assert np.array_equal(Y, run_gemm(sb, W, X))


def test_activation_dynamic_range(sb):
    O, I = 128, 2048
    planes, coeffs = synth.random_sbvr(O, I, 4, seed=90, coeff_sigma=1e-4)
    W = packed(sb, planes, coeffs)
    rng = np.random.default_rng(0)
    # (activations, coefficient scale): y stays within the fp16 normal range
    cases = {
        "huge": (np.full(I, 60000.0), 1.0),
        "tiny": (rng.standard_normal(I) * 1e-6, 1e4),          # fp16 subnormal x
        "mixed": (np.where(rng.random(I) < 0.01, 3000.0, 1e-3) * rng.choice([-1, 1], I), 1.0),
        "zero": (np.zeros(I), 1.0),
        "one_big": (np.r_[65504.0, np.full(I - 1, 2.0 ** -24)], 1.0),
    }
    c_big = (coeffs.view(np.float16) * np.float16(1e4)).view(np.uint16)
    W_big = packed(sb, planes, c_big)
    W_one = packed(sb, planes, coeffs)
    for name, (xv, cscale) in cases.items():
        W, c_used = (W_big, c_big) if cscale != 1.0 else (W_one, coeffs)
        x = xv.astype(np.float16)
        y_ref = oracle.sbvr_gemv(planes, c_used, x)
        y = run_gemv(sb, W, x)
        if np.abs(y_ref).max() == 0:
            assert np.all(y == 0), name
        else:
            assert rel_err(y, y_ref) <= TOL, (name, rel_err(y, y_ref))
    # the same cases through the small-batch kernels, one vector each (each
    # vector has its own activation scale), for 2-, 4- and 8-vector kernels
    for cscale, W, c_used in ((1.0, W_one, coeffs), (1e4, W_big, c_big)):
        xs = [v.astype(np.float16) for v, c in cases.values() if c == cscale]
        for B in (2, 4, 8):
            X = np.stack([xs[b % len(xs)] if b % 3 else (xs[b % len(xs)] * np.float16(0.5)) for b in range(B)])
            Y = run_gemm(sb, W, X)
            Y_ref = oracle.sbvr_gemv(planes, c_used, X)
            for b in range(B):
                if np.abs(Y_ref[b]).max() == 0:
                    assert np.all(Y[b] == 0), (cscale, B, b)
                else:
                    assert rel_err(Y[b], Y_ref[b]) <= TOL, (cscale, B, b, rel_err(Y[b], Y_ref[b]))


def test_cancellation_regression_single_row(sb):
    """O = 1, I = 128, k = 1, B = 8 (uniform planes, N(0, 0.01^2) binary16
    coefficients, N(0, 1) activations; the seed a random-shape sweep drew):
    vector 0's output cancels to -1.0e-4 against products whose root sum of
    squares is 0.063.  Plain gate per vector, through the small-batch kernel
    and through the batch-1 kernel."""
    O, I, k, B = 1, 128, 1, 8
    seed = O * 131 + I + 7 * k + B
    planes, coeffs = synth.random_sbvr(O, I, k, seed=seed)
    X = synth.activations(I, seed=seed + synth.X_SEED_OFFSET, batch=B)
    W = packed(sb, planes, coeffs)
    Y_ref = oracle.sbvr_gemv(planes, coeffs, X)
    assert abs(Y_ref[0, 0]) < 2e-4
    Y = run_gemm(sb, W, X)
    for b in range(B):
        assert rel_err(Y[b], Y_ref[b]) <= TOL, (b, rel_err(Y[b], Y_ref[b]))
        assert rel_err(run_gemv(sb, W, X[b]), Y_ref[b]) <= TOL, b


def outlier_activations(I, ratio, seed, batch=1, per_block=3):
    """N(0, 1) binary16 activations with `per_block` elements of every
    512-element block replaced by +-ratio (activation outliers: a few
    channels far above the rest)."""
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((batch, I))
    for b in range(batch):
        for g0 in range(0, I, 512):
            pos = g0 + rng.choice(min(512, I - g0), size=min(per_block, I - g0), replace=False)
            X[b, pos] = ratio * rng.choice([-1.0, 1.0], size=pos.size)
    return X.astype(np.float16)


@pytest.mark.parametrize("ratio", [100.0, 1000.0, 30000.0])
@pytest.mark.parametrize("O,I", [(1024, 4096), (4096, 4096), (14336, 4096), (4096, 14336)])
def test_activation_outliers_plain_gate(sb, O, I, ratio):
    """Activation blocks with a few outliers 100x, 1000x and 30000x above the
    N(0, 1) bulk: every other element of the block is many binary16 binades
    below the block maximum.  Batch 1 (one-shot and streaming kernels) and
    B = 2, 8 against the oracle with the plain gate."""
    planes, coeffs = synth.random_sbvr(O, I, 4, seed=O + 3 * I + int(ratio))
    W = packed(sb, planes, coeffs)
    X = outlier_activations(I, ratio, seed=int(ratio) + O, batch=8)
    Y_ref = oracle.sbvr_gemv(planes, coeffs, X)
    err1 = rel_err(run_gemv(sb, W, X[0]), Y_ref[0])
    Y2 = run_gemm(sb, W, X[:2])
    Y8 = run_gemm(sb, W, X)
    err2 = max(rel_err(Y2[b], Y_ref[b]) for b in range(2))
    err8 = max(rel_err(Y8[b], Y_ref[b]) for b in range(8))
    log(f"outliers x{ratio:g} {O}x{I}: B=1 {err1:.3e} B=2 {err2:.3e} B=8 {err8:.3e}")
    assert max(err1, err2, err8) <= TOL


def test_output_canary_and_error_paths(sb):
    O, I = 100, 512
    planes, coeffs = synth.random_sbvr(O, I, 4, seed=3)
    W = packed(sb, planes, coeffs)
    x = dev(synth.activations(I, seed=4))
    buf = torch.full((O + 64,), 7.0, dtype=torch.float16, device="cuda")
    st = sb.sbvr_gemv(O, I, 4, W.planes.data_ptr(), W.coeffs.data_ptr(), x.data_ptr(),
                      buf.data_ptr(), None, 0, 0)
    torch.cuda.synchronize()
    assert st == 0
    assert torch.all(buf[O:] == 7.0)
    y_ref = oracle.sbvr_gemv(planes, coeffs, synth.activations(I, seed=4))
    assert rel_err(buf[:O].cpu().numpy().astype(np.float64), y_ref) <= TOL
    # invalid calls launch nothing: output untouched
    buf.fill_(5.0)
    torch.cuda.synchronize()
    for args in [(O, I, 5), (O, 100, 4), (0, I, 4)]:
        st = sb.sbvr_gemv(*args, W.planes.data_ptr(), W.coeffs.data_ptr(), x.data_ptr(),
                          buf.data_ptr(), None, 0, 0)
        assert st != 0
    st = sb.sbvr_gemv(O, I, 4, W.planes.data_ptr(), W.coeffs.data_ptr(), x.data_ptr() + 2,
                      buf.data_ptr(), None, 0, 0)
    assert st == sb.SBVR_E_ALIGNMENT
    st = sb.sbvr_gemm_small_batch(O, I, 4, W.planes.data_ptr(), W.coeffs.data_ptr(), x.data_ptr(),
                                  buf.data_ptr(), 9, None, 0, 0)
    assert st == sb.SBVR_E_INVALID_ARG
    torch.cuda.synchronize()
    assert torch.all(buf == 5.0)


@pytest.mark.parametrize("O,I", [(4096, 4096), (14336, 4096)])
def test_graph_capture_replays_match_eager(sb, O, I):
    """Every GEMV-type entry point (one-shot and streaming kernels), the
    decompression, the prefill GEMM (two launch shapes) and the encoding
    kernels, captured in one graph: each replay reproduces the eager results
    bit for bit."""
    planes, coeffs = synth.random_sbvr(O, I, 4, seed=123)
    W = packed(sb, planes, coeffs)
    n_sets = (O * (I // 128) + 9) // 10
    pi, ix, tb = synth.random_indexed_sbvr(O, I, 4, n_sets, seed=126)
    Wi = packed_indexed(sb, pi, ix, tb)
    x = dev(synth.activations(I, seed=124))
    X = dev(synth.activations(I, seed=125, batch=4))
    Wf = dev(synth.weights(64, I, 0.02, seed=127))
    X16, X80 = dev(synth.activations(I, seed=128, batch=16)), dev(synth.activations(I, seed=129, batch=80))
    calls = {
        "gemv": lambda out=None: sb.gemv(W, x, out=out),
        "small_batch": lambda out=None: sb.gemm_small_batch(W, X, out=out),
        "a8": lambda out=None: sb.gemv_a8(W, x, out=out),
        "indexed": lambda out=None: sb.gemv_indexed(Wi, x, out=out),
        "indexed_a8": lambda out=None: sb.gemv_indexed(Wi, x, out=out, a8=True),
        "decompress": lambda out=None: sb.decompress(W, out=out),
        "decompress_indexed": lambda out=None: sb.decompress(Wi, out=out),
        "prefill_16": lambda out=None: sb.gemm_prefill(W, X16, out=out),
        "prefill_80": lambda out=None: sb.gemm_prefill(W, X80, out=out),
    }
    eager = {n: f().clone() for n, f in calls.items()}
    ep, ec = sb.encode(Wf, 4)
    outs = {n: torch.empty_like(v) for n, v in eager.items()}
    enc_p, enc_c = torch.empty_like(ep), torch.empty_like(ec)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for n, f in calls.items():
            f(out=outs[n])
        assert sb.sbvr_encode(64, I, 4, Wf.data_ptr(), 8, 8, 16, 4, 1, enc_p.data_ptr(), enc_c.data_ptr(), None,
                              int(s.cuda_stream)) == 0
    for rep in range(4):
        for v in outs.values():
            v.zero_()
        enc_p.zero_()
        enc_c.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for n in calls:
            assert torch.equal(outs[n], eager[n]), (n, rep)
        assert torch.equal(enc_p, ep) and torch.equal(enc_c, ec), rep
        _ = (x.float() * 2).sum().item()  # eager work between replays


# --------------------------------------------------------------------------
# Prefill path: decompression to binary16 (bit-exact) and a library GEMM
# --------------------------------------------------------------------------

def oracle_fp16(planes, coeffs):
    """binary16 bits of the exact decoded weights (numpy rounds binary64 to
    binary16 to nearest, ties to even; overflow gives infinity)."""
    with np.errstate(over="ignore"):
        return oracle.decompress(planes, coeffs).astype(np.float16).view(np.uint16)


def run_decompress(sb, planes, coeffs):
    M = sb.decompress(packed(sb, planes, coeffs))
    torch.cuda.synchronize()
    return M.cpu().numpy().view(np.uint16)


@pytest.mark.parametrize("parts,I", [((4096, 1024, 1024), 4096), ((14336, 14336), 4096), ((3, 1001), 640)])
def test_rows_concatenated_match_separate_calls(sb, parts, I):
    """Projections that share an input packed as one matrix (rows
    concatenated, as q|k|v and gate|up are in a serving stack): the fused
    call gives every row the same value as the separate calls (the per-row
    arithmetic depends only on I), and meets the gate against the oracle."""
    k = 4
    mats = [synth.random_sbvr(O, I, k, seed=77 + O + i) for i, O in enumerate(parts)]
    x = synth.activations(I, seed=78)
    sep = np.concatenate([run_gemv(sb, packed(sb, p, c), x) for p, c in mats])
    planes = np.concatenate([p for p, _ in mats])
    coeffs = np.concatenate([c for _, c in mats])
    fused = run_gemv(sb, packed(sb, planes, coeffs), x)
    assert np.array_equal(fused, sep)
    rows = np.random.default_rng(3).choice(planes.shape[0], size=min(512, planes.shape[0]), replace=False)
    y_ref = oracle.sbvr_gemv(planes, coeffs, x, rows=rows)
    assert rel_err(fused[rows], y_ref) <= TOL


# Workgroups take 1, 2 or 4 gblocks by the matrix's block count; the larger
# cases cover 2 and 4 with a gblock count that is not a multiple of them.
@pytest.mark.parametrize("O,I,k", [(1, 128, 4), (3, 128, 1), (1001, 640, 3), (7, 896, 4), (4097, 1152, 2),
                                   (130, 4224, 4), (16, 512, 1), (4096, 4096, 4), (1024, 14336, 2),
                                   (8192, 2560, 4), (16384, 2560, 4), (16000, 2176, 3), (16384, 2176, 1),
                                   (32768, 2176, 2),
                                   (14336, 4096, 4)])
def test_decompress_bit_exact(sb, O, I, k):
    planes, coeffs = synth.random_sbvr(O, I, k, seed=O * 7 + I + k)
    got = run_decompress(sb, planes, coeffs)
    want = oracle_fp16(planes, coeffs)
    assert got.shape == (O, I)
    assert np.array_equal(got, want), int((got != want).sum())


def test_decompress_rounding_edges(sb):
    """Coefficient sets whose subset sums are ties, subnormals, exact
    cancellations and overflows of binary16."""
    h = lambda v: np.float16(v).view(np.uint16)  # noqa: E731
    quads = [
        (1.0, 2.0 ** -11, 0.0, 0.0),              # 1 + half ulp: tie -> 1.0
        (1.0 + 2.0 ** -10, 2.0 ** -11, 0.0, 0.0),  # tie -> even neighbour above
        (2048.0, 1.0, 0.0, 0.0),                  # 2049: tie -> 2048
        (2050.0, 1.0, 0.0, 0.0),                  # 2051: tie -> 2052
        (2.0 ** -14, -(2.0 ** -24), 0.0, 0.0),     # largest subnormal
        (3 * 2.0 ** -24, 2.0 ** -24, -(2.0 ** -24), 0.0),  # subnormal sums
        (65504.0, 65504.0, 0.0, 0.0),             # overflow -> inf
        (65504.0, 16.0, 0.0, 0.0),                # 65520: tie at the top -> inf
        (65504.0, 8.0, -65504.0, 0.0),            # 65512 -> 65504; exact cancellations
        (-1.0, -(2.0 ** -11), 1.0, 2.0 ** -24),   # negative tie, mixed signs
        (0.1, 0.2, 0.3, -0.6),                    # inexact decimals
        (-0.0, 0.0, -0.0, 1e-4),
    ]
    O, I, k = len(quads) * 3, 512, 4
    coeffs = np.zeros((O, I // 128, k), dtype=np.uint16)
    for r in range(O):
        coeffs[r, :, :] = [h(v) for v in quads[r % len(quads)]]
    rng = np.random.default_rng(1)
    planes = rng.integers(0, 2 ** 32, size=(O, I // 128, k, 4), dtype=np.uint64).astype(np.uint32)
    planes[: len(quads)] = 0xFFFFFFFF  # every subset sum present: all bits set, then random
    planes[len(quads): 2 * len(quads), :, :, 0] = 0xFFFFFFFF
    got = run_decompress(sb, planes, coeffs)
    want = oracle_fp16(planes, coeffs)
    assert np.array_equal(got, want), np.argwhere(got != want)[:5]


def test_prefill_gemm_with_library_matmul(sb):
    """Prefill: Y = X W^T over T tokens (a linear layer's layout, as the
    bench times it) with the decompressed W and a library GEMM (fp32
    accumulation), against the oracle per token."""
    O, I, T = 1024, 4096, 64
    W = synth.weights(O, I, 0.02, seed=synth.seed_for(2, 0, 1), outlier_frac=0.001)
    planes, coeffs = oracle.encode_matrix(W, 4)
    X = synth.activations(I, seed=99, batch=T)
    M = sb.decompress(packed(sb, planes, coeffs))
    Y = torch.nn.functional.linear(dev(X), M)         # [T][O], fp16 in, fp32 accumulate
    torch.cuda.synchronize()
    Y = Y.cpu().numpy().astype(np.float64)
    Y_ref = oracle.sbvr_gemv(planes, coeffs, X)
    errs = [rel_err(Y[t], Y_ref[t]) for t in range(T)]
    log(f"prefill {O}x{I} T={T} worst err={max(errs):.3e}")
    assert max(errs) <= TOL


# --------------------------------------------------------------------------
# W4A8 decode path: online conversion of x to SBVR-8 activations (Sec. 4.3,
# Eq. 12) inside the GEMV; reference = oracle.sbvr_gemv_w4a8
# --------------------------------------------------------------------------

def run_gemv_a8(sb, W, x16):
    y = sb.gemv_a8(W, dev(x16))
    torch.cuda.synchronize()
    return y.cpu().numpy().astype(np.float64)


def selection_sbvr(O, I, k, cols):
    """Planes and coefficients with W_hat[o][cols[o]] = 1 and zero elsewhere:
    plane 0 has the one bit, coefficient 1.0; the other planes are empty."""
    G = I // 128
    planes = np.zeros((O, G, k, 4), dtype=np.uint32)
    coeffs = np.zeros((O, G, k), dtype=np.uint16)
    for o, j in enumerate(cols):
        g, t = divmod(int(j), 128)
        planes[o, g, 0, t // 32] |= np.uint32(1) << np.uint32(t % 32)
        coeffs[o, g, 0] = np.float16(1.0).view(np.uint16)
    return planes, coeffs


@pytest.mark.parametrize("O,I", SHAPES_8B + SHAPES_70B)
def test_a8_full_size_k4(sb, O, I):
    planes, coeffs = synth.random_sbvr(O, I, 4, seed=O + 11 * I)
    x = synth.activations(I, seed=O + 2 * I + synth.X_SEED_OFFSET)
    y = run_gemv_a8(sb, packed(sb, planes, coeffs), x)
    err = rel_err(y, oracle.sbvr_gemv_w4a8(planes, coeffs, x))
    log(f"a8 full {O}x{I} k=4 err={err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("k", [1, 2, 3])
@pytest.mark.parametrize("O,I", [(4096, 4096), (4096, 14336)])
def test_a8_full_size_low_bit(sb, O, I, k):
    planes, coeffs = synth.random_sbvr(O, I, k, seed=O + 11 * I + k)
    x = synth.activations(I, seed=O + 2 * I + k + synth.X_SEED_OFFSET)
    y = run_gemv_a8(sb, packed(sb, planes, coeffs), x)
    err = rel_err(y, oracle.sbvr_gemv_w4a8(planes, coeffs, x))
    log(f"a8 full {O}x{I} k={k} err={err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("O,I,k", [(1, 128, 4), (3, 128, 1), (1001, 640, 3), (7, 896, 4),
                                   (4097, 1152, 2), (33, 2560, 4), (12291, 3968, 4)])
def test_a8_ragged_shapes(sb, O, I, k):
    """Both batch-1 kernels (one-shot for short rows, streaming for long),
    partial tiles and partial gblocks."""
    planes, coeffs = synth.random_sbvr(O, I, k, seed=O + I + k)
    x = synth.activations(I, seed=O * 3 + k)
    y = run_gemv_a8(sb, packed(sb, planes, coeffs), x)
    err = rel_err(y, oracle.sbvr_gemv_w4a8(planes, coeffs, x))
    assert err <= TOL, err


@pytest.mark.parametrize("I", [640, 4096])
def test_a8_codes_through_a_selection_matrix(sb, I):
    """y[o] = s_g q_j for a matrix that selects column j: every output checks
    one 8-bit code and its group scale.  A code off by one moves y by s_g,
    at least 1/127 of |y| -- several binary16 ulps -- so agreement within one
    ulp means every code and scale matches the oracle's.  Groups span normal,
    subnormal, zero and single-element-dominated magnitudes."""
    G = I // 128
    rng = np.random.default_rng(I)
    x = rng.standard_normal(I)
    mags = [1.0, 3e3, 1e-6, 0.0, 6000.0, 0.5, 2.0 ** -20, 7.0]
    for g in range(G):
        x[g * 128:(g + 1) * 128] *= mags[g % len(mags)]
    if G > 5:
        x[5 * 128 + 3] = 65504.0  # one element dominates its group
    x16 = x.astype(np.float16)
    assert np.all(np.isfinite(x16))
    cols = np.arange(I)
    planes, coeffs = selection_sbvr(I, I, 4, cols)
    assert np.array_equal(oracle.decompress(planes, coeffs), np.eye(I))
    y = run_gemv_a8(sb, packed(sb, planes, coeffs), x16)
    q, s = oracle.act_quantize(x16)
    y_ref = q.astype(np.float64) * np.repeat(s.astype(np.float64), 128)
    assert np.array_equal(y_ref, oracle.sbvr_gemv_w4a8(planes, coeffs, x16))
    ulp = fp16_ulp(y_ref.astype(np.float16))
    bad = np.abs(y - y_ref.astype(np.float16).astype(np.float64)) > ulp
    assert not bad.any(), (np.flatnonzero(bad)[:8], y[bad][:8], y_ref[bad][:8])
    # zero groups give exact zeros
    zero_groups = [g for g in range(G) if not np.any(x16[g * 128:(g + 1) * 128])]
    for g in zero_groups:
        assert np.all(y[g * 128:(g + 1) * 128] == 0)


def test_a8_ties_round_to_even(sb):
    """Groups whose maximum is 127 * 2^-7 have s = 2^-7 exactly, so x = m/2^7
    + 1/2^8 lies halfway between two codes: the code is the even one, and
    y = s q is exact in binary16."""
    I = 512
    m = np.arange(-126, 126, dtype=np.float64)
    x = np.concatenate([(m + 0.5) / 128.0, [127 / 128.0, -127 / 128.0]])
    x = np.resize(x, I)
    for g in range(I // 128):  # every group holds its maximum 127/128
        x[g * 128] = 127 / 128.0
    x16 = x.astype(np.float16)
    assert np.array_equal(x16.astype(np.float64), x)
    planes, coeffs = selection_sbvr(I, I, 2, np.arange(I))
    y = run_gemv_a8(sb, packed(sb, planes, coeffs), x16)
    q_even = np.rint(x * 128.0)  # numpy rint: ties to even
    assert np.array_equal(y, q_even / 128.0)


def test_a8_within_quantisation_bound_of_fp16_path(sb):
    """Independent of the oracle's conversion: |x - x_hat| <= s_g / 2 per
    element, so the W4A8 and fp16-activation results differ by at most
    sum_j |W_hat[o][j]| s_g(j) / 2 (plus the two binary16 output roundings)."""
    O, I = 512, 4096
    planes, coeffs = synth.random_sbvr(O, I, 4, seed=77)
    x16 = synth.activations(I, seed=78)
    W = packed(sb, planes, coeffs)
    y8 = run_gemv_a8(sb, W, x16)
    y16 = run_gemv(sb, W, x16)
    What = oracle.decompress(planes, coeffs)
    xg = np.abs(x16.astype(np.float64)).reshape(-1, 128).max(axis=1) / 127.0
    bound = np.abs(What) @ np.repeat(xg, 128) / 2
    slack = fp16_ulp(y8) + fp16_ulp(y16) + 1e-3 * np.abs(y16).max()
    assert np.all(np.abs(y8 - y16) <= bound * (1 + 1e-6) + slack)
    # and the conversion does change the result (the path is not the fp16 one)
    assert not np.array_equal(y8, y16)


def test_a8_error_paths_and_canary(sb):
    O, I = 100, 512
    planes, coeffs = synth.random_sbvr(O, I, 4, seed=5)
    W = packed(sb, planes, coeffs)
    xh = synth.activations(I, seed=6)
    x = dev(xh)
    buf = torch.full((O + 64,), 7.0, dtype=torch.float16, device="cuda")
    st = sb.sbvr_gemv_a8(O, I, 4, W.planes.data_ptr(), W.coeffs.data_ptr(), x.data_ptr(),
                         buf.data_ptr(), None, 0, 0)
    torch.cuda.synchronize()
    assert st == 0
    assert torch.all(buf[O:] == 7.0)
    assert rel_err(buf[:O].cpu().numpy().astype(np.float64),
                   oracle.sbvr_gemv_w4a8(planes, coeffs, xh)) <= TOL
    buf.fill_(5.0)
    torch.cuda.synchronize()
    for args in [(O, I, 5), (O, 100, 4), (0, I, 4)]:
        st = sb.sbvr_gemv_a8(*args, W.planes.data_ptr(), W.coeffs.data_ptr(), x.data_ptr(),
                             buf.data_ptr(), None, 0, 0)
        assert st != 0
    st = sb.sbvr_gemv_a8(O, I, 4, W.planes.data_ptr(), W.coeffs.data_ptr(), x.data_ptr() + 2,
                         buf.data_ptr(), None, 0, 0)
    assert st == sb.SBVR_E_ALIGNMENT
    st = sb.sbvr_gemv_a8(O, I, 4, None, W.coeffs.data_ptr(), x.data_ptr(), buf.data_ptr(), None, 0, 0)
    assert st == sb.SBVR_E_INVALID_ARG
    torch.cuda.synchronize()
    assert torch.all(buf == 5.0)


def test_a8_codes_near_half_integers(sb):
    """Elements whose x / s lies within 2^-12 of a half-integer (found by
    scanning every binary16 value below the group maximum), where a code
    taken from an approximate quotient could differ from the rounded
    correctly-rounded quotient; includes quotients that round in binary32 to
    a half-integer exactly (then ties go to even)."""
    amaxes = [1.0, 0.7001953125, 3.140625, 0.0010004043579101562, 1000.5, 12.34375, 65504.0, 2.0 ** -14]
    all16 = np.arange(1, 0x7c00, dtype=np.uint16).view(np.float16).astype(np.float64)
    groups, n_ties = [], 0
    for a in amaxes:
        a16 = np.float16(a)
        s = np.float32(np.float32(a16) / np.float32(127.0))
        cand = all16[all16 < float(a16)]
        t = cand / float(s)
        near = cand[np.abs(np.abs(t - np.floor(t)) - 0.5) < 2.0 ** -12]
        t32 = (near.astype(np.float32) / s).astype(np.float64)
        n_ties += int(np.sum(t32 - np.floor(t32) == 0.5))
        rng = np.random.default_rng(len(groups))
        pick = rng.permutation(near)[:127] if near.size else near
        g = np.resize(np.concatenate([pick, -pick]) if pick.size else [0.0], 127)
        groups.append(np.concatenate([[float(a16)], g]))
    assert n_ties > 0  # the scan does reach binary32 ties
    x16 = np.concatenate(groups).astype(np.float16)
    I = x16.size
    planes, coeffs = selection_sbvr(I, I, 4, np.arange(I))
    y = run_gemv_a8(sb, packed(sb, planes, coeffs), x16)
    q, s = oracle.act_quantize(x16)
    y_ref = q.astype(np.float64) * np.repeat(s.astype(np.float64), 128)
    ulp = fp16_ulp(y_ref.astype(np.float16))
    bad = np.abs(y - y_ref.astype(np.float16).astype(np.float64)) > ulp
    assert not bad.any(), (np.flatnonzero(bad)[:8], y[bad][:8], y_ref[bad][:8])


# --------------------------------------------------------------------------
# Coefficient-cache format (Sec. 4.4): table of coefficient sets + per-group
# index; reference = oracle.sbvr_gemv_indexed (gathered coefficients)
# --------------------------------------------------------------------------

def packed_indexed(sb, planes, index, table):
    W = sb.pack_indexed(dev(planes.view(np.int32)), dev(index.view(np.int16)), dev(table.view(np.int16)))
    torch.cuda.synchronize()
    return W


def run_gemv_indexed(sb, W, x16, a8=False):
    y = sb.gemv_indexed(W, dev(x16), a8=a8)
    torch.cuda.synchronize()
    return y.cpu().numpy().astype(np.float64)


def cache_sets(O, I):
    """Coefficient sets for an O x I matrix: one per ten groups (an encoder
    cache with a 90 % hit rate), within the 16-bit index."""
    return max(1, min(65536, (O * (I // 128) + 9) // 10))


@pytest.mark.parametrize("O,I,k,N", [(1, 128, 4, 1), (5, 640, 3, 7), (17, 384, 2, 65536), (1000, 1024, 1, 300),
                                     (4096, 4096, 4, 13108), (1024, 14336, 4, 2000), (9, 896, 4, 3)])
def test_pack_indexed_round_trip(sb, O, I, k, N):
    planes, index, table = synth.random_indexed_sbvr(O, I, k, N, seed=O + I + k + N)
    W = packed_indexed(sb, planes, index, table)
    p2, i2, t2 = sb.unpack_indexed(W)
    torch.cuda.synchronize()
    assert np.array_equal(p2.cpu().numpy().view(np.uint32), planes)
    assert np.array_equal(i2.cpu().numpy().view(np.uint16), index)
    assert np.array_equal(t2.cpu().numpy().view(np.uint16), table)
    assert W.index.numel() == sb.sbvr_packed_index_bytes(O, I, k) >= 2 * O * (I // 128)
    assert W.table.numel() == sb.sbvr_packed_table_bytes(N, k) == 8 * N


@pytest.mark.parametrize("O,I", SHAPES_8B + SHAPES_70B)
def test_indexed_full_size_k4(sb, O, I):
    N = cache_sets(O, I)
    planes, index, table = synth.random_indexed_sbvr(O, I, 4, N, seed=O + 13 * I)
    x = synth.activations(I, seed=O + 3 * I + synth.X_SEED_OFFSET)
    y = run_gemv_indexed(sb, packed_indexed(sb, planes, index, table), x)
    err = rel_err(y, oracle.sbvr_gemv_indexed(planes, index, table, x))
    log(f"indexed full {O}x{I} k=4 N={N} err={err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("k", [1, 2, 3])
@pytest.mark.parametrize("O,I", [(4096, 4096), (4096, 14336), (14336, 4096)])
def test_indexed_full_size_low_bit(sb, O, I, k):
    N = cache_sets(O, I)
    planes, index, table = synth.random_indexed_sbvr(O, I, k, N, seed=O + 13 * I + k)
    x = synth.activations(I, seed=O + 3 * I + k + synth.X_SEED_OFFSET)
    y = run_gemv_indexed(sb, packed_indexed(sb, planes, index, table), x)
    err = rel_err(y, oracle.sbvr_gemv_indexed(planes, index, table, x))
    log(f"indexed full {O}x{I} k={k} N={N} err={err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("O,I,k,N", [(1, 128, 4, 1), (3, 128, 1, 2), (1001, 640, 3, 50), (7, 896, 4, 65536),
                                     (4097, 1152, 2, 999), (33, 2560, 4, 5), (1000, 16384, 1, 4000)])
def test_indexed_ragged_shapes(sb, O, I, k, N):
    planes, index, table = synth.random_indexed_sbvr(O, I, k, N, seed=2 * O + I + k)
    x = synth.activations(I, seed=O * 7 + k)
    y = run_gemv_indexed(sb, packed_indexed(sb, planes, index, table), x)
    assert rel_err(y, oracle.sbvr_gemv_indexed(planes, index, table, x)) <= TOL


@pytest.mark.parametrize("O,I,k", [(4096, 4096, 4), (1024, 4096, 2), (14336, 4096, 4), (4096, 14336, 3),
                                   (520, 1920, 1)])
def test_indexed_equals_per_group_bit_for_bit(sb, O, I, k):
    """The same coefficients stored per group (gathered by the oracle) go
    through the same arithmetic: identical binary16 results, for fp16 and
    SBVR-8 activations, one-shot and streaming kernels."""
    N = cache_sets(O, I)
    planes, index, table = synth.random_indexed_sbvr(O, I, k, N, seed=O + I + 5 * k)
    coeffs = oracle.gather_coefficients(index, table)
    x = synth.activations(I, seed=O + 11)
    Wi = packed_indexed(sb, planes, index, table)
    Wp = packed(sb, planes, coeffs)
    assert np.array_equal(run_gemv_indexed(sb, Wi, x), run_gemv(sb, Wp, x))
    assert np.array_equal(run_gemv_indexed(sb, Wi, x, a8=True), run_gemv_a8(sb, Wp, x))


@pytest.mark.parametrize("O,I", [(4096, 4096), (14336, 4096), (4096, 14336)])
def test_indexed_a8_against_oracle(sb, O, I):
    N = cache_sets(O, I)
    planes, index, table = synth.random_indexed_sbvr(O, I, 4, N, seed=O + 2 * I + 1)
    x = synth.activations(I, seed=O + 17)
    y = run_gemv_indexed(sb, packed_indexed(sb, planes, index, table), x, a8=True)
    err = rel_err(y, oracle.sbvr_gemv_w4a8(planes, oracle.gather_coefficients(index, table), x))
    log(f"indexed W4A8 {O}x{I} err={err:.3e}")
    assert err <= TOL


def test_indexed_out_of_range_index_reads_zero(sb):
    """An index past the table is a caller error the library does not fault
    on: those groups decode with zero coefficients."""
    for O, I in [(256, 2048), (14336, 4096)]:
        N = 100
        planes, index, table = synth.random_indexed_sbvr(O, I, 4, N, seed=O)
        bad = index.copy()
        rng = np.random.default_rng(1)
        hit = rng.random(bad.shape) < 0.05
        bad[hit] = rng.integers(N, 65536, size=int(hit.sum()))
        coeffs = oracle.gather_coefficients(np.where(hit, 0, bad), table)
        coeffs[hit] = 0
        x = synth.activations(I, seed=3)
        y = run_gemv_indexed(sb, packed_indexed(sb, planes, bad, table), x)
        assert rel_err(y, oracle.sbvr_gemv(planes, coeffs, x)) <= TOL


def test_indexed_error_paths_and_canary(sb):
    O, I, N = 100, 512, 9
    planes, index, table = synth.random_indexed_sbvr(O, I, 4, N, seed=8)
    W = packed_indexed(sb, planes, index, table)
    xh = synth.activations(I, seed=9)
    x = dev(xh)
    buf = torch.full((O + 64,), 7.0, dtype=torch.float16, device="cuda")
    args = (W.planes.data_ptr(), W.index.data_ptr(), W.table.data_ptr())
    st = sb.sbvr_gemv_indexed(O, I, 4, N, *args, x.data_ptr(), buf.data_ptr(), None, 0, 0)
    torch.cuda.synchronize()
    assert st == 0 and torch.all(buf[O:] == 7.0)
    assert rel_err(buf[:O].cpu().numpy().astype(np.float64), oracle.sbvr_gemv_indexed(planes, index, table, xh)) <= TOL
    buf.fill_(5.0)
    torch.cuda.synchronize()
    for fn in (sb.sbvr_gemv_indexed, sb.sbvr_gemv_indexed_a8):
        for shape in [(O, I, 5, N), (O, 100, 4, N), (0, I, 4, N), (O, I, 4, 0), (O, I, 4, 65537)]:
            assert fn(*shape, *args, x.data_ptr(), buf.data_ptr(), None, 0, 0) != 0
        assert fn(O, I, 4, N, *args, x.data_ptr() + 2, buf.data_ptr(), None, 0, 0) == sb.SBVR_E_ALIGNMENT
        assert fn(O, I, 4, N, args[0], args[1] + 2, args[2], x.data_ptr(), buf.data_ptr(), None, 0, 0) \
            == sb.SBVR_E_ALIGNMENT
        assert fn(O, I, 4, N, args[0], None, args[2], x.data_ptr(), buf.data_ptr(), None, 0, 0) \
            == sb.SBVR_E_INVALID_ARG
    torch.cuda.synchronize()
    assert torch.all(buf == 5.0)
    assert sb.sbvr_packed_table_bytes(N, 4) == 8 * N and sb.sbvr_packed_table_bytes(0, 4) == 0
    assert sb.sbvr_packed_table_bytes(65537, 4) == 0


@pytest.mark.parametrize("O,I,k,N", [(1, 128, 4, 1), (1001, 640, 3, 50), (4097, 1152, 2, 999), (33, 2560, 1, 7),
                                     (4096, 4096, 4, 13108), (14336, 2560, 3, 5000)])
def test_decompress_indexed_bit_exact(sb, O, I, k, N):
    """Prefill decompression of the cache format: bit-exact against rounding
    the oracle's exact decoding of the gathered coefficients, and identical to
    the per-group decompression of the same coefficients; indices past the
    table decode with zero coefficients."""
    planes, index, table = synth.random_indexed_sbvr(O, I, k, N, seed=3 * O + I + k)
    rng = np.random.default_rng(O)
    bad = rng.random(index.shape) < 0.02
    index = index.copy()
    index[bad] = N + rng.integers(0, 65536 - N, size=int(bad.sum())) if N < 65536 else index[bad]
    coeffs = oracle.gather_coefficients(np.where(bad, 0, index), table)
    coeffs[bad] = 0
    Wi = packed_indexed(sb, planes, index, table)
    M = sb.decompress(Wi)
    torch.cuda.synchronize()
    got = M.cpu().numpy().view(np.uint16)
    assert np.array_equal(got, oracle_fp16(planes, coeffs))
    Mp = sb.decompress(packed(sb, planes, coeffs))
    torch.cuda.synchronize()
    assert np.array_equal(got, Mp.cpu().numpy().view(np.uint16))


def test_largest_accepted_shape_sampled_rows(sb):
    """O * I just below 2^31 (the largest shape the library accepts; 1.2 GB of
    packed weights, 256 gblocks per row): batch 1, W4A8 and B = 8 against the
    oracle on sampled rows, including the first and last."""
    O, I, k = 16383, 131072, 4
    assert O * I < 2 ** 31 - 1
    planes, coeffs = synth.random_sbvr(O, I, k, seed=2024)
    W = packed(sb, planes, coeffs)
    rows = np.unique(np.r_[0, 1, O - 2, O - 1, np.random.default_rng(0).integers(0, O, 44)])
    x = synth.activations(I, seed=2025)
    y = run_gemv(sb, W, x)
    assert rel_err(y[rows], oracle.sbvr_gemv(planes, coeffs, x, rows=rows)) <= TOL
    y8 = run_gemv_a8(sb, W, x)
    assert rel_err(y8[rows], oracle.sbvr_gemv_w4a8(planes, coeffs, x, rows=rows)) <= TOL
    X = synth.activations(I, seed=2026, batch=8)
    Y = run_gemm(sb, W, X)
    Y_ref = oracle.sbvr_gemv(planes, coeffs, X, rows=rows)
    assert max(rel_err(Y[b][rows], Y_ref[b]) for b in range(8)) <= TOL
    log(f"largest shape {O}x{I}: sampled rows within {TOL}")

@pytest.mark.parametrize("O,I,k", [(262143, 8192, 4), (524287, 4096, 4), (262143, 8192, 1)])
def test_tallest_accepted_shapes_sampled_rows(sb, O, I, k):
    """O * I just below 2^31 with short rows: the streaming kernel's tiles per
    workgroup are capped by the dynamic LDS its per-tile row sums take
    (16 wavefronts at I = 8192, the depth-4 launch of 256 workgroups at
    I = 4096, 16-row tiles at k = 1), so these launches use more workgroups;
    batch 1 and W4A8 against the oracle on sampled rows, first and last
    included."""
    assert O * I < 2 ** 31 - 1
    planes, coeffs = synth.random_sbvr(O, I, k, seed=O + k)
    W = packed(sb, planes, coeffs)
    rows = np.unique(np.r_[0, 1, O - 2, O - 1, np.random.default_rng(1).integers(0, O, 44)])
    x = synth.activations(I, seed=O + 7)
    y = run_gemv(sb, W, x)
    assert rel_err(y[rows], oracle.sbvr_gemv(planes, coeffs, x, rows=rows)) <= TOL
    y8 = run_gemv_a8(sb, W, x)
    assert rel_err(y8[rows], oracle.sbvr_gemv_w4a8(planes, coeffs, x, rows=rows)) <= TOL
    log(f"tall shape {O}x{I} k={k}: sampled rows within {TOL}")

@pytest.mark.parametrize("O,I", [(4096, 4096), (14336, 4096), (4096, 14336)])
def test_repeated_calls_are_bit_identical(sb, O, I):
    """Each kernel reduces in a fixed order, so repeated calls on the same
    inputs give the same bits: the one-shot kernel (4096 x 4096), the
    streaming kernel with one gblock per wavefront (14336 x 4096) and with
    several (4096 x 14336), for fp16 and SBVR-8 activations and a 5-vector
    small batch."""
    planes, coeffs = synth.random_sbvr(O, I, 4, seed=O + 3 * I)
    W = packed(sb, planes, coeffs)
    x = synth.activations(I, seed=O + 5)
    X = synth.activations(I, seed=O + 6, batch=5)
    first = (run_gemv(sb, W, x), run_gemv_a8(sb, W, x), run_gemm(sb, W, X))
    for _ in range(3):
        again = (run_gemv(sb, W, x), run_gemv_a8(sb, W, x), run_gemm(sb, W, X))
        for a, b in zip(first, again):
            assert np.array_equal(a.view(np.uint64), b.view(np.uint64))  # exact binary16 values as float64
