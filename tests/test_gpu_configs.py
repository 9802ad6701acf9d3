"""The benchmark configurations' own weights, encoded at full size, through
every decode entry point, and the decode-step graph, against the oracle.

Weights follow the configurations: Llama-3-8B projection shapes from
N(0, 0.02^2) with 0.1 % outliers at +-8 sigma (k = 4, 3, 2), Llama-3-70B
shapes from N(0, 0.015^2) (k = 4); activations N(0, 1) in binary16.  Each
matrix is encoded whole by the GPU encoder (sbvr_encode).  The oracle never
takes a GPU result as its input: it encodes a sample of rows itself (the
first, the last and random ones), the GPU encoding of those rows must equal
it bit for bit, and the oracle's GEMV of its own encoding of those rows is
the reference for the GPU outputs on the same rows, with the gate
max|y - y_ref| / max|y_ref| <= 1e-3 over the sampled rows, per vector.
"""
import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = 1e-3
N_ROWS = 64


@pytest.fixture(scope="module")
def sb():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2509_18172_amd as m
    return m


def log(msg):
    print(msg, flush=True)


def rel_err(y, y_ref):
    y = np.asarray(y, dtype=np.float64)
    den = np.abs(y_ref).max()
    return float(np.abs(y - y_ref).max() / den) if den > 0 else float(np.abs(y).max())


def sample_rows(O, seed):
    rng = np.random.default_rng(seed)
    mid = rng.choice(np.arange(1, O - 1), size=min(N_ROWS - 2, O - 2), replace=False)
    return np.unique(np.r_[0, mid, O - 1]).astype(np.int64)


def encode_checked(sb, W, k, rows):
    """GPU-encode the whole matrix and pack it; return (packed weight, the
    oracle's own planes and coefficients of `rows`), after checking that the
    GPU encoding of those rows is the oracle's bit for bit."""
    Wd = torch.from_numpy(np.ascontiguousarray(W)).cuda()
    planes, coeffs = sb.encode(Wd, k)
    packed = sb.pack(planes, coeffs)
    p_rows = planes[torch.from_numpy(rows).cuda()].cpu().numpy().view(np.uint32)
    c_rows = coeffs[torch.from_numpy(rows).cuda()].cpu().numpy().view(np.uint16)
    del Wd, planes, coeffs
    p_ref, c_ref = oracle.encode_matrix(W[rows], k)
    assert np.array_equal(p_rows, p_ref), "GPU planes differ from the oracle's on the sampled rows"
    assert np.array_equal(c_rows, c_ref), "GPU coefficients differ from the oracle's on the sampled rows"
    return packed, p_ref, c_ref


def check_decode_paths(sb, packed, p_ref, c_ref, rows, I, seed, batches, a8=True, what=""):
    rows_t = torch.from_numpy(rows).cuda()
    X = synth.activations(I, seed=seed + synth.X_SEED_OFFSET, batch=max(batches + (1,)))
    y = sb.gemv(packed, torch.from_numpy(X[0]).cuda())[rows_t].cpu().numpy()
    errs = {"B=1": rel_err(y, oracle.sbvr_gemv(p_ref, c_ref, X[0]))}
    if a8:
        y8 = sb.gemv_a8(packed, torch.from_numpy(X[0]).cuda())[rows_t].cpu().numpy()
        errs["W4A8"] = rel_err(y8, oracle.sbvr_gemv_w4a8(p_ref, c_ref, X[0]))
    for B in batches:
        Y = sb.gemm_small_batch(packed, torch.from_numpy(X[:B]).cuda())[:, rows_t].cpu().numpy()
        Y_ref = oracle.sbvr_gemv(p_ref, c_ref, X[:B])
        errs[f"B={B}"] = max(rel_err(Y[b], Y_ref[b]) for b in range(B))
    log(f"{what}: " + " ".join(f"{n} {e:.3e}" for n, e in errs.items()))
    for n, e in errs.items():
        assert e <= TOL, (what, n, e)


@pytest.mark.parametrize("proj", ["q", "k", "gate", "down"])
def test_llama8b_encoded_full_size(sb, proj):
    """Llama-3-8B shapes with outliers: k = 4 through sbvr_gemv, sbvr_gemv_a8
    and sbvr_gemm_small_batch (B = 2, 4, 8); k = 3 and 2 through sbvr_gemv and
    B = 8."""
    O, I = synth.LLAMA8B[proj]
    seed = synth.seed_for(1, 0, synth.PROJ[proj])
    W = synth.weights(O, I, 0.02, seed=seed, outlier_frac=0.001)
    rows = sample_rows(O, seed)
    for k in (4, 3, 2):
        packed, p_ref, c_ref = encode_checked(sb, W, k, rows)
        check_decode_paths(sb, packed, p_ref, c_ref, rows, I, seed + k,
                           (2, 4, 8) if k == 4 else (8,), a8=(k == 4), what=f"8B {proj} {O}x{I} k={k}")
        del packed
        torch.cuda.empty_cache()


@pytest.mark.parametrize("proj", ["q", "k", "gate", "down"])
def test_llama70b_encoded_full_size(sb, proj):
    """Llama-3-70B shapes, N(0, 0.015^2), k = 4: sbvr_gemv, sbvr_gemv_a8 and
    sbvr_gemm_small_batch (B = 2, 8)."""
    O, I = synth.LLAMA70B[proj]
    seed = synth.seed_for(3, 0, synth.PROJ[proj])
    W = synth.weights(O, I, 0.015, seed=seed)
    rows = sample_rows(O, seed)
    packed, p_ref, c_ref = encode_checked(sb, W, 4, rows)
    del W
    check_decode_paths(sb, packed, p_ref, c_ref, rows, I, seed, (2, 8), what=f"70B {proj} {O}x{I} k=4")


def test_decode_step_graph_against_oracle(sb):
    """Two Llama-3-8B decoder layers (14 GEMVs, weights encoded from
    independently seeded N(0, 0.02^2) matrices) and one Llama-3-70B layer (7
    GEMVs, SBVR tensors drawn directly) captured in one HIP graph on one
    stream, issued the way the benchmark issues its decode step
    (sbvr_gemv with preallocated outputs).  After three replays (with eager
    work between them) every output is checked against the oracle on sampled
    rows, first and last included, and each replay must give the same bits.
    The same GEMVs captured as grouped launches (q|k|v and gate|up of each
    layer in one launch) must reproduce those bits."""
    stream = torch.cuda.Stream()
    calls, refs = [], []
    for layer in range(2):
        for name in synth.PROJ:
            O, I = synth.LLAMA8B[name]
            seed = synth.seed_for(4, layer, synth.PROJ[name])
            W = synth.weights(O, I, 0.02, seed=seed)
            rows = sample_rows(O, seed)
            packed, p_ref, c_ref = encode_checked(sb, W, 4, rows)
            del W
            x = synth.activations(I, seed=seed + synth.X_SEED_OFFSET)
            calls.append((packed, torch.from_numpy(x).cuda(), torch.empty(O, dtype=torch.float16, device="cuda")))
            refs.append((f"8B layer {layer} {name}", rows, oracle.sbvr_gemv(p_ref, c_ref, x)))
    for name in synth.PROJ:
        O, I = synth.LLAMA70B[name]
        seed = synth.seed_for(3, 1, synth.PROJ[name])
        planes, coeffs = synth.random_sbvr(O, I, 4, seed=seed)
        rows = sample_rows(O, seed)
        packed = sb.pack(torch.from_numpy(planes.view(np.int32)).cuda(), torch.from_numpy(coeffs.view(np.int16)).cuda())
        x = synth.activations(I, seed=seed + synth.X_SEED_OFFSET)
        calls.append((packed, torch.from_numpy(x).cuda(), torch.empty(O, dtype=torch.float16, device="cuda")))
        refs.append((f"70B {name}", rows, oracle.sbvr_gemv(planes[rows], coeffs[rows], x)))
        del planes, coeffs
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):  # eager warm-up of every shape before capture
        for W, x, y in calls:
            sb.gemv(W, x, out=y, stream=stream)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        for W, x, y in calls:
            sb.gemv(W, x, out=y, stream=stream)
    first = None
    for rep in range(3):
        for _, _, y in calls:
            y.fill_(float("nan"))  # eager work between replays; every output must be rewritten
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        outs = [y.cpu().numpy().view(np.uint16).copy() for _, _, y in calls]
        if first is None:
            first = outs
        else:
            assert all(np.array_equal(a, b) for a, b in zip(first, outs)), f"replay {rep} changed bits"
    worst = 0.0
    for (what, rows, y_ref), out in zip(refs, first):
        e = rel_err(out.view(np.float16)[rows], y_ref)
        worst = max(worst, e)
        assert e <= TOL, (what, e)
    log(f"decode graph: {len(calls)} GEMVs in one graph, 3 replays identical, worst sampled err {worst:.3e}")

    # the same 21 GEMVs as the grouped decode step issues them (q|k|v and
    # gate|up of each layer as one sbvr_gemv_grouped launch, 12 launches): the
    # graph's outputs must be the bits checked above
    names = list(synth.PROJ)
    groups = [("q", "k", "v"), ("o",), ("gate", "up"), ("down",)]
    launches = []
    for base in (0, 7, 14):
        for grp in groups:
            launches.append([calls[base + names.index(n)] for n in grp])
    g2 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g2, stream=stream):
        for members in launches:
            sb.gemv_grouped([m[0] for m in members], [m[1] for m in members], outs=[m[2] for m in members],
                            stream=stream)
    for rep in range(2):
        for _, _, y in calls:
            y.fill_(float("nan"))
        torch.cuda.synchronize()
        g2.replay()
        torch.cuda.synchronize()
        for (what, _, _), (_, _, y), want in zip(refs, calls, first):
            assert np.array_equal(y.cpu().numpy().view(np.uint16), want), (what, rep)
    log(f"grouped decode graph: {len(launches)} launches, the same bits on 2 replays")
