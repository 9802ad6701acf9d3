"""The seeded input generator: chunked Box-Muller equals its one-pass
definition (u1 from words [0, m), u2 from words [m, 2m) of the stream), and
the stream continues after the 2m words (the outlier draws depend on it)."""
import numpy as np

import synth


def one_pass_normal(seed, n):
    bg = np.random.PCG64(seed)
    m = (n + 1) // 2
    r = np.asarray(bg.random_raw(2 * m), dtype=np.uint64)
    u1 = 1.0 - (r[:m] >> np.uint64(11)).astype(np.float64) / 2.0 ** 53
    u2 = (r[m:] >> np.uint64(11)).astype(np.float64) / 2.0 ** 53
    rad = np.sqrt(-2.0 * np.log(u1))
    z = np.empty(2 * m)
    z[0::2] = rad * np.cos(2.0 * np.pi * u2)
    z[1::2] = rad * np.sin(2.0 * np.pi * u2)
    return z[:n], bg


def test_chunked_normals_match_the_one_pass_definition():
    for n, chunk in ((1, 1), (2, 1), (101, 7), (1000, 64), (4097, 4096)):
        want, bg = one_pass_normal(31 + n, n)
        st = synth.Stream(31 + n)
        m = (n + 1) // 2
        z = np.empty(2 * m)
        for a, zc, zs in st._pairs(m, chunk):
            z[2 * a:2 * (a + zc.size):2] = zc
            z[2 * a + 1:2 * (a + zc.size):2] = zs
        assert np.array_equal(z[:n], want), (n, chunk)
        assert np.array_equal(st.raw(3), np.asarray(bg.random_raw(3), dtype=np.uint64)), (n, chunk)


def test_weights_are_fp32_of_scaled_normals_plus_outliers():
    O, I, sigma = 9, 384, 0.02
    W = synth.weights(O, I, sigma, seed=5, outlier_frac=0.01)
    z, _ = one_pass_normal(5, O * I)
    plain = (sigma * z).astype(np.float32).reshape(O, I)
    out = W != plain
    assert out.sum() == round(0.01 * O * I)
    assert np.all(np.abs(W[out]) == np.float32(8 * sigma))
