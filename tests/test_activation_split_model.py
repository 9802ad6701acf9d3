"""Host-side model of the activation split the GPU kernels use for binary16
activations, checked against the error bound the kernels' documentation
states (no GPU needed).

The kernels scale a 512-element block by 2^(sigma + inv_alpha) in binary16
(sigma = min(14 - e, 29) for a block maximum in [2^(e-1), 2^e); inv_alpha in
{1, 0, -1}; two exact power-of-two products), cut the result three times to
two mantissa bits (mask 0xFF00) and keep the top byte of each piece, which is
read as an E5M2 number.  This
model does the same steps with numpy's binary16 arithmetic (each operation
rounded to nearest, the IEEE rule the GPU's binary16 instructions follow) and
checks, over every finite binary16 value below a block maximum:
  - the four bytes decode to x * 2^(sigma + inv_alpha) exactly whenever
    |x| >= 2^-18 * max;
  - otherwise the error is below 2^-27 * max (in x units).
"""
import numpy as np
import pytest

ALL = np.arange(0x10000, dtype=np.uint32).astype(np.uint16)
FINITE = ALL[(ALL & 0x7C00) != 0x7C00].view(np.float16)


def scale_exponent(amax):
    if amax == 0:
        return 0
    _, e = np.frexp(np.float64(amax))
    return min(14 - int(e), 29)


def pow2_h(e):
    assert -14 <= e <= 15
    return np.float16(2.0 ** e)


def split_model(x, sigma, inv_alpha):
    """x: float16 array -> (x', four uint8 limb arrays) as the kernels do it."""
    s0 = min(sigma, 14)
    w = (x * pow2_h(s0 + inv_alpha)).astype(np.float16)
    w = (w * pow2_h(sigma - s0)).astype(np.float16)
    pieces = []
    r = w
    for _ in range(3):
        p = (r.view(np.uint16) & np.uint16(0xFF00)).view(np.float16)
        pieces.append(p)
        r = (r - p).astype(np.float16)
    pieces.append(r)
    return w, [(p.view(np.uint16) >> 8).astype(np.uint8) for p in pieces]


def e5m2_value(byte):
    """E5M2 (sign, 5 exponent bits with bias 15, 2 mantissa bits; subnormals
    below 2^-14) read by its definition, in binary64."""
    b = byte.astype(np.int64)
    sign = np.where(b & 0x80, -1.0, 1.0)
    ex = (b >> 2) & 0x1F
    man = b & 3
    val = np.where(ex == 0, man / 4.0 * 2.0 ** -14, (1 + man / 4.0) * 2.0 ** (ex - 15.0))
    assert not np.any(ex == 0x1F), "a limb must never be Inf/NaN"
    return sign * val


@pytest.mark.parametrize("amax", [65504.0, 3.75, 1.0, 0.4, 2.0 ** -14, 3e-5, 1e-6, 2.0 ** -24])
@pytest.mark.parametrize("inv_alpha", [1, 0, -1])
def test_split_is_exact_above_the_stated_floor(amax, inv_alpha):
    amax = float(np.float16(amax))
    sigma = scale_exponent(amax)
    x = FINITE[np.abs(FINITE.astype(np.float64)) <= amax]
    w, limbs = split_model(x, sigma, inv_alpha)
    recon = sum(e5m2_value(l) for l in limbs)
    exact = x.astype(np.float64) * 2.0 ** (sigma + inv_alpha)
    # every limb fits the E5M2 range the matrix-core operand takes
    assert np.abs(recon).max() < 57344
    big = np.abs(x.astype(np.float64)) >= 2.0 ** -18 * amax
    assert np.array_equal(recon[big], exact[big]), (amax, inv_alpha)
    err_x = np.abs(recon - exact) / 2.0 ** (sigma + inv_alpha)
    assert err_x.max() < 2.0 ** -27 * amax, (amax, inv_alpha, err_x.max() / amax)


def test_split_pieces_are_top_bytes():
    """Each piece the cut leaves has a zero low byte whenever its bits lie at
    or above 2^-16 (that is what lets the top byte stand for it)."""
    sigma = scale_exponent(1.0)
    x = FINITE[np.abs(FINITE.astype(np.float64)) <= 1.0]
    w, limbs = split_model(x, sigma, 0)
    s = np.abs(w.astype(np.float64)) >= 2.0 ** -6
    r = w[s]
    for _ in range(3):
        p = (r.view(np.uint16) & np.uint16(0xFF00)).view(np.float16)
        r = (r - p).astype(np.float16)
    assert np.all((r.view(np.uint16) & 0xFF) == 0)
