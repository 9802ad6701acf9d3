"""Seeded synthetic inputs shared by the tests, the smoke check and the bench.

This module holds none of the SBVR arithmetic: it only draws numbers.

* Uniform and normal variates come from numpy's PCG64 bit generator (its raw
  64-bit stream is fixed by the PCG64 definition) through a Box-Muller
  transform written here, so a seed names the same bytes on every machine.
* Weight matrices model decode-stage LLM linear layers: N(0, sigma^2) in
  fp32, optionally with a fraction of outliers at exactly +-8 sigma placed at
  distinct positions chosen by a partial Fisher-Yates shuffle.
* Activations are N(0, 1) rounded to fp16.
* ``random_sbvr`` draws SBVR-format tensors directly (uniform bit planes,
  fp16 coefficients ~ N(0, sigma_c^2)); they stand in for encoded weights
  where running the encoder would take too long (full-size parity, bench).

Seed convention: seed(config, layer, proj) = 1000*config + 16*layer + proj;
activations use the weight seed + 500000.
"""
from __future__ import annotations

import numpy as np

GROUP = 128
X_SEED_OFFSET = 500_000

# projection index within a decoder layer
PROJ = {"q": 0, "k": 1, "v": 2, "o": 3, "gate": 4, "up": 5, "down": 6}


def seed_for(config: int, layer: int = 0, proj: int = 0) -> int:
    return 1000 * config + 16 * layer + proj


CHUNK = 1 << 20  # Box-Muller pairs per chunk


class Stream:
    """Counter-free stream of raw 64-bit words from PCG64(seed)."""

    def __init__(self, seed: int):
        self._bg = np.random.PCG64(int(seed))

    def raw(self, n: int) -> np.ndarray:
        return np.asarray(self._bg.random_raw(int(n)), dtype=np.uint64)

    @staticmethod
    def _unit(r: np.ndarray) -> np.ndarray:
        """Doubles in [0, 1) from the top 53 bits of raw words."""
        return (r >> np.uint64(11)).astype(np.float64) * (1.0 / 9007199254740992.0)

    def uniform01(self, n: int) -> np.ndarray:
        """Doubles in [0, 1) from the top 53 bits of each raw word."""
        return self._unit(self.raw(n))

    def _pairs(self, m: int, chunk: int = CHUNK):
        """Box-Muller over the next 2m raw words: pair i takes u1 = 1 - unit
        of word i and u2 = unit of word m + i.  Yields (first pair, rad*cos,
        rad*sin) chunk by chunk (bounded temporaries) and leaves the stream
        after the 2m words."""
        g1 = self._bg
        g2 = np.random.PCG64()
        g2.state = g1.state
        g2.advance(m)
        for a in range(0, m, chunk):
            c = min(chunk, m - a)
            u1 = 1.0 - self._unit(np.asarray(g1.random_raw(c), dtype=np.uint64))  # (0, 1]
            u2 = self._unit(np.asarray(g2.random_raw(c), dtype=np.uint64))
            rad = np.sqrt(-2.0 * np.log(u1))
            yield a, rad * np.cos(2.0 * np.pi * u2), rad * np.sin(2.0 * np.pi * u2)
        g1.advance(m)

    def normal(self, n: int) -> np.ndarray:
        """Standard normals by Box-Muller, two per pair of uniforms: z[2i] and
        z[2i+1] from words i and m + i of the next 2m = 2 ceil(n/2) words."""
        m = (int(n) + 1) // 2
        z = np.empty(2 * m)
        for a, zc, zs in self._pairs(m):
            z[2 * a:2 * (a + zc.size):2] = zc
            z[2 * a + 1:2 * (a + zc.size):2] = zs
        return z[:n]

    def below(self, bound: int) -> int:
        """Integer in [0, bound) from one raw word (multiply-shift)."""
        r = int(self.raw(1)[0])
        return (r * int(bound)) >> 64


def weights(O: int, I: int, sigma: float, seed: int, outlier_frac: float = 0.0) -> np.ndarray:
    """fp32 [O][I] weights: fp32(sigma * z), plus round(frac*O*I) outliers at +-8 sigma."""
    st = Stream(seed)
    n = O * I
    W = np.empty(n + (n & 1), dtype=np.float32)  # fp32(sigma * z), z = st.normal(n)
    for a, zc, zs in st._pairs((n + 1) // 2):
        W[2 * a:2 * (a + zc.size):2] = (sigma * zc).astype(np.float32)
        W[2 * a + 1:2 * (a + zc.size):2] = (sigma * zs).astype(np.float32)
    W = W[:n]
    n_out = int(round(outlier_frac * O * I))
    if n_out:
        total = O * I
        swapped: dict[int, int] = {}
        pos = np.empty(n_out, dtype=np.int64)
        for t in range(n_out):  # partial Fisher-Yates over [0, total)
            j = t + st.below(total - t)
            vt, vj = swapped.get(t, t), swapped.get(j, j)
            swapped[t], swapped[j] = vj, vt
            pos[t] = vj
        signs = np.where((st.raw(n_out) & np.uint64(1)) == 1, 1.0, -1.0)
        W.reshape(-1)[pos] = (signs * 8.0 * sigma).astype(np.float32)
    return W.reshape(O, I)


def activations(I: int, seed: int, batch: int | None = None, scale: float = 1.0) -> np.ndarray:
    """fp16 activations ~ N(0, scale^2), shape [I] or [batch][I]."""
    n = I if batch is None else batch * I
    x = (scale * Stream(seed).normal(n)).astype(np.float16)
    return x if batch is None else x.reshape(batch, I)


def random_sbvr(O: int, I: int, K: int, seed: int, coeff_sigma: float = 0.01):
    """Canonical SBVR tensors drawn directly: planes uint32 [O][G][K][4]
    (uniform bits) and coeffs uint16 [O][G][K] (fp16 of N(0, coeff_sigma^2))."""
    G = I // GROUP
    st = Stream(seed)
    raw = st.raw((O * G * K * 4 + 1) // 2)
    planes = raw.view(np.uint32)[: O * G * K * 4].reshape(O, G, K, 4).copy()
    coeffs = (coeff_sigma * st.normal(O * G * K)).astype(np.float16).view(np.uint16)
    return planes, coeffs.reshape(O, G, K).copy()


def random_indexed_sbvr(O: int, I: int, K: int, n_sets: int, seed: int, coeff_sigma: float = 0.01):
    """Coefficient-cache SBVR tensors drawn directly: planes uint32 [O][G][K][4]
    (uniform bits), a table uint16 [n_sets][K] of coefficient sets (fp16 of
    N(0, coeff_sigma^2)) and index uint16 [O][G], uniform in [0, n_sets)
    (multiply-shift of a raw 32-bit word)."""
    assert 1 <= n_sets <= 65536
    G = I // GROUP
    st = Stream(seed)
    raw = st.raw((O * G * K * 4 + 1) // 2)
    planes = raw.view(np.uint32)[: O * G * K * 4].reshape(O, G, K, 4).copy()
    table = (coeff_sigma * st.normal(n_sets * K)).astype(np.float16).view(np.uint16).reshape(n_sets, K).copy()
    r32 = st.raw((O * G + 1) // 2).view(np.uint32)[: O * G].astype(np.uint64)
    index = ((r32 * np.uint64(n_sets)) >> np.uint64(32)).astype(np.uint16).reshape(O, G)
    return planes, index, table


# Decode-projection shapes (out x in) of the Llama-3-8B / 70B decoder layers.
LLAMA8B = {"q": (4096, 4096), "k": (1024, 4096), "v": (1024, 4096), "o": (4096, 4096),
           "gate": (14336, 4096), "up": (14336, 4096), "down": (4096, 14336)}
LLAMA70B = {"q": (8192, 8192), "k": (1024, 8192), "v": (1024, 8192), "o": (8192, 8192),
            "gate": (28672, 8192), "up": (28672, 8192), "down": (8192, 28672)}
