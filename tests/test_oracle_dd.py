"""Pins of the data-dependent-filter oracle (Alg. 5; oracle/dd.py) -- CPU only.

The tiling against the plain definition sum_{j+k=t} y_j rho_k, against the
closed form of two geometric sequences, against causality, and by counting:
every pair (j, k) with j + k < L is covered exactly once, each tile reads
only positions already revealed and writes only later ones.  The variant
printed in Alg. 5 (only the largest U per step) is shown to miss pairs,
which is why the oracle takes every U.
"""
import numpy as np
import pytest

from oracle.dd import dd_tiles_after_step, product_naive, relaxed_dd


def _pairs(L, tiles_fn):
    """Coverage count of every pair (j, k), j + k < L: red cells and tiles."""
    cnt = np.zeros((L, L), dtype=np.int64)
    cnt[0, 0] += 1
    for t in range(1, L):
        cnt[t, 0] += 1
        cnt[0, t] += 1
    for t in range(L):
        for kind, U, lo, d0, d1 in tiles_fn(t, L):
            assert lo + U - 1 <= t and U + U - 1 <= t     # inputs already revealed
            assert d0 >= t + 1                            # outputs not yet emitted
            fixed = range(U, 2 * U)
            recent = range(lo, lo + U)
            blocks = [(fixed, fixed)] if kind == "square" else [(fixed, recent), (recent, fixed)]
            for js, ks in blocks:
                for j in js:
                    for k in ks:
                        if j + k < L:
                            assert d0 <= j + k < d1
                            cnt[j, k] += 1
    return cnt


@pytest.mark.parametrize("L", [1, 2, 3, 5, 8, 16, 37, 64, 100, 256])
def test_every_pair_covered_exactly_once(L):
    cnt = _pairs(L, dd_tiles_after_step)
    j, k = np.indices((L, L))
    assert np.array_equal(cnt[j + k < L], np.ones(int((j + k < L).sum()), dtype=np.int64))
    assert cnt[j + k >= L].sum() == 0


def _largest_u_only(t, L):
    """Alg. 5 as printed: one U per step, the largest power of two dividing t+1."""
    i1 = t + 1
    U = i1 & -i1
    if i1 == U:
        if U < 2:
            return []
        U //= 2
        d0 = 2 * U
        return [("square", U, U, d0, min(d0 + 2 * U - 1, L))] if d0 < L else []
    d0 = t + 1
    return [("rect", U, t - U + 1, d0, min(d0 + 2 * U - 1, L))] if d0 < L else []


def test_largest_u_only_misses_pairs():
    cnt = _pairs(16, _largest_u_only)
    assert cnt[1, 3] == 0 and cnt[3, 1] == 0      # y_1 rho_3, y_3 rho_1 (z_4)
    assert (cnt[np.add.outer(np.arange(16), np.arange(16)) < 16] == 0).sum() > 0


def test_tiles_of_a_few_steps():
    assert dd_tiles_after_step(0, 100) == []
    assert dd_tiles_after_step(1, 100) == [("square", 1, 1, 2, 3)]
    assert dd_tiles_after_step(2, 100) == [("rect", 1, 2, 3, 4)]
    assert dd_tiles_after_step(3, 100) == [("rect", 1, 3, 4, 5), ("square", 2, 2, 4, 7)]
    assert dd_tiles_after_step(7, 100) == [("rect", 1, 7, 8, 9), ("rect", 2, 6, 8, 11),
                                           ("square", 4, 4, 8, 15)]
    assert dd_tiles_after_step(11, 100) == [("rect", 1, 11, 12, 13), ("rect", 2, 10, 12, 15),
                                            ("rect", 4, 8, 12, 19)]
    assert dd_tiles_after_step(7, 10) == [("rect", 1, 7, 8, 9), ("rect", 2, 6, 8, 10),
                                          ("square", 4, 4, 8, 10)]


@pytest.mark.parametrize("L", [1, 2, 3, 17, 64, 100, 257])
def test_matches_the_definition(L):
    rng = np.random.default_rng(L)
    y = rng.normal(size=(L, 3))
    rho = rng.normal(size=(L, 3))
    z = relaxed_dd(y, rho)
    assert np.allclose(z, product_naive(y, rho), atol=1e-11, rtol=0)
    for c in range(3):
        assert np.allclose(z[:, c], np.convolve(y[:, c], rho[:, c])[:L], atol=1e-11, rtol=0)


def test_geometric_closed_form():
    """y_j = a^j, rho_k = b^k: z_t = (a^{t+1} - b^{t+1}) / (a - b)."""
    L = 200
    a, b = 0.97, -0.9
    t = np.arange(L)
    z = relaxed_dd(a ** t[:, None], b ** t[:, None])[:, 0]
    assert np.allclose(z, (a ** (t + 1) - b ** (t + 1)) / (a - b), atol=1e-12, rtol=0)


def test_causality():
    L, t0 = 130, 77
    rng = np.random.default_rng(5)
    y, rho = rng.normal(size=(L, 2)), rng.normal(size=(L, 2))
    y2, rho2 = y.copy(), rho.copy()
    y2[t0 + 1:] += 3.0
    rho2[t0 + 1:] -= 2.0
    z1, z2 = relaxed_dd(y, rho), relaxed_dd(y2, rho2)
    assert np.array_equal(z1[: t0 + 1], z2[: t0 + 1])
    assert not np.allclose(z1[t0 + 1:], z2[t0 + 1:])


def test_fixed_filter_is_the_ordinary_convolution():
    """A rho that does not depend on the data is the data-independent case."""
    L = 300
    rng = np.random.default_rng(8)
    y = rng.normal(size=(L, 4))
    h = rng.normal(size=(L, 4)) * np.exp(-np.arange(L) / 50.0)[:, None]
    from oracle import conv
    assert np.allclose(relaxed_dd(y, h), conv.causal_conv_naive(y, h), atol=1e-11, rtol=0)
