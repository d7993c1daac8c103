"""Pins of the CPU oracle against what the paper and mathematics fix -- CPU only.

The oracle is checked against library routines it does not use (np.convolve,
np.cumsum), hand-computed values, closed forms of the geometric filter, brute
force on tiny inputs, exact integer arithmetic and invariants (causality,
exactly-once coverage).  A few tests plant plausible mistakes in copies of
oracle functions and check that the pins catch them.
"""
import os

import numpy as np
import pytest

from oracle import conv, feedback, relaxed
from oracle.relaxed import filters_to_columns, lazy_online, relaxed_online

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _hand_cases():
    rows = []
    with open(os.path.join(GOLDEN, "conv_hand.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(np.array([float(v) for v in line.split()]))
    return [rows[i:i + 3] for i in range(0, len(rows), 3)]


def _int_data(rng, L, C, r=3):
    return rng.integers(-r, r + 1, size=(L, C)).astype(np.float64)


# ------------------------------------------------------------------ plain definitions

@pytest.mark.parametrize("case", range(3))
def test_naive_matches_hand_values(case):
    y, h, z = _hand_cases()[case]
    got = conv.causal_conv_naive(y[:, None], h[:, None])[:, 0]
    assert np.array_equal(got, z)


@pytest.mark.parametrize("L", [1, 2, 3, 17, 64, 129])
def test_naive_matches_library_convolution(L):
    rng = np.random.default_rng(L)
    y, h = rng.standard_normal((2, L))
    want = np.convolve(y, h)[:L]
    got = conv.causal_conv_naive(y[:, None], h[:, None])[:, 0]
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-13)


def test_naive_constant_filter_is_running_sum():
    rng = np.random.default_rng(1)
    y = _int_data(rng, 200, 5)
    z = conv.causal_conv_naive(y, np.ones((200, 5)))
    assert np.array_equal(z, np.cumsum(y, axis=0))


def test_naive_impulse_gives_shifted_filter():
    rng = np.random.default_rng(2)
    L, s0 = 50, 13
    h = rng.standard_normal((L, 3))
    y = np.zeros((L, 3))
    y[s0] = 1.0
    z = conv.causal_conv_naive(y, h)
    assert np.array_equal(z[:s0], np.zeros((s0, 3)))
    assert np.array_equal(z[s0:], h[: L - s0])


def test_naive_time_invariance_and_linearity():
    rng = np.random.default_rng(3)
    L, sh = 80, 9
    y1, y2, h = rng.standard_normal((3, L, 2))
    z1 = conv.causal_conv_naive(y1, h)
    z2 = conv.causal_conv_naive(y2, h)
    np.testing.assert_allclose(conv.causal_conv_naive(2 * y1 - y2, h), 2 * z1 - z2, atol=1e-12)
    ys = np.zeros_like(y1)
    ys[sh:] = y1[: L - sh]
    np.testing.assert_allclose(conv.causal_conv_naive(ys, h)[sh:], z1[: L - sh], atol=1e-12)


@pytest.mark.parametrize("L", [1, 5, 64, 1000])
def test_static_fft_matches_library_convolution(L):
    rng = np.random.default_rng(L + 100)
    y, h = rng.standard_normal((2, L, 3))
    want = np.stack([np.convolve(y[:, c], h[:, c])[:L] for c in range(3)], axis=1)
    np.testing.assert_allclose(conv.causal_conv_fft(y, h), want, rtol=0, atol=1e-11 * np.abs(want).max())


@pytest.mark.parametrize("r", [0.5, 0.9, 0.999])
def test_geometric_closed_forms(r):
    L = 300
    t = np.arange(L, dtype=np.float64)
    # y = 1 -> geometric series (1 - r^{t+1}) / (1 - r)
    z = conv.geometric_recurrence(np.ones((L, 1)), np.array([r]))[:, 0]
    np.testing.assert_allclose(z, (1 - r ** (t + 1)) / (1 - r), rtol=1e-12)
    # y = e_{s0} -> r^{t-s0} from s0 on
    s0 = 17
    e = np.zeros((L, 1))
    e[s0] = 1
    z = conv.geometric_recurrence(e, np.array([r]))[:, 0]
    assert np.array_equal(z[:s0], np.zeros(s0))
    np.testing.assert_allclose(z[s0:], r ** (t[s0:] - s0), rtol=1e-12)


def test_geometric_filter_convolution_equals_recurrence():
    """LTI-SSM view: the filter rho_k = r^k convolved with y equals the
    one-state recurrence (App. "State Space Models")."""
    rng = np.random.default_rng(4)
    L = 400
    r = np.array([0.9, 0.99, 0.9995])
    y = rng.standard_normal((L, 3))
    h = r[None, :] ** np.arange(L)[:, None]
    np.testing.assert_allclose(conv.causal_conv_naive(y, h), conv.geometric_recurrence(y, r),
                               rtol=1e-10, atol=1e-10)


# ------------------------------------------------------------------ contribution block tau

@pytest.mark.parametrize("U", [1, 2, 4, 8, 32])
def test_tau_is_middle_of_linear_convolution(U):
    """Lemma 1 / App. B: the tile is outputs [U, 2U) of the linear convolution
    of the U-block with the filter prefix h[0, 2U)."""
    rng = np.random.default_rng(U)
    yb = _int_data(rng, U, 4)
    h = _int_data(rng, 2 * U, 4)
    want = np.stack([np.convolve(yb[:, c], h[:, c])[U:2 * U] for c in range(4)], axis=1)
    assert np.array_equal(relaxed.tau_direct(yb, h, U), want)
    assert np.array_equal(relaxed.tau_direct_vec(yb, h, U), want)
    np.testing.assert_allclose(relaxed.tau_fft(yb, h, U), want, rtol=0, atol=1e-9)


@pytest.mark.parametrize("U", [1, 4, 16, 64])
def test_tau_equals_masked_full_convolution(U):
    """The tile equals the contribution of y[i-U, i) alone to z[i, i+U)."""
    rng = np.random.default_rng(U + 7)
    L, i = 4 * U, 2 * U
    y = rng.standard_normal((L, 2))
    h = rng.standard_normal((L, 2))
    ym = np.zeros_like(y)
    ym[i - U:i] = y[i - U:i]
    want = conv.causal_conv_naive(ym, h)[i:i + U]
    np.testing.assert_allclose(relaxed.tau_fft(y[i - U:i], h[: 2 * U], U), want, atol=1e-12)
    np.testing.assert_allclose(relaxed.tau_direct(y[i - U:i], h[: 2 * U], U), want, atol=1e-12)


def test_tau_ignores_h0():
    """Only lags 1..2U-1 enter the tile: h_0 may be anything."""
    rng = np.random.default_rng(9)
    U = 8
    yb = rng.standard_normal((U, 3))
    h = rng.standard_normal((2 * U, 3))
    h2 = h.copy()
    h2[0] = 1e6
    np.testing.assert_allclose(relaxed.tau_fft(yb, h, U), relaxed.tau_fft(yb, h2, U), atol=1e-6)
    assert np.array_equal(relaxed.tau_direct(yb, h, U), relaxed.tau_direct(yb, h2, U))


# ------------------------------------------------------------------ relaxed online (O2)

@pytest.mark.parametrize("L", list(range(1, 40)) + [64, 100, 128])
@pytest.mark.parametrize("tau", ["direct", "direct_vec"])
def test_relaxed_bit_exact_on_integers(L, tau):
    """Brute force on tiny L, including non-powers of two: exact equality with
    the lazy sum and with np.convolve on small-integer data."""
    rng = np.random.default_rng(1000 + L)
    M, C = 2, 3
    y = rng.integers(-3, 4, size=(L, M, C)).astype(np.float64)
    h = rng.integers(-3, 4, size=(L, M, C)).astype(np.float64)
    z, yy = relaxed_online(h, feedback.teacher_forced(y), tau=tau)
    assert np.array_equal(yy, y)
    for m in range(M):
        assert np.array_equal(z[:, m], conv.causal_conv_naive(y[:, m], h[:, m]))
        for c in range(C):
            assert np.array_equal(z[:, m, c], np.convolve(y[:, m, c], h[:, m, c])[:L])


@pytest.mark.parametrize("L", [64, 100, 512, 1024])
def test_relaxed_fft_tau_close_to_exact(L):
    rng = np.random.default_rng(L)
    y = rng.standard_normal((L, 1, 4))
    h = rng.standard_normal((L, 1, 4))
    z, _ = relaxed_online(h, feedback.teacher_forced(y), tau="fft")
    want = conv.causal_conv_fft(y[:, 0], h[:, 0])
    np.testing.assert_allclose(z[:, 0], want, rtol=0, atol=1e-12 * np.abs(want).max())


@pytest.mark.parametrize("L,M", [(1, 1), (2, 1), (7, 2), (33, 3), (64, 1), (100, 2)])
def test_relaxed_closed_loop_matches_lazy(L, M):
    """Closed loop (the tanh chain): relaxed tiling and lazy loop agree."""
    rng = np.random.default_rng(L * 10 + M)
    C = 3
    h = rng.standard_normal((L, M, C)) * np.exp(-np.arange(L) / 30.0)[:, None, None]
    x = 0.1 * rng.standard_normal((L, M, C))
    rule = feedback.tanh_chain(x, M)
    z1, y1 = lazy_online(h, rule)
    z2, y2 = relaxed_online(h, rule, tau="auto", fft_min_U=4)
    np.testing.assert_allclose(z2, z1, rtol=0, atol=1e-12 * max(1.0, np.abs(z1).max()))
    np.testing.assert_allclose(y2, y1, rtol=0, atol=1e-12)


def test_chain_rule_values():
    """The chain's first positions written out for M = 2 (zero filters past
    lag 0 make each z_t = h_0 * y_t)."""
    L, M = 3, 2
    h = np.zeros((L, M, 1))
    h[0] = 2.0
    x = np.arange(1, L * M + 1, dtype=np.float64).reshape(L, M, 1) / 10
    z, y = relaxed_online(h, feedback.tanh_chain(x, M))
    assert y[0, 0, 0] == x[0, 0, 0]
    assert y[0, 1, 0] == 0.5 * np.tanh(2 * y[0, 0, 0]) + x[0, 1, 0]
    assert y[1, 0, 0] == 0.5 * np.tanh(2 * y[0, 1, 0]) + x[1, 0, 0]
    assert np.array_equal(z, 2 * y)


def test_geometric_filter_closed_loop():
    """O2 with h_k = r^k equals the recurrence z_t = r z_{t-1} + y_t, closed loop."""
    L, M = 300, 2
    r = np.array([[0.9, 0.99], [0.95, 0.9995]])          # [M, C]
    h = r[None] ** np.arange(L)[:, None, None]
    x = 0.1 * np.random.default_rng(5).standard_normal((L, M, 2))
    z, y = relaxed_online(h, feedback.tanh_chain(x, M))
    for m in range(M):
        np.testing.assert_allclose(z[:, m], conv.geometric_recurrence(y[:, m], r[m]),
                                   rtol=1e-10, atol=1e-10)


def test_causality_future_inputs_do_not_change_past_outputs():
    rng = np.random.default_rng(11)
    L, t0 = 256, 97
    h = rng.standard_normal((L, 1, 3))
    y = rng.standard_normal((L, 1, 3))
    y2 = y.copy()
    y2[t0 + 1:] = rng.standard_normal((L - t0 - 1, 1, 3))
    z, _ = relaxed_online(h, feedback.teacher_forced(y))
    z2, _ = relaxed_online(h, feedback.teacher_forced(y2))
    assert np.array_equal(z[: t0 + 1], z2[: t0 + 1])
    assert not np.array_equal(z[t0 + 1:], z2[t0 + 1:])


def test_nan_poison_reaches_every_later_output_of_its_column_only():
    rng = np.random.default_rng(12)
    L, t0 = 128, 37
    h = rng.standard_normal((L, 2, 3))
    y = rng.standard_normal((L, 2, 3))
    y[t0, 1, 2] = np.nan
    z, _ = relaxed_online(h, feedback.teacher_forced(y))
    assert np.all(np.isnan(z[t0:, 1, 2]))
    mask = np.ones(z.shape, dtype=bool)
    mask[t0:, 1, 2] = False
    assert np.all(np.isfinite(z[mask]))


def test_filters_to_columns_layout():
    h = np.arange(2 * 3 * 5, dtype=np.float64).reshape(2, 3, 5)   # [M, D, L]
    hc = filters_to_columns(h, B=2)
    assert hc.shape == (5, 2, 6)
    for m in range(2):
        for b in range(2):
            for d in range(3):
                assert np.array_equal(hc[:, m, b * 3 + d], h[m, d])


# ------------------------------------------------------------------ planted mistakes

def _run_with(monkeypatch, name, fn, L=64):
    monkeypatch.setitem(relaxed.TAUS, name, fn)
    rng = np.random.default_rng(99)
    y = rng.integers(-3, 4, size=(L, 1, 2)).astype(np.float64)
    h = rng.integers(-3, 4, size=(L, 1, 2)).astype(np.float64)
    z, _ = relaxed_online(h, feedback.teacher_forced(y), tau=name)
    return z[:, 0], conv.causal_conv_naive(y[:, 0], h[:, 0])


def test_planted_lag_off_by_one_is_caught(monkeypatch):
    def bad(yb, h, U):
        out = np.zeros(yb.shape)
        for j in range(U):
            for k in range(U):
                out[j] += yb[k] * h[U + j - k - 1]
        return out
    z, want = _run_with(monkeypatch, "direct", bad)
    assert not np.array_equal(z, want)


def test_planted_transposed_block_is_caught(monkeypatch):
    def bad(yb, h, U):
        return relaxed.tau_direct(yb[::-1], h, U)
    z, want = _run_with(monkeypatch, "direct", bad)
    assert not np.array_equal(z, want)


def test_planted_wrong_fft_window_is_caught(monkeypatch):
    def bad(yb, h, U):
        n = 2 * U
        w = np.fft.irfft(np.fft.rfft(yb, n=n, axis=0) * np.fft.rfft(h[:n], n=n, axis=0), n=n, axis=0)
        return w[U - 1:n - 1]
    z, want = _run_with(monkeypatch, "fft", bad)
    assert np.abs(z - want).max() > 0.5


def test_planted_missing_red_cell_is_caught(monkeypatch):
    monkeypatch.setattr(relaxed.RelaxedOnline, "red",
                        lambda self, m, y_m: (self.y.__setitem__((self.t, m), y_m), self.acc[self.t, m])[1])
    rng = np.random.default_rng(3)
    L = 32
    y = rng.integers(-3, 4, size=(L, 1, 2)).astype(np.float64)
    h = rng.integers(1, 4, size=(L, 1, 2)).astype(np.float64)
    z, _ = relaxed_online(h, feedback.teacher_forced(y))
    assert not np.array_equal(z[:, 0], conv.causal_conv_naive(y[:, 0], h[:, 0]))
