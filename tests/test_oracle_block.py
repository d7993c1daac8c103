"""Pins of the synthetic model's blocks and sampler in the oracle (Sec. 5) --
CPU only.

GELU against values of the standard normal CDF from any table and against
its symmetry; the MLP against a scalar loop with math.erf and against a
weight choice that makes it the identity; the closed loop of the whole model
(identity blocks) against a linear solve that never steps through time; and
zero weights, where every block output is its bias.
"""
import math

import numpy as np
import pytest

import datagen
from oracle import conv
from oracle.block import activations, gelu, mlp, mlp_chain
from oracle.relaxed import filters_to_columns, lazy_online, relaxed_online


def test_gelu_table_values():
    # Phi(1), Phi(2), Phi(-1) of the standard normal distribution
    phi1, phi2 = 0.8413447460685429, 0.9772498680518208
    assert gelu(1.0) == pytest.approx(phi1, abs=1e-15)
    assert gelu(2.0) == pytest.approx(2 * phi2, abs=1e-15)
    assert gelu(-1.0) == pytest.approx(-(1 - phi1), abs=1e-15)
    assert gelu(0.0) == 0.0
    assert gelu(12.0) == pytest.approx(12.0, abs=1e-15)
    assert abs(gelu(-12.0)) < 1e-30


def test_gelu_odd_part_is_identity():
    # Phi(x) + Phi(-x) = 1  =>  gelu(x) - gelu(-x) = x
    x = np.random.default_rng(0).normal(size=1000) * 3
    assert np.allclose(gelu(x) - gelu(-x), x, atol=1e-14, rtol=0)


def _scalar_mlp(x, w_up, b_up, w_down, b_down):
    D = len(x)
    hidden = []
    for n in range(2 * D):
        s = float(b_up[n])
        for k in range(D):
            s += float(w_up[n][k]) * float(x[k])
        hidden.append(s * 0.5 * (1.0 + math.erf(s / math.sqrt(2.0))))
    out = []
    for n in range(D):
        s = float(b_down[n])
        for k in range(2 * D):
            s += float(w_down[n][k]) * hidden[k]
        out.append(s)
    return np.array(out)


def test_mlp_against_scalar_loop():
    w = datagen.Workload("blk", 2, 3, 5, 64, decay=10.0, seed=4)
    w_up, b_up, w_down, b_down = datagen.mlp_weights_np(w)
    x = np.random.default_rng(1).normal(size=(3, 5))
    got = mlp(x, w_up[1], b_up[1], w_down[1], b_down[1])
    for b in range(3):
        want = _scalar_mlp(x[b], w_up[1], b_up[1], w_down[1], b_down[1])
        assert np.allclose(got[b], want, atol=1e-13, rtol=0)


def _identity_weights(M, D):
    eye = np.eye(D)
    w_up = np.broadcast_to(np.concatenate([eye, -eye], axis=0), (M, 2 * D, D))
    w_down = np.broadcast_to(np.concatenate([eye, -eye], axis=1), (M, D, 2 * D))
    return w_up, np.zeros((M, 2 * D)), w_down, np.zeros((M, D))


def test_mlp_reduces_to_identity():
    """W_up = [I; -I], W_down = [I, -I], no biases: gelu(x) - gelu(-x) = x."""
    D = 7
    w_up, b_up, w_down, b_down = _identity_weights(1, D)
    x = np.random.default_rng(2).normal(size=(4, D)) * 2
    assert np.allclose(mlp(x, w_up[0], b_up[0], w_down[0], b_down[0]), x, atol=1e-14, rtol=0)


def test_identity_blocks_closed_loop_solves_the_linear_system():
    """With identity blocks the model is linear: a^0 = eps + S P a^0, P the
    product of the layers' lower-triangular Toeplitz matrices, S the shift by
    one position.  The stepped oracle must equal the solve of (I - S P)."""
    M, B, D, L = 3, 2, 3, 40
    w = datagen.Workload("idl", M, B, D, L, decay=6.0, seed=8)
    h = filters_to_columns(datagen.filters_np(w), B)           # [L, M, C]
    # each layer a contraction (sum |h| = 1/2), so the system is well conditioned
    h = h / (2 * np.abs(h).sum(axis=0, keepdims=True))
    eps = datagen.noise_np(w).astype(np.float64)                # [L, B, D]
    rule = mlp_chain(_identity_weights(M, D), eps, M, B, D)
    z, y = relaxed_online(h, rule)
    S = np.eye(L, k=-1)
    for c in range(B * D):
        P = np.eye(L)
        for m in range(M):
            T = np.zeros((L, L))
            for k in range(L):
                T += np.eye(L, k=-k) * h[k, m, c]
            P = T @ P
        a0 = np.linalg.solve(np.eye(L) - S @ P, eps.reshape(L, -1)[:, c])
        assert np.allclose(y[:, 0, c], a0, atol=1e-10, rtol=1e-10)
        assert np.allclose(z[:, M - 1, c], P @ a0, atol=1e-10, rtol=1e-10)


def test_zero_weights_give_the_biases():
    M, B, D, L = 2, 2, 4, 50
    w = datagen.Workload("zw", M, B, D, L, decay=8.0, seed=2)
    h = filters_to_columns(datagen.filters_np(w), B)
    eps = datagen.noise_np(w).astype(np.float64)
    b_up = np.random.default_rng(3).normal(size=(M, 2 * D))
    b_down = np.random.default_rng(4).normal(size=(M, D))
    weights = (np.zeros((M, 2 * D, D)), b_up, np.zeros((M, D, 2 * D)), b_down)
    z, y = relaxed_online(h, mlp_chain(weights, eps, M, B, D))
    assert np.array_equal(y[0, 0], eps[0].reshape(-1))
    assert np.allclose(y[1:, 0], np.tile(b_down[M - 1], B)[None, :] + eps[1:].reshape(L - 1, -1),
                       atol=1e-15, rtol=0)
    assert np.allclose(y[:, 1], np.tile(b_down[0], B)[None, :], atol=1e-15, rtol=0)
    # layer 1 sees a constant input: z_t = b * sum_{k<=t} h_k
    zc = conv.causal_conv_naive(y[:, 1:2], h[:, 1:2])
    assert np.allclose(z[:, 1:2], zc, atol=1e-12, rtol=0)
    a = activations(z, weights, B, D)
    assert np.allclose(a[:, 1], np.tile(b_down[1], B)[None, :], atol=1e-15, rtol=0)


def test_relaxed_and_lazy_agree_on_the_mlp_model():
    M, B, D, L = 2, 2, 6, 96
    w = datagen.Workload("mlp", M, B, D, L, decay=20.0, seed=6)
    h = filters_to_columns(datagen.filters_np(w), B)
    rule = mlp_chain(datagen.mlp_weights_np(w), datagen.noise_np(w), M, B, D)
    z1, y1 = relaxed_online(h, rule)
    z2, y2 = lazy_online(h, rule)
    scale = np.abs(z2).max()
    assert np.abs(z1 - z2).max() <= 1e-12 * scale
    assert np.abs(y1 - y2).max() <= 1e-12 * max(1.0, np.abs(y2).max())


def test_recipe_keeps_the_closed_loop_bounded():
    """The weight scales of the synthetic recipe keep activations O(1) over a
    long closed loop (no blow-up for the fp32 path to chase)."""
    w = datagen.Workload("bounded", 2, 2, 8, 2048, decay=256.0, seed=9)
    h = filters_to_columns(datagen.filters_np(w), w.B)
    z, y = relaxed_online(h, mlp_chain(datagen.mlp_weights_np(w), datagen.noise_np(w),
                                       w.M, w.B, w.D))
    assert np.isfinite(z).all()
    assert np.abs(y).max() < 10 and np.abs(z).max() < 100
