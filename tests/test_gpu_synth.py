"""GPU parity of the synthetic end-to-end model (include/lcsm_synth.h; needs an
MI355X).

The model of the experiments (Sec. 5): per layer the long-convolution mixer
and an MLP block (hidden 2D, exact GELU); the next token's input is the last
layer's output plus noise.  Bars: every block output of every layer and
position against the fp64 oracle (the relaxed oracle driven by the model's
input rule, ``oracle.block.mlp_chain``), max|a_gpu - a_ref| <= 1e-4 *
max|a_ref|; with blocks that are the identity, the same against the oracle's
linear model; with half-state storage, bit for bit the full-state outputs.
"""
import dataclasses

import numpy as np
import pytest
import torch

import datagen
from oracle.block import activations, mlp_chain
from oracle.relaxed import filters_to_columns, relaxed_online

from gpu_harness import TOL, dev, lcsm_mod, rel_err, say

pytestmark = pytest.mark.gpu


def _weights_torch(ws):
    return tuple(torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev()) for a in ws)


def _gpu_run(model, eps, n):
    """Positions 0..n-1; returns act [n, M, B, D] (numpy)."""
    act = torch.full((n, model.M, model.B, model.D), float("nan"), dtype=torch.float32,
                     device=dev())
    for t in range(n):
        model.step(eps[t], act[t])
    torch.cuda.synchronize()
    return act.cpu().numpy()


def _oracle(h_mdl, weights, eps_np, M, B, D, n):
    """Block outputs a^{m+1}_t [n, M, B*D] of the first n positions."""
    h = filters_to_columns(h_mdl[:, :, :n], B)
    z, _ = relaxed_online(h, mlp_chain(weights, eps_np[:n], M, B, D))
    return activations(z, weights, B, D)


def _make(w, filters=None, weights=None, options=None):
    lcsm = lcsm_mod()
    if filters is None:
        filters = datagen.filters_torch(w, dev())
    if weights is None:
        weights = datagen.mlp_weights_torch(w, dev())
    return lcsm.Synth(filters, *weights, w.B, options=options)


@pytest.mark.parametrize("shape", [(1, 1, 16, 1024), (2, 3, 16, 300), (3, 2, 40, 1000),
                                   (2, 17, 8, 200), (1, 4, 64, 2048), (2, 9, 1500, 64)])
def test_synth_matches_oracle(shape):
    """Includes the 16-channel 1024-position workload's shape, a ragged batch
    (17 rows: two product launches of 16 and 1), every tile kind, and products
    on the matrix cores with ragged blocks (9 of 16 rows; 3000 and 1500
    units and inputs, neither a multiple of 16)."""
    M, B, D, L = shape
    say(f"[synth] M={M} B={B} D={D} L={L}")
    w = datagen.Workload("synth", M, B, D, L, decay=L / 5, seed=50 + M + B)
    model = _make(w)
    eps = datagen.noise_torch(w, dev())
    act = _gpu_run(model, eps, L)
    assert model.position == L
    ref = _oracle(datagen.filters_np(w), datagen.mlp_weights_np(w), datagen.noise_np(w), M, B, D, L)
    err = rel_err(act.reshape(L, M, -1), ref)
    say(f"  rel err {err:.3e}, max |a| {np.abs(ref).max():.3f}")
    assert err <= TOL


def test_synth_identity_blocks():
    """W_up = [I; -I], W_down = [I, -I], no biases: each block is the identity
    (gelu(x) - gelu(-x) = x) and the model is linear in the noise."""
    M, B, D, L = 3, 2, 8, 600
    w = datagen.Workload("synthid", M, B, D, L, decay=60.0, seed=11)
    say(f"[synth identity blocks] M={M} B={B} D={D} L={L}")
    h = datagen.filters_np(w).astype(np.float64)
    h = (h / (2 * np.abs(h).sum(axis=2, keepdims=True))).astype(np.float32)  # contractions
    eye = np.eye(D)
    weights = (np.broadcast_to(np.concatenate([eye, -eye], 0), (M, 2 * D, D)),
               np.zeros((M, 2 * D)),
               np.broadcast_to(np.concatenate([eye, -eye], 1), (M, D, 2 * D)),
               np.zeros((M, D)))
    model = _make(w, torch.from_numpy(h).to(dev()), _weights_torch(weights))
    act = _gpu_run(model, datagen.noise_torch(w, dev()), L)
    ref = _oracle(h, weights, datagen.noise_np(w), M, B, D, L)
    err = rel_err(act.reshape(L, M, -1), ref)
    say(f"  rel err {err:.3e}")
    assert err <= TOL


def test_synth_half_state_equals_full_state_and_reset_repeats():
    M, B, D, L = 2, 3, 24, 1200
    w = datagen.Workload("synthhalf", M, B, D, L, decay=300.0, seed=13)
    say(f"[synth half state] M={M} B={B} D={D} L={L}")
    filters = datagen.filters_torch(w, dev())
    weights = datagen.mlp_weights_torch(w, dev())
    eps = datagen.noise_torch(w, dev())
    full = _make(w, filters, weights)
    half = _make(w, filters, weights, {"half_state": 1})
    a_full = _gpu_run(full, eps, L)
    a_half = _gpu_run(half, eps, L)
    assert np.array_equal(a_full, a_half)
    half.reset()
    assert half.position == 0
    assert np.array_equal(a_half, _gpu_run(half, eps, L))


@pytest.mark.parametrize("name,n", [("m1b8d768l8k", 1024), ("m18b4d768l32k", 128),
                                    ("m32b16d2048l16k", 16)])
def test_synth_workload_width_prefix(name, n):
    """The workloads' full widths (768 channels, 8 and 4 batch rows, 1 and 18
    layers; 2048 channels, 16 batch rows, 32 layers: full 16-row matrix-core
    blocks) over the first n positions of the generation."""
    w = datagen.WORKLOADS[name]
    if w.M * w.B * w.D >= 1 << 19:
        # the products' widths are what is checked; a short context keeps the
        # mixer's state (and its column-major mirror) small
        w = dataclasses.replace(w, L=256)
    say(f"[synth prefix] {name} M={w.M} B={w.B} D={w.D} L={w.L} positions={n}")
    # the generator's torch view (bit-identical to its numpy view) draws the
    # 42M weights of 18 layers in seconds; the oracle gets the same values
    weights = datagen.mlp_weights_torch(w, dev())
    model = _make(w, weights=weights)
    act = _gpu_run(model, datagen.noise_torch(w, dev(), 0, n), n)
    ref = _oracle(datagen.filters_np(w, lags=n), tuple(t.cpu().numpy() for t in weights),
                  datagen.noise_np(w, 0, n), w.M, w.B, w.D, n)
    err = rel_err(act.reshape(n, w.M, -1), ref)
    say(f"  rel err {err:.3e}")
    assert err <= TOL


def test_synth_errors():
    lcsm = lcsm_mod()
    w = datagen.Workload("syntherr", 1, 2, 8, 140, decay=30.0, seed=1)
    model = _make(w)
    eps = datagen.noise_torch(w, dev())
    with pytest.raises(ValueError):
        model.step(eps[0][:1])
    _gpu_run(model, eps, w.L)
    with pytest.raises(lcsm.LcsmError) as ex:
        model.step(eps[0])
    assert ex.value.code == lcsm.LCSM_EDONE
    model.reset()
    model.step(eps[0])
    assert model.position == 1
