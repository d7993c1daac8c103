"""GPU parity of half-state storage (App. C; lcsm_options.half_state; needs an
MI355X).

The state keeps T rows per layer (T the largest power of two below L): the
gray tile of i = T stores its outputs for positions [T, L) over its own
inputs, and later positions live at row p - T.  Bars: every output against
the fp64 oracle, max|z_gpu - z_ref| <= 1e-4 * max|z_ref|; on small-integer
data the rounded outputs equal the exact int64 convolution; and every output
equal to that of the full-state context on the same inputs (the arithmetic is
the same, only the addresses differ).  The option sets put the in-place tile
in one LDS pass (unclipped and clipped destinations, whole and ragged panels)
and in the multi-pass form with one and with many column chunks.
"""
import numpy as np
import pytest
import torch

import datagen
from oracle import conv, feedback
from oracle.relaxed import filters_to_columns, relaxed_online

from gpu_harness import TOL, dev, lcsm_mod, make_ctx, oracle_sampled, rel_err, say

pytestmark = pytest.mark.gpu

OPTIONS = {
    "default": {},
    # every tile above U = 1 an FFT tile, one LDS pass up to 2U = 8192
    "lds_from_2": {"direct_max_u": 1, "lds_fft_max_n": 8192, "col_fft_min_n": 1 << 20},
    # every tile with 2U > 16, the swap included, in three passes
    "multipass_from_16": {"direct_max_u": 1, "lds_fft_max_n": 16, "col_fft_min_n": 1 << 20},
    # three passes with a 1 MiB scratch: the swap in many column chunks
    "tiny_scratch": {"direct_max_u": 4, "lds_fft_max_n": 32, "scratch_mib": 1, "col_fft_min_n": 1 << 20},
    # the swap (and every FFT tile) on transposed column chunks, many chunks
    "col_tiny_scratch": {"direct_max_u": 4, "col_fft_min_n": 16, "scratch_mib": 1},
}


def _half(opts):
    return dict(opts, half_state=1)


def _full(opts=None):
    """Options of the full-state context a half-state one equals bit for bit:
    half-state storage runs the column-tile sizes on transposed chunks, so the
    full-state context does too (on the column-major mirror its large tiles
    are summed in a different order)."""
    return dict(opts or {}, col_tile_form=1)


def _run(ctx, y):
    z = torch.full_like(y, float("nan"))
    ctx.run(y, z)
    torch.cuda.synchronize()
    return z.cpu().numpy()


def _oracle(w, y):
    h = filters_to_columns(datagen.filters_np(w), w.B)
    return conv.causal_conv_fft(y.cpu().numpy().reshape(w.L, -1).astype(np.float64),
                                h.reshape(h.shape[0], -1))


@pytest.mark.parametrize("opt", ["default", "lds_from_2", "multipass_from_16", "tiny_scratch",
                                 "col_tiny_scratch"])
@pytest.mark.parametrize("shape", [(2, 3, 40, 300), (1, 4, 64, 2048), (3, 2, 33, 1000),
                                   (1, 2, 48, 4500), (2, 2, 24, 8192)])
def test_half_state_matches_oracle_and_full_state(opt, shape):
    M, B, D, L = shape
    say(f"[half state] M={M} B={B} D={D} L={L} options={opt}")
    w = datagen.Workload("half", M, B, D, L, decay=L / 3, seed=40 + L % 97)
    filt = datagen.filters_torch(w, dev())
    full, _ = make_ctx(w, filt, _full(OPTIONS[opt]))
    half, _ = make_ctx(w, filt, _half(OPTIONS[opt]))
    y = datagen.y_torch(w, dev())
    zf = _run(full, y)
    zh = _run(half, y)
    assert not np.isnan(zh).any()
    assert np.array_equal(zf, zh)
    err = rel_err(zh.reshape(L, -1), _oracle(w, y))
    say(f"  rel err {err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("opt", ["default", "multipass_from_16", "tiny_scratch", "col_tiny_scratch"])
def test_half_state_integer_data_rounds_to_exact(opt):
    M, B, D, L = 2, 3, 20, 1500
    w = datagen.Workload("halfint", M, B, D, L, decay=1.0, seed=9)
    h, y = datagen.int_filters_np(w, 3), datagen.int_y_np(w, 3)
    say(f"[half state int] M={M} B={B} D={D} L={L} options={opt}")
    ctx, _ = make_ctx(w, torch.from_numpy(h).to(dev()), _half(OPTIONS[opt]))
    z = _run(ctx, torch.from_numpy(y).to(dev()))
    ex = np.zeros((L, M, B, D), dtype=np.int64)
    hi, yi = h.astype(np.int64), y.astype(np.int64)
    for k in range(L):
        ex[k:] += yi[: L - k] * hi[None, :, None, :, k]
    assert np.abs(z.astype(np.float64) - ex).max() < 0.25
    assert np.array_equal(np.rint(z).astype(np.int64), ex)


def _layer_path(ctx, y, M, L):
    z = torch.full_like(y, float("nan"))
    for t in range(L):
        for m in range(M):
            ctx.step_layer(m, y[t, m], z[t, m])
        ctx.advance()
    torch.cuda.synchronize()
    return z.cpu().numpy()


@pytest.mark.parametrize("opt", ["default", "multipass_from_16"])
def test_half_state_layer_path_chain_and_reset(opt):
    """lcsm_step_layer / lcsm_advance and the built-in chain cross the swap
    as lcsm_step does: each path equals the full-state context's same path
    (the run and layer paths themselves agree to rounding only: the fused
    red-cell FFT tile rounds differently from the unfused one), and a reset
    context repeats the same bits."""
    w = datagen.Workload("halfpaths", 3, 2, 40, 1200, decay=300.0, seed=14)
    say(f"[half state paths] M=3 B=2 D=40 L=1200 options={opt}")
    filt = datagen.filters_torch(w, dev())
    full, _ = make_ctx(w, filt, _full(OPTIONS[opt]))
    half, _ = make_ctx(w, filt, _half(OPTIONS[opt]))
    y = datagen.y_torch(w, dev())
    za = _run(half, y)
    half.reset()
    zb = _layer_path(half, y, w.M, w.L)
    assert np.array_equal(zb, _layer_path(full, y, w.M, w.L))
    assert rel_err(za, zb.astype(np.float64)) <= 1e-5
    half.reset()
    assert np.array_equal(za, _run(half, y))
    # the closed loop (tanh chain) against the full-state context
    x = datagen.x_torch(w, dev())
    half.reset()
    full.reset()
    zc = torch.empty_like(x)
    zd = torch.empty_like(x)
    for t in range(w.L):
        half.step_chain(x[t], zc[t])
        full.step_chain(x[t], zd[t])
    torch.cuda.synchronize()
    assert torch.equal(zc, zd)


def test_half_state_closed_loop_matches_oracle():
    w = datagen.WORKLOADS["m1b1d16l1k"]
    say(f"[half state closed loop] {w.name}")
    ctx, _ = make_ctx(w, options={"half_state": 1})
    x = datagen.x_torch(w, dev())
    z = torch.empty_like(x)
    for t in range(w.L):
        ctx.step_chain(x[t], z[t])
    torch.cuda.synchronize()
    h = filters_to_columns(datagen.filters_np(w), w.B)
    zr, _ = relaxed_online(h, feedback.tanh_chain(datagen.x_np(w).reshape(w.L, w.M, -1), w.M))
    err = rel_err(z.cpu().numpy().reshape(w.L, w.M, -1), zr)
    say(f"  closed-loop rel err {err:.3e}")
    assert err <= TOL


def test_half_state_prefill():
    """A prompt of T/2 positions (the largest a half state holds), then the
    generation across the swap; a prompt of T is rejected."""
    lcsm = lcsm_mod()
    w = datagen.Workload("halfprefill", 2, 2, 48, 4096, decay=1024.0, seed=21)
    T = 2048
    say(f"[half state prefill] M=2 B=2 D=48 L=4096 P={T // 2}")
    filt = datagen.filters_torch(w, dev())
    full, _ = make_ctx(w, filt, _full())
    half, _ = make_ctx(w, filt, {"half_state": 1})
    y = datagen.y_torch(w, dev())
    out = []
    for ctx in (full, half):
        z = torch.full_like(y, float("nan"))
        ctx.prefill(y[:T // 2], z[:T // 2])
        ctx.run(y[T // 2:], z[T // 2:])
        torch.cuda.synchronize()
        out.append(z.cpu().numpy())
    assert np.array_equal(out[0], out[1])
    assert rel_err(out[1].reshape(w.L, -1), _oracle(w, y)) <= TOL
    half.reset()
    z = torch.empty_like(y)
    with pytest.raises(lcsm.LcsmError) as ex:
        half.prefill(y[:T], z[:T])
    assert ex.value.code == lcsm.LCSM_EINVAL
    assert half.position == 0


def test_half_state_bench_workload_all_columns():
    w = datagen.WORKLOADS["m1b8d768l8k"]
    say(f"[half state] {w.name} all columns")
    ctx, _ = make_ctx(w, options={"half_state": 1})
    y = datagen.y_torch(w, dev())
    z = _run(ctx, y)
    err = rel_err(z.reshape(w.L, -1), _oracle(w, y))
    say(f"  rel err {err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("name", ["m18b4d768l32k", "m18b1d1024l128k", "m32b16d2048l16k"])
def test_half_state_full_size_equals_full_state(name):
    """At the full sizes (multi-pass swap tiles of 2T = 32768, 131072 and
    16384 points, in 512 MiB column chunks) every output of the half-state
    context equals the full-state one, position chunk by position chunk;
    sampled columns also against the oracle."""
    w = datagen.WORKLOADS[name]
    say(f"[half state full size] {name}")
    filt = datagen.filters_torch(w, dev())
    full, _ = make_ctx(w, filt, _full())
    half, _ = make_ctx(w, filt, {"half_state": 1})
    cols = datagen.sample_columns(w, 6, seed=77)
    cm, cb, cd = (torch.as_tensor(cols[:, k], device=dev()) for k in range(3))
    chunk = 256 if w.M * w.B * w.D <= (1 << 17) else 64
    zf = torch.empty((chunk, w.M, w.B, w.D), dtype=torch.float32, device=dev())
    zh = torch.empty_like(zf)
    got = []
    for t0 in range(0, w.L, chunk):
        t1 = min(w.L, t0 + chunk)
        y = datagen.y_torch(w, dev(), t0, t1).contiguous()
        full.run(y, zf, n=t1 - t0)
        half.run(y, zh, n=t1 - t0)
        if not torch.equal(zf[: t1 - t0], zh[: t1 - t0]):
            pytest.fail(f"half-state outputs differ in positions [{t0}, {t1})")
        got.append(zh[: t1 - t0, cm, cb, cd].cpu())
    torch.cuda.synchronize()
    z = torch.cat(got).numpy()
    err = rel_err(z, oracle_sampled(w, cols))
    say(f"  sampled rel err {err:.3e}")
    assert err <= TOL
