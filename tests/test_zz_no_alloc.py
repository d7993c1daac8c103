"""lcsm_run_noalloc (the allocation-free lcsm_run) against lcsm_run, through
the C ABI, on the GPU (needs an MI355X).

Two calls in a row on contexts of different shapes, the second smaller (the
static scratch then still holds the first call's data): each is compared
with lcsm_run on a twin context within the fp32 tolerance, and with the fp64
oracle.  Column tiles and three-pass tiles are forced on small shapes so that
both kinds of staged tile run in several chunks of the static scratch."""
import ctypes

import numpy as np
import pytest
import torch

import datagen
from oracle import conv

from gpu_harness import TOL, dev, lcsm_mod, rel_err, say

pytestmark = pytest.mark.gpu

CASES = [
    # (M, B, D, L, options): column tiles from 2U = 256 (several 64-column
    # chunks per layer), three-pass tiles above 2U = 2048
    (3, 4, 700, 4096, {"col_fft_min_n": 256, "lds_fft_max_n": 2048}),
    # smaller: three-pass only, one layer
    (1, 2, 37, 1500, {"lds_fft_max_n": 64, "col_fft_min_n": 1 << 20}),
]


def _pair(M, B, D, L, opts, seed):
    lcsm = lcsm_mod()
    w = datagen.Workload("noalloc", M, B, D, L, decay=L / 4, seed=seed)
    h = datagen.filters_torch(w, dev())
    y = datagen.y_torch(w, dev())
    a = lcsm.Lcsm(h, B, options=opts)
    b = lcsm.Lcsm(h, B, options=opts)
    return w, y, a, b


def test_run_noalloc_matches_run_twice():
    lib = lcsm_mod().raw()
    for k, (M, B, D, L, opts) in enumerate(CASES):
        say(f"[run_noalloc] call {k + 1}: M={M} B={B} D={D} L={L} opts={opts}")
        w, y, ca, cb = _pair(M, B, D, L, opts, seed=40 + k)
        za = torch.full_like(y, float("nan"))
        zb = torch.full_like(y, float("nan"))
        slab = M * B * D
        r = lib.lcsm_run_noalloc(ca._ctx, L, ctypes.c_void_p(y.data_ptr()), slab,
                                 ctypes.c_void_p(za.data_ptr()), slab)
        assert r == 0, lib.lcsm_last_error(ca._ctx)
        cb.run(y, zb)
        torch.cuda.synchronize()
        assert ca.position == L
        zr = zb.cpu().numpy().reshape(L, -1).astype(np.float64)
        zn = za.cpu().numpy().reshape(L, -1)
        assert np.isfinite(zn).all()
        err = rel_err(zn, zr)
        say(f"  vs lcsm_run: rel err {err:.3e}")
        assert err <= TOL
        # and against the fp64 oracle on every column
        hn = datagen.filters_np(w)
        hc = np.broadcast_to(hn.transpose(2, 0, 1)[:, :, None, :], (L, M, B, D)).reshape(L, -1)
        zo = conv.causal_conv_fft(datagen.y_np(w).reshape(L, -1), hc)
        err_o = rel_err(zn, zo)
        say(f"  vs oracle: rel err {err_o:.3e}")
        assert err_o <= TOL
        ca.close()
        cb.close()


def test_run_noalloc_errors():
    lcsm = lcsm_mod()
    lib = lcsm.raw()
    fake = ctypes.c_void_p(4096)
    assert lib.lcsm_run_noalloc(None, 1, fake, 0, fake, 0) == lcsm.LCSM_EINVAL
    w = datagen.Workload("noalloc_e", 1, 1, 8, 64, decay=16.0, seed=2)
    ctx = lcsm.Lcsm(datagen.filters_torch(w, dev()), 1)
    assert lib.lcsm_run_noalloc(ctx._ctx, -1, fake, 0, fake, 0) == lcsm.LCSM_EINVAL
    assert lib.lcsm_run_noalloc(ctx._ctx, 1, None, 0, fake, 0) == lcsm.LCSM_EINVAL
    ctx.close()
