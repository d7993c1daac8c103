"""lcsm_run_chain (stretches of chained steps in one launch) on the GPU
(needs an MI355X).

Where the shape allows (full state, at most 30 layers, at most 8192 columns
per layer) the chained steps of a stretch inside an aligned block of 32
positions whose gray tiles are direct tiles of U <= 16 run in one launch
that keeps the block's rows of every column in registers; the results must
equal the loop of single lcsm_step_chain calls bit for bit: one and several
layers (odd counts, and 30: sixteen waves), ragged shapes, lengths that are
not powers of two, the column-major mirror's tiles and stretches cut before
their block ends (direct tiles only up to U = 4, so the accumulators held in
registers go back to the state), every tile direct (the direct tiles of
U = 32 end a stretch), runs split into several calls at positions inside
blocks, and the shapes that take one position at a time (half-state
storage, more than 30 layers, more than 8192 columns).  Two shapes are also
checked against the fp64 oracle's closed loop."""
import numpy as np
import pytest
import torch

import datagen
from oracle import feedback
from oracle.relaxed import filters_to_columns, relaxed_online

from gpu_harness import TOL, dev, lcsm_mod, rel_err, say

pytestmark = pytest.mark.gpu

CASES = [
    ((1, 1, 16, 1024), None),
    ((3, 2, 33, 300), None),
    ((2, 3, 40, 2048), None),
    ((2, 4, 48, 2048), {"direct_max_u": 4, "col_fft_min_n": 16}),   # mirrored tiles from U = 8
    ((2, 2, 20, 700), {"direct_max_u": 1 << 20}),                   # every tile direct
    ((30, 1, 40, 300), None),                                       # sixteen waves
    ((18, 1, 64, 4096), None),
    ((2, 2, 24, 1200), {"half_state": 1}),                          # one position at a time
    ((34, 1, 8, 300), None),                                        # more layers than one launch takes
    ((1, 2, 4100, 200), None),                                      # more columns than one launch takes
    ((2, 1, 8, 1), None),                                           # one position, no tile
    ((1, 3, 8, 33), None),                                          # a last block of one position
]


def _ctx(w, opts):
    lcsm = lcsm_mod()
    h = datagen.filters_torch(w, dev())
    return lcsm.Lcsm(h, w.B, options=opts)


@pytest.mark.parametrize("shape,opts", CASES)
def test_run_chain_equals_single_steps(shape, opts):
    M, B, D, L = shape
    say(f"[run_chain] M={M} B={B} D={D} L={L} opts={opts}")
    w = datagen.Workload("chainrun", M, B, D, L, decay=L / 4, seed=M + 3 * B + D)
    x = datagen.x_torch(w, dev())
    ctx = _ctx(w, opts)
    z_ref = torch.empty_like(x)
    with torch.cuda.stream(ctx.stream):
        for t in range(L):
            ctx.step_chain(x[t], z_ref[t])
    torch.cuda.synchronize()
    ctx.reset()
    z = torch.full_like(x, float("nan"))
    ctx.run_chain(x, z)
    torch.cuda.synchronize()
    assert ctx.position == L
    assert torch.equal(z, z_ref)
    # in pieces that cut stretches in their middle
    ctx.reset()
    z2 = torch.full_like(x, float("nan"))
    cuts = [0, 5, 37, 38, 600, L]
    cuts = sorted({min(c, L) for c in cuts})
    for a, b in zip(cuts[:-1], cuts[1:]):
        ctx.run_chain(x[a:b], z2[a:b])
    torch.cuda.synchronize()
    assert torch.equal(z2, z_ref)
    ctx.close()


@pytest.mark.parametrize("name", ["m1b1d16l1k", "layers4"])
def test_run_chain_matches_the_oracle_closed_loop(name):
    """The 1024-position workload, and 4 layers over 300 positions with
    fast-decaying filters: lengths over which an fp32 closed loop still
    follows the fp64 one (further on the chaotic loop amplifies rounding)."""
    w = (datagen.WORKLOADS[name] if name in datagen.WORKLOADS
         else datagen.Workload("chainrunref", 4, 2, 24, 300, decay=200.0, seed=25))
    M, B, D, L = w.M, w.B, w.D, w.L
    say(f"[run_chain vs oracle] M={M} B={B} D={D} L={L}")
    h = datagen.filters_np(w)
    x = datagen.x_np(w)
    ctx = lcsm_mod().Lcsm(torch.from_numpy(h).to(dev()), w.B)
    xd = torch.from_numpy(x).to(dev())
    z = torch.empty_like(xd)
    ctx.run_chain(xd, z)
    torch.cuda.synchronize()
    ctx.close()
    zr, _ = relaxed_online(filters_to_columns(h, w.B), feedback.tanh_chain(x.reshape(L, M, -1), M))
    err = rel_err(z.cpu().numpy().reshape(L, M, -1), zr)
    say(f"  rel err {err:.3e}")
    assert err <= TOL


def test_run_chain_errors():
    lcsm = lcsm_mod()
    w = datagen.Workload("chainrunerr", 1, 1, 8, 40, decay=10.0, seed=2)
    x = datagen.x_torch(w, dev())
    ctx = _ctx(w, None)
    z = torch.empty_like(x)
    ctx.run_chain(x, z)
    with pytest.raises(lcsm.LcsmError) as e:
        ctx.run_chain(x[:1], z[:1])
    assert e.value.code == lcsm.LCSM_EDONE
    lib = lcsm.raw()
    assert lib.lcsm_run_chain(None, 1, x.data_ptr(), 8, z.data_ptr(), 8) == lcsm.LCSM_EINVAL
    ctx.reset()
    assert lib.lcsm_run_chain(ctx._ctx, -1, x.data_ptr(), 8, z.data_ptr(), 8) == lcsm.LCSM_EINVAL
    assert lib.lcsm_run_chain(ctx._ctx, 0, x.data_ptr(), 8, z.data_ptr(), 8) == lcsm.LCSM_OK
    ctx.close()
