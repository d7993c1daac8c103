"""GPU parity of the fused-caller views (lcsm_h0, lcsm_pending, lcsm_commit,
lcsm_tile; needs an MI355X).

A caller that does the red cell in its own kernel reads the pending
accumulators of position t, computes z_t = h0 * y_t + acc_t, writes y_t over
the pending row and commits.  Bars: the lag-0 view equals the filters' first
taps bit for bit; at every position the pending accumulators equal those of
a context driven by lcsm_step_layer / lcsm_advance on the same inputs bit for
bit (the slots receive y_t either way and the gray tiles are the same
launches); the outputs agree with that context's to the rounding of the
final multiply-add, and with the fp64 oracle to max|z_gpu - z_ref| <=
1e-4 * max|z_ref|.  The per-context schedule query equals the shape query.
"""
import numpy as np
import pytest
import torch

import datagen
from oracle import conv
from oracle.relaxed import filters_to_columns

from gpu_harness import TOL, dev, lcsm_mod, make_ctx, rel_err, say

pytestmark = pytest.mark.gpu

OPTIONS = {
    "default": {},
    "fft_from_2": {"direct_max_u": 1, "col_fft_min_n": 1 << 20},
    "col_from_4": {"direct_max_u": 1, "col_fft_min_n": 4},
    "colT_from_4": {"direct_max_u": 1, "col_fft_min_n": 4, "col_tile_form": 1},
}


@pytest.mark.parametrize("half", [False, True])
@pytest.mark.parametrize("opt", ["default", "fft_from_2", "col_from_4", "colT_from_4"])
def test_pending_commit_equals_step(opt, half):
    M, B, D, L = 2, 3, 40, 700
    say(f"[fused caller] M={M} B={B} D={D} L={L} options={opt} half_state={half}")
    w = datagen.Workload("fused", M, B, D, L, decay=L / 4, seed=31)
    filt = datagen.filters_torch(w, dev())
    opts = dict(OPTIONS[opt], half_state=int(half))
    ref, _ = make_ctx(w, filt, opts)
    fc, _ = make_ctx(w, filt, opts)
    h0 = fc.h0()
    assert tuple(h0.shape) == (M, D)
    assert torch.equal(h0, filt[:, :, 0])
    y = datagen.y_torch(w, dev())
    za = torch.empty_like(y)
    zb = torch.empty_like(y)
    for t in range(L):
        acc = fc.pending()
        if t % 37 == 0 or t in (L // 2, L - 1):
            assert torch.equal(acc, ref.pending()), f"pending rows differ at t={t}"
        torch.addcmul(acc, h0[:, None, :], y[t], out=zb[t])
        acc.copy_(y[t])
        fc.commit()
        for m in range(M):
            ref.step_layer(m, y[t, m], za[t, m])
        ref.advance()
    torch.cuda.synchronize()
    assert fc.position == L == ref.position
    a, b = za.cpu().numpy(), zb.cpu().numpy()
    scale = np.abs(a).max()
    diff = np.abs(a - b).max()
    say(f"  max |layer path - fused| {diff:.3e} (scale {scale:.3e})")
    assert diff <= 4 * np.finfo(np.float32).eps * scale
    hcol = filters_to_columns(datagen.filters_np(w), B)
    zr = conv.causal_conv_fft(y.cpu().numpy().reshape(L, -1).astype(np.float64),
                              hcol.reshape(hcol.shape[0], -1))
    err = rel_err(b.reshape(L, -1), zr)
    say(f"  rel err vs oracle {err:.3e}")
    assert err <= TOL


def test_fused_caller_errors_and_schedule():
    lcsm = lcsm_mod()
    w = datagen.Workload("fusederr", 2, 2, 24, 300, decay=50.0, seed=8)
    ctx, _ = make_ctx(w)
    for t in range(w.L):
        assert ctx.tile(t) == ctx.plan(t)
    with pytest.raises(lcsm.LcsmError) as ex:
        ctx.tile(w.L)
    assert ex.value.code == lcsm.LCSM_EINVAL
    # commit between per-layer steps is refused and leaves the position alone
    y = datagen.y_torch(w, dev(), 0, 1)
    ctx.step_layer(0, y[0, 0].contiguous())
    with pytest.raises(lcsm.LcsmError) as ex:
        ctx.commit()
    assert ex.value.code == lcsm.LCSM_ESTATE
    assert ctx.position == 0
    ctx.step_layer(1, y[0, 1].contiguous())
    ctx.advance()
    assert ctx.position == 1
    # the pending view is gone once the run is over
    ctx.reset()
    ys = datagen.y_torch(w, dev())
    ctx.run(ys, torch.empty_like(ys))
    with pytest.raises(lcsm.LcsmError) as ex:
        ctx.pending()
    assert ex.value.code == lcsm.LCSM_EDONE
    with pytest.raises(lcsm.LcsmError) as ex:
        ctx.commit()
    assert ex.value.code == lcsm.LCSM_EDONE
    torch.cuda.synchronize()
