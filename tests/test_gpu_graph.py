"""Replayed generations (lcsm_graph_capture / lcsm_graph_launch) on the GPU:
the path the benchmark times (needs an MI355X).

A recorded generation is lcsm_reset plus n steps, split into HIP graphs of
a bounded number of positions (App. B.2's CUDA-graph dispatch, without one
graph's node count growing with the generation).  Checks:

* replays equal host-launched steps on the same ring inputs bit for bit,
  again on a second replay (the reset is inside the recording), for
  teacher-forced and chained inputs and for several segment lengths;
* the benchmark's own recording (a ring of 256 input slabs, graphs of 8192
  positions) on the 32768- and 131072-position workloads, every position of
  sampled columns against the fp64 oracle on the same ring-periodic inputs;
* argument errors leave the context usable.
"""
import numpy as np
import pytest
import torch

import datagen

from gpu_harness import TOL, dev, lcsm_mod, oracle_sampled, rel_err, say, say_maxima

pytestmark = pytest.mark.gpu

SHAPES = [(2, 3, 40, 300, None), (1, 2, 64, 1000, {"direct_max_u": 4}),
          (3, 2, 96, 4096, {"col_fft_min_n": 512})]


def _ctx(w, options=None, stream=None):
    lcsm = lcsm_mod()
    h = datagen.filters_torch(w, dev())
    return lcsm.Lcsm(h, w.B, options=options, stream=stream or torch.cuda.Stream(dev()))


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("seg", [1, 97, 0])
def test_replay_equals_host_launches(shape, seg):
    M, B, D, L, opts = shape
    say(f"[graph replay vs host] M={M} B={B} D={D} L={L} opts={opts} seg={seg}")
    w = datagen.Workload("graph", M, B, D, L, decay=L / 4, seed=M + B + D)
    R = 37
    y = datagen.y_torch(w, dev(), 0, R)
    ctx = _ctx(w, opts)
    # host launches, reading the ring the same way
    z_host = torch.empty((L, M, B, D), dtype=torch.float32, device=dev())
    with torch.cuda.stream(ctx.stream):
        ctx.reset()
        for t in range(L):
            ctx.step(y[t % R], z_host[t])
    torch.cuda.synchronize()
    z = torch.full_like(z_host, float("nan"))
    g = ctx.capture(y, z, n=L, seg=seg)
    expect = -(-L // (seg or lcsm_mod().GRAPH_DEFAULT_SEG))
    assert g.segments == expect
    assert ctx.position == L
    for rep in range(2):
        z.fill_(float("nan"))
        torch.cuda.synchronize()
        g.launch()
        torch.cuda.synchronize()
        assert ctx.position == L
        assert torch.equal(z, z_host), f"replay {rep} differs from host launches"
    g.close()
    ctx.close()


@pytest.mark.parametrize("shape,seg,ring", [((1, 1, 16, 1024), 128, 0), ((3, 2, 33, 300), 128, 0),
                                            ((2, 2, 20, 700), 97, 48)])
def test_replay_chain_equals_host_launches(shape, seg, ring):
    """The recorded chained steps (the small steps of each 32-position block
    in one launch) equal host-launched lcsm_step_chain bit for bit, on every
    replay; with 97-position graphs and a 48-slab input and output ring the
    graph boundaries and the ring's wrap fall inside blocks."""
    M, B, D, L = shape
    say(f"[graph replay, chain] M={M} B={B} D={D} L={L} seg={seg} ring={ring}")
    w = datagen.Workload("graphc", M, B, D, L, decay=200.0, seed=7)
    R = ring or L
    x = datagen.x_torch(w, dev(), 0, R)
    ctx = _ctx(w)
    z_host = torch.empty_like(x)
    with torch.cuda.stream(ctx.stream):
        ctx.reset()
        for t in range(L):
            ctx.step_chain(x[t % R], z_host[t % R])
    torch.cuda.synchronize()
    z = torch.full_like(x, float("nan"))
    g = ctx.capture(x, z, n=L, chain=True, seg=seg)
    for rep in range(2):
        z.fill_(float("nan"))
        g.launch()
        torch.cuda.synchronize()
        assert torch.equal(z, z_host), f"replay {rep} differs from host launches"
    g.close()
    ctx.close()


@pytest.mark.parametrize("name", ["m18b4d768l32k", "m18b1d1024l128k"])
def test_benchmark_recording_against_oracle(name):
    """The benchmark's recording: a ring of 256 input slabs, graphs of 8192
    positions (4 and 16 of them here).  Outputs go to a buffer of all L
    positions so that every position of the sampled columns is compared."""
    w = datagen.WORKLOADS[name]
    say(f"[benchmark recording vs oracle] {w.name} M={w.M} B={w.B} D={w.D} L={w.L}")
    R = 256
    y = datagen.y_torch(w, dev(), 0, R)
    z = torch.empty((w.L, w.M, w.B, w.D), dtype=torch.float32, device=dev())
    ctx = _ctx(w)
    g = ctx.capture(y, z, n=w.L, seg=8192)
    say(f"  {g.segments} graphs recorded")
    assert g.segments == w.L // 8192
    g.launch()
    torch.cuda.synchronize()
    cols = datagen.sample_columns(w, 48)
    m = torch.as_tensor(cols[:, 0], device=dev())
    b = torch.as_tensor(cols[:, 1], device=dev())
    d = torch.as_tensor(cols[:, 2], device=dev())
    zg = z[:, m, b, d].cpu().numpy()
    g.close()
    ctx.close()
    del z
    # the ring-periodic inputs the recording consumed: y at position t is slab t mod R
    yr = np.stack([datagen.y_np(w, t_idx=np.arange(R), m_idx=[mm], b_idx=[bb], d_idx=[dd])[:, 0, 0, 0]
                   for mm, bb, dd in cols], axis=1)
    y_cols = yr[np.arange(w.L) % R]
    zr = oracle_sampled(w, cols, y_cols=y_cols)
    err = rel_err(zg, zr)
    say(f"  rel err {err:.3e} over {len(cols)} columns x {w.L} positions")
    say_maxima(zg, zr, cols)
    assert err <= TOL


def test_capture_argument_errors():
    lcsm = lcsm_mod()
    w = datagen.Workload("graphe", 1, 2, 8, 64, decay=16.0, seed=3)
    y = datagen.y_torch(w, dev(), 0, 4)
    z = torch.empty_like(y)
    ctx = _ctx(w)
    for kw in ({"n": 0}, {"n": w.L + 1}, {"seg": lcsm.GRAPH_MAX_SEG + 1}, {"seg": -3}):
        with pytest.raises(lcsm.LcsmError) as e:
            ctx.capture(y, z, **kw)
        assert e.value.code == lcsm.LCSM_EINVAL
    # the null stream cannot be captured
    h = datagen.filters_torch(w, dev())
    ctx0 = lcsm.Lcsm(h, w.B, stream=torch.cuda.default_stream(dev()))
    if ctx0.stream.cuda_stream == 0:
        with pytest.raises(lcsm.LcsmError) as e:
            ctx0.capture(y, z)
        assert e.value.code == lcsm.LCSM_EINVAL
    ctx0.close()
    # still usable after the rejected calls
    g = ctx.capture(y, z, n=w.L)
    g.launch()
    torch.cuda.synchronize()
    z_ref = torch.empty_like(y)
    with torch.cuda.stream(ctx.stream):
        ctx.reset()
        for t in range(w.L):
            ctx.step(y[t % 4], z_ref[t % 4])
    torch.cuda.synchronize()
    assert torch.equal(z, z_ref)
    g.close()
    ctx.close()


def test_launch_after_host_steps_continues_correctly():
    """A replay starts with a reset whatever the context did before: host
    steps past the recorded length, then the replay, then host steps from
    there must equal an all-host run (the mirror's copy bookkeeping follows
    the replay, not the host steps before it)."""
    M, B, D, L = 2, 4, 48, 2048
    w = datagen.Workload("graphm", M, B, D, L, decay=L / 4, seed=17)
    opts = {"direct_max_u": 4, "col_fft_min_n": 16}   # mirrored tiles from U = 8
    lcsm = lcsm_mod()
    assert lcsm.plan_tile(M, B, D, L, 7, opts)[3] == lcsm.TILE_FFT_CM
    say(f"[graph launch after host steps] M={M} B={B} D={D} L={L} opts={opts}")
    y = datagen.y_torch(w, dev())
    ctx = _ctx(w, opts)
    z_ref = torch.empty_like(y)
    with torch.cuda.stream(ctx.stream):
        ctx.reset()
        for t in range(L):
            ctx.step(y[t], z_ref[t])
    torch.cuda.synchronize()
    n = 600
    z = torch.full_like(y, float("nan"))
    g = ctx.capture(y, z, n=n, seg=256)
    with torch.cuda.stream(ctx.stream):
        ctx.reset()
        scratch = torch.empty_like(y[0])
        for t in range(1500):                    # well past n, across mirror boundaries
            ctx.step(y[t], scratch)
    g.launch()
    assert ctx.position == n
    with torch.cuda.stream(ctx.stream):
        for t in range(n, L):
            ctx.step(y[t], z[t])
    torch.cuda.synchronize()
    assert torch.equal(z, z_ref)
    g.close()
    ctx.close()
