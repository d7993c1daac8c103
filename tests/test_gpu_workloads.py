"""Full-size workloads on the GPU: teacher-forced parity on sampled columns
against the fp64 static-FFT oracle (needs an MI355X).

All L positions of all layers, batch rows and channels are computed by the
library in the launch configuration the benchmark uses; the oracle checks a
fixed sample of columns that includes the batch/channel boundaries of the
first and last layer."""
import pytest

import datagen
from gpu_harness import TOL, make_ctx, oracle_sampled, rel_err, run_sampled, say, say_maxima

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["m18b4d768l32k", "m18b1d1024l128k", "m32b16d2048l16k"])
def test_workload_sampled_columns(name):
    w = datagen.WORKLOADS[name]
    say(f"[sampled parity] {w.name} M={w.M} B={w.B} D={w.D} L={w.L}")
    cols = datagen.sample_columns(w, 48)
    ctx, filters = make_ctx(w)
    z = run_sampled(ctx, w, cols, chunk=128)
    del filters
    ctx.close()
    zr = oracle_sampled(w, cols)
    err = rel_err(z, zr)
    say(f"  rel err {err:.3e} over {len(cols)} columns")
    say_maxima(z, zr, cols)
    assert err <= TOL


@pytest.mark.parametrize("D", [16, 3])
def test_maximum_length(D):
    """L = 2^19, the longest sequence the library accepts: every tile size up
    to U = 2^18 runs, the largest through the longest three-pass split
    (4096-point rows, 128-point columns).  16 channels make every panel whole
    (the fast kernels); 3 channels leave panels partial (the general ones).
    All columns are checked against the fp64 static-FFT oracle."""
    import numpy as np

    w = datagen.Workload("maxlen", 1, 1, D, 1 << 19, decay=65536.0, seed=11)
    say(f"[maximum length] M={w.M} B={w.B} D={w.D} L={w.L}")
    cols = np.array([(0, 0, d) for d in range(D)], dtype=np.int64)
    ctx, filters = make_ctx(w)
    z = run_sampled(ctx, w, cols, chunk=4096)
    del filters
    ctx.close()
    zr = oracle_sampled(w, cols)
    err = rel_err(z, zr)
    say(f"  rel err {err:.3e} over {len(cols)} columns")
    assert err <= TOL
