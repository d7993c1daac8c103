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


def chunk_edge_columns(w, scratch_mib=512):
    """Columns on both sides of every scratch-chunk boundary of the column
    tiles (library defaults: a scratch of scratch_mib MiB, U floats per
    column, chunks rounded down to 64 columns and, where a chunk holds at
    least one layer of B*D columns, to whole layers).  Global column
    g = m*B*D + b*D + d; the last column before and the first after each
    boundary are returned as (m, b, d) triples, for the tile sizes of the
    workload that run on column chunks (2U = 4096 ... 16384 here)."""
    import numpy as np
    BD, total = w.B * w.D, w.M * w.B * w.D
    edges = set()
    for N in (4096, 8192, 16384):
        if N // 2 >= w.L:
            continue
        U = N // 2
        chunk = (scratch_mib << 20) // (4 * U) // 64 * 64
        chunk = min(chunk, -(-total // 64) * 64)
        if BD % 64 == 0 and chunk >= BD:
            chunk = chunk // BD * BD
        for g0 in range(chunk, total, chunk):
            for g in (g0 - 1, g0):
                m, c = divmod(g, BD)
                edges.add((m, c // w.D, c % w.D))
    # a bounded subset: the first two and the last two boundaries' columns
    # plus every one inside the second layer
    edges = sorted(edges)
    keep = set(edges[:4] + edges[-4:]) | {e for e in edges if e[0] == 1}
    return np.array(sorted(keep), dtype=np.int64).reshape(-1, 3)


@pytest.mark.parametrize("name", ["m18b4d768l32k", "m18b1d1024l128k", "m32b16d2048l16k"])
def test_workload_sampled_columns(name):
    import numpy as np
    w = datagen.WORKLOADS[name]
    say(f"[sampled parity] {w.name} M={w.M} B={w.B} D={w.D} L={w.L}")
    cols = datagen.sample_columns(w, 48)
    edges = chunk_edge_columns(w)
    if len(edges):
        cols = np.unique(np.concatenate([cols, edges]), axis=0)
        say(f"  + {len(edges)} columns at scratch-chunk boundaries of the column tiles")
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
