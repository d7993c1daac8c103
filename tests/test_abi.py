"""The C ABI loads, exports what include/*.h declare, validates arguments
on the host and plans the same tiles as the oracle's schedule -- CPU only
(no call here reaches the device)."""
import ctypes
import os
import re

import pytest

from oracle.schedule import tile_after_step

import paper_2410_12982_amd.lcsm as lcsm  # noqa: E402  (built by conftest if missing)

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    import glob
    names = set()
    for path in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = re.sub(r"/\*.*?\*/", "", open(path).read(), flags=re.S)
        names |= set(re.findall(r"\b(lcsm_[a-z0-9_]+)\s*\(", text))
    return sorted(names)


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert len(names) >= 19
    lib = lcsm.raw()
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(lcsm.EXPORTED) == names


@pytest.mark.parametrize("L", [1, 2, 3, 12, 100, 1024, 8192])
def test_plan_tile_matches_oracle_schedule(L):
    for t in range(L):
        i, U, n, kind = lcsm.plan_tile(1, 1, 1, L, t)
        want = tile_after_step(t, L)
        if want is None:
            assert (i, U, n, kind) == (0, 0, 0, lcsm.TILE_NONE)
        else:
            wi, wU, s0, s1, d0, d1 = want
            assert (i, U, n) == (wi, wU, d1 - d0)
            assert kind != lcsm.TILE_NONE


def test_plan_tile_large_L_every_step():
    L = 1 << 17
    for t in range(0, L, 97):
        i, U, n, _ = lcsm.plan_tile(18, 1, 1024, L, t)
        want = tile_after_step(t, L)
        assert want is None or (i, U, n) == (want[0], want[1], want[5] - want[4])


def test_tile_kind_selection_follows_options():
    o = {"direct_max_u": 8, "lds_fft_max_n": 64}
    kinds = {}
    for t in range(1023):
        _, U, _, k = lcsm.plan_tile(1, 1, 4, 1024, t, o)
        kinds[U] = k
    assert all(kinds[u] == lcsm.TILE_DIRECT for u in (1, 2, 4, 8))
    assert all(kinds[u] == lcsm.TILE_FFT for u in (16, 32))
    assert all(kinds[u] == lcsm.TILE_FFT_HBM for u in (64, 128, 256, 512))


@pytest.mark.parametrize("shape", [(0, 1, 1, 8), (1, 0, 1, 8), (1, 1, 0, 8), (1, 1, 1, 0),
                                   (1, 1, 1, -5), (1 << 16, 1 << 8, 1 << 8, 8), (1, 1, 1, 1 << 30),
                                   (16385, 1, 1, 8), (1, 65536, 1, 8), (1, 1, 1, (1 << 19) + 1)])
def test_workspace_bytes_rejects_bad_shapes(shape):
    with pytest.raises(lcsm.LcsmError) as e:
        lcsm.workspace_bytes(*shape)
    assert e.value.code == lcsm.LCSM_EINVAL


def test_workspace_bytes_covers_state_and_filters():
    M, B, D, L = 3, 4, 40, 300
    n = lcsm.workspace_bytes(M, B, D, L)
    assert n >= 4 * (M * L * B * D + M * L * D)
    assert n % 256 == 0


@pytest.mark.parametrize("opts", [{"direct_max_u": 3}, {"lds_fft_max_n": 100},
                                  {"direct_max_u": -1}, {"lds_fft_max_n": 8},
                                  {"lds_fft_max_n": 16384}, {"scratch_mib": -1}])
def test_bad_options_rejected(opts):
    with pytest.raises(lcsm.LcsmError) as e:
        lcsm.workspace_bytes(1, 1, 1, 16, opts)
    assert e.value.code == lcsm.LCSM_EINVAL


def test_reserved_options_must_be_zero():
    o = lcsm.Options()
    o.reserved[1] = 1
    with pytest.raises(lcsm.LcsmError):
        lcsm.workspace_bytes(1, 1, 1, 16, o)


def test_options_struct_matches_header():
    text = open(os.path.join(ROOT, "include", "lcsm.h")).read()
    body = text[text.index("typedef struct lcsm_options"):text.index("} lcsm_options;")]
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    fields = re.findall(r"int\s+([a-z_]+)(?:\[(\d+)\])?;", body)
    assert [f for f, _ in fields] == [f for f, _ in lcsm.Options._fields_]
    assert ctypes.sizeof(lcsm.Options) == 32


@pytest.mark.parametrize("L,T", [(4096, 2048), (1000, 512), (513, 512), (8192, 4096)])
def test_half_state_saves_the_rows_past_T(L, T):
    """Half-state storage (App. C): T = the largest power of two below L
    state rows per layer instead of L; everything else is unchanged."""
    M, B, D = 3, 4, 40
    full = lcsm.workspace_bytes(M, B, D, L)
    half = lcsm.workspace_bytes(M, B, D, L, {"half_state": 1})
    saved = 4 * M * (L - T) * B * D
    assert abs((full - half) - saved) < 256
    # the schedule does not change
    for t in (0, T - 2, T - 1, T, L - 2, L - 1):
        assert lcsm.plan_tile(M, B, D, L, t, {"half_state": 1}) == lcsm.plan_tile(M, B, D, L, t)


@pytest.mark.parametrize("L,opts", [(128, {}), (64, {}), (1, {}), (2, {}),
                                    (4096, {"direct_max_u": 2048}),
                                    (4096, {"direct_max_u": 1 << 20})])
def test_half_state_needs_an_fft_swap_tile(L, opts):
    """The tile of side T overwrites its own inputs, which only the FFT
    tiles can do: a direct tile of side T is rejected, as is L < 2."""
    o = dict(opts, half_state=1)
    with pytest.raises(lcsm.LcsmError) as e:
        lcsm.workspace_bytes(1, 1, 16, L, o)
    assert e.value.code == lcsm.LCSM_EINVAL
    with pytest.raises(lcsm.LcsmError):
        lcsm.plan_tile(1, 1, 16, max(L, 2), 0, o)


def test_half_state_flag_is_0_or_1():
    for v in (2, -1, 7):
        with pytest.raises(lcsm.LcsmError) as e:
            lcsm.workspace_bytes(1, 1, 16, 4096, {"half_state": v})
        assert e.value.code == lcsm.LCSM_EINVAL
    # the smallest lengths it takes with the default crossover (T = 128 > 64)
    lcsm.workspace_bytes(1, 1, 16, 129, {"half_state": 1})
    lcsm.workspace_bytes(1, 1, 16, 256, {"half_state": 1})


def test_workspace_grows_with_fft_levels():
    M, B, D, L = 2, 4, 96, 4096
    direct = lcsm.workspace_bytes(M, B, D, L, {"direct_max_u": 1 << 20})
    fft = lcsm.workspace_bytes(M, B, D, L)
    # spectra of U = 128..2048: M * (U+1) * D complex values each
    spectra = sum(8 * M * (u + 1) * D for u in (128, 256, 512, 1024, 2048))
    assert fft >= direct + spectra
    # the multi-pass scratch obeys the cap but never drops below one chunk
    small = lcsm.workspace_bytes(M, B, D, L, {"lds_fft_max_n": 16, "scratch_mib": 1})
    big = lcsm.workspace_bytes(M, B, D, L, {"lds_fft_max_n": 16, "scratch_mib": 4096})
    assert small < big
    assert small >= direct + spectra + 8 * 4096 * 16


def test_plan_tile_default_kinds_for_workloads():
    # default at 18432 columns: direct up to U = 32, one LDS pass up to 2U = 1024,
    # the column-tile sizes 2U = 2048 ... 32768 (the last as two halves) on the
    # column-major mirror, multi-pass above
    L = 1 << 17
    kinds = {}
    for t in range(L - 1):
        _, U, _, k = lcsm.plan_tile(18, 1, 1024, L, t)
        kinds[U] = k
    assert all(kinds[1 << q] == lcsm.TILE_DIRECT for q in range(6))
    assert all(kinds[1 << q] == lcsm.TILE_FFT for q in range(6, 10))
    assert all(kinds[1 << q] == lcsm.TILE_FFT_CM for q in range(10, 15))
    assert all(kinds[1 << q] == lcsm.TILE_FFT_HBM for q in range(15, 17))
    # the transposed column chunks instead when asked for, and with half-state:
    # from 2U = 8192 (4096 from 2^15 columns)
    for opts in ({"col_tile_form": 1}, {"half_state": 1}):
        for q in range(10, 12):
            assert lcsm.plan_tile(18, 1, 1024, L, (1 << q) - 1, opts)[3] == lcsm.TILE_FFT
        for q in range(12, 15):
            assert lcsm.plan_tile(18, 1, 1024, L, (1 << q) - 1, opts)[3] == lcsm.TILE_FFT_COL
        for shape in ((18, 4, 768, 32768), (32, 16, 2048, 16384)):
            assert lcsm.plan_tile(*shape, 2047, opts)[3] == lcsm.TILE_FFT_COL
            assert lcsm.plan_tile(*shape, 1023, opts)[3] == lcsm.TILE_FFT
    # fewer than 2^14 columns (the 6144-column workload): no column tiles
    assert lcsm.plan_tile(1, 8, 768, 8192, 4095)[3] == lcsm.TILE_FFT
    for shape in ((18, 4, 768, 32768), (32, 16, 2048, 16384), (1, 1, 32768, 8192)):
        assert lcsm.plan_tile(*shape, 1023)[3] == lcsm.TILE_FFT_CM
        assert lcsm.plan_tile(*shape, 511)[3] == lcsm.TILE_FFT
    assert lcsm.plan_tile(1, 1, 16383, 8192, 1023)[3] == lcsm.TILE_FFT
    # the column tiles when asked for: 2U from col_fft_min_n up to 32768
    on = {"col_fft_min_n": 4096}
    for q, want in ((10, lcsm.TILE_FFT), (11, lcsm.TILE_FFT_CM), (13, lcsm.TILE_FFT_CM),
                    (14, lcsm.TILE_FFT_CM), (15, lcsm.TILE_FFT_HBM)):
        t = (1 << q) - 1
        assert lcsm.plan_tile(18, 1, 1024, L, t, on)[3] == want
    for bad in (3, 2, -4, 100):
        with pytest.raises(lcsm.LcsmError):
            lcsm.workspace_bytes(1, 1, 16, 4096, {"col_fft_min_n": bad})
    for bad in (2, -1):
        with pytest.raises(lcsm.LcsmError):
            lcsm.workspace_bytes(1, 1, 16, 4096, {"col_tile_form": bad})


@pytest.mark.parametrize("shape", [(18, 4, 768, 32768), (3, 1, 7, 4096), (2, 5, 3, 1000)])
def test_mirror_memory(shape):
    """The column-major mirror holds M * ceil(B*D/2) pairs of L complex
    values (batch pairs when B is even, neighbouring columns otherwise):
    the workspace grows by that much over the transposed column tiles."""
    M, B, D, L = shape
    opts = {"col_fft_min_n": 256}
    mirror = lcsm.workspace_bytes(M, B, D, L, opts)
    transposed = lcsm.workspace_bytes(M, B, D, L, dict(opts, col_tile_form=1))
    pairs = (B // 2) * D if B % 2 == 0 else (B * D + 1) // 2
    assert 0 <= (mirror - transposed) - 8 * M * pairs * L < 512


def test_init_validates_before_touching_the_device():
    lib = lcsm.raw()
    ctx = ctypes.c_void_p(123)
    fake = ctypes.c_void_p(4096)
    # null out-pointer, null filters, bad shape, too-small or misaligned workspace
    assert lib.lcsm_init(None, fake, 1, 1, 1, 8, None, None, 0, None) == lcsm.LCSM_EINVAL
    assert lib.lcsm_init(ctypes.byref(ctx), None, 1, 1, 1, 8, None, None, 0, None) == lcsm.LCSM_EINVAL
    assert ctx.value is None
    assert lib.lcsm_init(ctypes.byref(ctx), fake, 1, 0, 1, 8, None, None, 0, None) == lcsm.LCSM_EINVAL
    need = lcsm.workspace_bytes(1, 1, 1, 8)
    assert lib.lcsm_init(ctypes.byref(ctx), fake, 1, 1, 1, 8, None, fake, need - 1, None) == lcsm.LCSM_ENOMEM
    assert lib.lcsm_init(ctypes.byref(ctx), fake, 1, 1, 1, 8, None, ctypes.c_void_p(4096 + 4),
                         need, None) == lcsm.LCSM_EINVAL


def test_null_context_calls():
    lib = lcsm.raw()
    fake = ctypes.c_void_p(4096)
    assert lib.lcsm_step(None, fake, fake) == lcsm.LCSM_EINVAL
    assert lib.lcsm_step_chain(None, fake, fake) == lcsm.LCSM_EINVAL
    assert lib.lcsm_step_layer(None, 0, fake, fake) == lcsm.LCSM_EINVAL
    assert lib.lcsm_advance(None) == lcsm.LCSM_EINVAL
    assert lib.lcsm_reset(None) == lcsm.LCSM_EINVAL
    assert lib.lcsm_run(None, 1, fake, 0, fake, 0) == lcsm.LCSM_EINVAL
    assert lib.lcsm_run_chain(None, 1, fake, 0, fake, 0) == lcsm.LCSM_EINVAL
    assert lib.lcsm_run_noalloc(None, 1, fake, 0, fake, 0) == lcsm.LCSM_EINVAL
    t = ctypes.c_int()
    assert lib.lcsm_position(None, ctypes.byref(t)) == lcsm.LCSM_EINVAL
    i, U, n, k = (ctypes.c_int() for _ in range(4))
    assert lib.lcsm_tile(None, 0, ctypes.byref(i), ctypes.byref(U), ctypes.byref(n),
                         ctypes.byref(k)) == lcsm.LCSM_EINVAL
    p, st = ctypes.c_void_p(), ctypes.c_size_t()
    assert lib.lcsm_h0(None, ctypes.byref(p), ctypes.byref(st)) == lcsm.LCSM_EINVAL
    assert lib.lcsm_pending(None, ctypes.byref(p), ctypes.byref(st)) == lcsm.LCSM_EINVAL
    assert lib.lcsm_commit(None) == lcsm.LCSM_EINVAL
    g = ctypes.c_void_p(1234)
    assert lib.lcsm_graph_capture(None, 0, 8, fake, 0, 0, fake, 0, 0, 0,
                                  ctypes.byref(g)) == lcsm.LCSM_EINVAL
    assert g.value is None  # *out is cleared before any other check
    assert lib.lcsm_graph_launch(None) == lcsm.LCSM_EINVAL
    assert lib.lcsm_graph_segments(None, ctypes.byref(t)) == lcsm.LCSM_EINVAL
    lib.lcsm_graph_destroy(None)
    lib.lcsm_destroy(None)
    assert lib.lcsm_last_error(None) == b""


def test_strerror_covers_codes():
    seen = {lcsm.strerror(c) for c in (0, -1, -2, -3, -4, -5)}
    assert len(seen) == 6
    assert lcsm.strerror(-99) == "unknown error code"


def test_single_hip_runtime_in_process():
    """The binding binds to torch's HIP runtime; a second copy must not load."""
    assert len(lcsm.hip_runtimes()) <= 1


def test_default_crossover_depends_on_shape():
    """Direct tiles up to U = 32 always; U = 64 direct only below 2^14 columns
    (small launches are latency-bound; from 2^14 columns the FFT tile of
    2U = 128 runs in wide panels and is faster), FFT above."""
    def kind_at_u(M, B, D, L, u):
        # the tile after step t = u - 1 has i = u, side lowbit(u) = u
        return lcsm.plan_tile(M, B, D, L, u - 1)[3]
    for shape in [(1, 8, 768, 8192), (1, 1, 16383, 1024)]:
        assert kind_at_u(*shape, 32) == lcsm.TILE_DIRECT
        assert kind_at_u(*shape, 64) == lcsm.TILE_DIRECT
        assert kind_at_u(*shape, 128) == lcsm.TILE_FFT
    for shape in [(18, 4, 768, 32768), (18, 1, 1024, 1 << 17), (1, 1, 16384, 1024)]:
        assert kind_at_u(*shape, 32) == lcsm.TILE_DIRECT
        assert kind_at_u(*shape, 64) == lcsm.TILE_FFT
        assert kind_at_u(*shape, 128) == lcsm.TILE_FFT
    wide = (32, 16, 2048, 16384)
    assert kind_at_u(*wide, 32) == lcsm.TILE_DIRECT
    assert kind_at_u(*wide, 64) == lcsm.TILE_FFT
    # an explicit option overrides the shape rule
    assert lcsm.plan_tile(*wide, 63, {"direct_max_u": 64})[3] == lcsm.TILE_DIRECT


def test_synth_init_validates_before_touching_the_device():
    """lcsm_synth_init rejects null pointers, D not a multiple of 4 and what
    lcsm_init rejects, without any device work."""
    lib = lcsm.raw()
    out = ctypes.c_void_p()
    p = ctypes.c_void_p(256)  # never dereferenced: validation fails first
    assert lib.lcsm_synth_init(None, p, p, p, p, p, 1, 1, 16, 64, None, None) == lcsm.LCSM_EINVAL
    assert lib.lcsm_synth_init(ctypes.byref(out), None, p, p, p, p, 1, 1, 16, 64, None,
                               None) == lcsm.LCSM_EINVAL
    assert lib.lcsm_synth_init(ctypes.byref(out), p, p, p, None, p, 1, 1, 16, 64, None,
                               None) == lcsm.LCSM_EINVAL
    for D in (1, 2, 6, 18):
        assert lib.lcsm_synth_init(ctypes.byref(out), p, p, p, p, p, 1, 1, D, 64, None,
                                   None) == lcsm.LCSM_EINVAL
    assert lib.lcsm_synth_init(ctypes.byref(out), p, p, p, p, p, 0, 1, 16, 64, None,
                               None) == lcsm.LCSM_EINVAL
    o = lcsm.Options()
    o.half_state = 1
    assert lib.lcsm_synth_init(ctypes.byref(out), p, p, p, p, p, 1, 1, 16, 64, None,
                               ctypes.byref(o)) == lcsm.LCSM_EINVAL
    assert not out.value
    for f in (lib.lcsm_synth_step, ):
        assert f(None, p, p) == lcsm.LCSM_EINVAL
    assert lib.lcsm_synth_reset(None) == lcsm.LCSM_EINVAL
    assert lib.lcsm_synth_position(None, ctypes.byref(ctypes.c_int())) == lcsm.LCSM_EINVAL
    lib.lcsm_synth_destroy(None)
    assert lib.lcsm_synth_last_error(None) == b""


def test_dd_workspace_and_validation():
    """Data-dependent contexts: two state arrays; options checked; tiles
    wider than one LDS pass accepted (run as block pairs) -- all host-side."""
    M, B, D, L = 2, 3, 16, 1000
    n = lcsm.dd_workspace_bytes(M, B, D, L)
    assert n >= 2 * 4 * M * L * B * D and n % 256 == 0
    for opts in ({"half_state": 1}, {"scratch_mib": 4}, {"direct_max_u": 3},
                 {"lds_fft_max_n": 100}, {"lds_fft_max_n": 16384}):
        with pytest.raises(lcsm.LcsmError) as e:
            lcsm.dd_workspace_bytes(M, B, D, L, opts)
        assert e.value.code == lcsm.LCSM_EINVAL
    o = lcsm.Options()
    o.reserved[1] = 5
    with pytest.raises(lcsm.LcsmError):
        lcsm.dd_workspace_bytes(M, B, D, L, o)
    # tiles wider than one LDS pass run as block pairs: any length is accepted, and the
    # twiddle table stops at the single-pass transform (8192 points, 64 KiB)
    state = 2 * 4 * 131072 * 16
    n = lcsm.dd_workspace_bytes(1, 1, 16, 131072)
    assert state < n <= state + 8 * 2 * 8192 + 256
    assert lcsm.dd_workspace_bytes(1, 1, 16, 16385) > lcsm.dd_workspace_bytes(1, 1, 16, 16384)
    lcsm.dd_workspace_bytes(1, 1, 16, 16385, {"direct_max_u": 8192})
    small = lcsm.dd_workspace_bytes(1, 1, 16, 4096, {"lds_fft_max_n": 1024})  # U = 1024: 2x2 blocks
    assert small <= 2 * 4 * 4096 * 16 + 8 * 2 * 1024 + 256
    for shape in ((0, 1, 1, 8), (1, 1, 1, 0), (16385, 1, 1, 8)):
        with pytest.raises(lcsm.LcsmError):
            lcsm.dd_workspace_bytes(*shape)
    lib = lcsm.raw()
    out = ctypes.c_void_p()
    assert lib.lcsm_dd_init(None, 1, 1, 16, 64, None, None, 0, None) == lcsm.LCSM_EINVAL
    assert lib.lcsm_dd_init(ctypes.byref(out), 1, 1, 16, 64, None, ctypes.c_void_p(256), 16,
                            None) == lcsm.LCSM_ENOMEM
    assert lib.lcsm_dd_init(ctypes.byref(out), 1, 1, 16, 64, None, ctypes.c_void_p(260), 1 << 20,
                            None) == lcsm.LCSM_EINVAL
    assert not out.value
    p = ctypes.c_void_p(256)
    assert lib.lcsm_dd_step(None, p, p, p) == lcsm.LCSM_EINVAL
    assert lib.lcsm_dd_reset(None) == lcsm.LCSM_EINVAL
    assert lib.lcsm_dd_position(None, ctypes.byref(ctypes.c_int())) == lcsm.LCSM_EINVAL
    lib.lcsm_dd_destroy(None)
    assert lib.lcsm_dd_last_error(None) == b""


def test_base_workspace_and_validation():
    """The lazy/eager baselines (include/lcsm_base.h): workspace sizes and
    argument checks, on the host."""
    M, B, D, L = 3, 2, 40, 1000
    lazy = lcsm.base_workspace_bytes(lcsm.BASE_LAZY, M, B, D, L)
    eager = lcsm.base_workspace_bytes(lcsm.BASE_EAGER, M, B, D, L)
    state, filt = 4 * M * L * B * D, 4 * M * L * D
    assert eager >= state + filt and eager - (state + filt) < 1024
    # lazy also holds ceil(L/256) partial sums per column
    assert lazy - eager >= 4 * 4 * M * B * D
    assert lcsm.base_workspace_bytes(lcsm.BASE_LAZY | lcsm.BASE_NP, M, B, D, L) == lazy
    for kind, shape in ((4, (1, 1, 1, 8)), (-1, (1, 1, 1, 8)), (0, (0, 1, 1, 8)),
                        (0, (1, 1, 1, (1 << 19) + 1)), (1, (1, 1 << 16, 1, 8))):
        with pytest.raises(lcsm.LcsmError) as e:
            lcsm.base_workspace_bytes(kind, *shape)
        assert e.value.code == lcsm.LCSM_EINVAL
    lib = lcsm.raw()
    ctx = ctypes.c_void_p(1234)
    fake = ctypes.c_void_p(4096)
    assert lib.lcsm_base_init(ctypes.byref(ctx), 0, None, 1, 1, 1, 8, None, None, 0) == lcsm.LCSM_EINVAL
    assert ctx.value is None
    assert lib.lcsm_base_init(ctypes.byref(ctx), 7, fake, 1, 1, 1, 8, None, None, 0) == lcsm.LCSM_EINVAL
    need = lcsm.base_workspace_bytes(0, 1, 1, 1, 8)
    assert lib.lcsm_base_init(ctypes.byref(ctx), 0, fake, 1, 1, 1, 8, None, fake,
                              need - 1) == lcsm.LCSM_ENOMEM
    assert lib.lcsm_base_step(None, fake, fake) == lcsm.LCSM_EINVAL
    assert lib.lcsm_base_reset(None) == lcsm.LCSM_EINVAL
    t = ctypes.c_int()
    assert lib.lcsm_base_position(None, ctypes.byref(t)) == lcsm.LCSM_EINVAL
    lib.lcsm_base_destroy(None)
    assert lib.lcsm_base_last_error(None) == b""
