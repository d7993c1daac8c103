"""Python binding of the C ABI in ``include/lcsm.h``, ``lcsm_base.h``, ``lcsm_dd.h`` and ``lcsm_synth.h`` (ctypes).

Argument marshalling only: every step of the computation runs in the HIP
kernels of ``liblcsm.so``.  PyTorch supplies device memory (the workspace and
the caller's tensors) and the stream.  If the library has not been built the
import of this module fails; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
import weakref

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "liblcsm.so")

LCSM_OK = 0
LCSM_EINVAL = -1
LCSM_ENOMEM = -2
LCSM_EDEVICE = -3
LCSM_EDONE = -4
LCSM_ESTATE = -5

TILE_NONE, TILE_DIRECT, TILE_FFT, TILE_FFT_HBM, TILE_FFT_COL, TILE_FFT_CM = 0, 1, 2, 3, 4, 5
GRAPH_CHAIN = 1
BASE_LAZY, BASE_EAGER, BASE_NP = 0, 1, 2
BASE_KINDS = {"lazy": BASE_LAZY, "lazy_np": BASE_LAZY | BASE_NP, "eager": BASE_EAGER,
              "eager_np": BASE_EAGER | BASE_NP}
GRAPH_DEFAULT_SEG, GRAPH_MAX_SEG = 8192, 16384
TILE_KIND_NAMES = {TILE_NONE: "none", TILE_DIRECT: "direct", TILE_FFT: "fft_lds",
                   TILE_FFT_HBM: "fft_hbm", TILE_FFT_COL: "fft_col", TILE_FFT_CM: "fft_cm"}

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2410_12982_amd.build`")

# torch brings its own HIP runtime (libamdhip64, soname libamdhip64.so.7).  It
# must be mapped before liblcsm.so is opened, so that the library binds to the
# same runtime instance as the tensors it is handed; opened first, liblcsm.so
# would pull in the system runtime and the process would hold two.
import torch  # noqa: E402,F401

_lib = ctypes.CDLL(LIB_PATH)


def hip_runtimes():
    """Paths of the HIP runtime libraries mapped into this process."""
    try:
        with open("/proc/self/maps") as f:
            return sorted({ln.split()[-1] for ln in f if "libamdhip64" in ln})
    except OSError:
        return []


if len(hip_runtimes()) > 1:
    raise ImportError("two HIP runtimes are loaded in this process (" + ", ".join(hip_runtimes())
                      + "); import torch before anything that loads libamdhip64")


class Options(ctypes.Structure):
    """``lcsm_options``: 0 selects the library default."""
    _fields_ = [("direct_max_u", ctypes.c_int), ("lds_fft_max_n", ctypes.c_int),
                ("scratch_mib", ctypes.c_int), ("half_state", ctypes.c_int),
                ("col_fft_min_n", ctypes.c_int), ("col_tile_form", ctypes.c_int),
                ("reserved", ctypes.c_int * 2)]


_c_int_p = ctypes.POINTER(ctypes.c_int)
_vp = ctypes.c_void_p

_SIGS = {
    "lcsm_workspace_bytes": (ctypes.c_int, [ctypes.c_int] * 4 + [ctypes.POINTER(Options),
                                                                  ctypes.POINTER(ctypes.c_size_t)]),
    "lcsm_init": (ctypes.c_int, [ctypes.POINTER(_vp), _vp] + [ctypes.c_int] * 4
                  + [_vp, _vp, ctypes.c_size_t, ctypes.POINTER(Options)]),
    "lcsm_step": (ctypes.c_int, [_vp, _vp, _vp]),
    "lcsm_step_chain": (ctypes.c_int, [_vp, _vp, _vp]),
    "lcsm_step_layer": (ctypes.c_int, [_vp, ctypes.c_int, _vp, _vp]),
    "lcsm_advance": (ctypes.c_int, [_vp]),
    "lcsm_run": (ctypes.c_int, [_vp, ctypes.c_int, _vp, ctypes.c_size_t, _vp, ctypes.c_size_t]),
    "lcsm_run_noalloc": (ctypes.c_int, [_vp, ctypes.c_int, _vp, ctypes.c_size_t, _vp, ctypes.c_size_t]),
    "lcsm_run_chain": (ctypes.c_int, [_vp, ctypes.c_int, _vp, ctypes.c_size_t, _vp, ctypes.c_size_t]),
    "lcsm_prefill": (ctypes.c_int, [_vp, ctypes.c_int, _vp, ctypes.c_size_t, _vp, ctypes.c_size_t]),
    "lcsm_reset": (ctypes.c_int, [_vp]),
    "lcsm_position": (ctypes.c_int, [_vp, _c_int_p]),
    "lcsm_plan_tile": (ctypes.c_int, [ctypes.c_int] * 4 + [ctypes.POINTER(Options), ctypes.c_int]
                       + [_c_int_p] * 4),
    "lcsm_tile": (ctypes.c_int, [_vp, ctypes.c_int] + [_c_int_p] * 4),
    "lcsm_h0": (ctypes.c_int, [_vp, ctypes.POINTER(_vp), ctypes.POINTER(ctypes.c_size_t)]),
    "lcsm_pending": (ctypes.c_int, [_vp, ctypes.POINTER(_vp), ctypes.POINTER(ctypes.c_size_t)]),
    "lcsm_commit": (ctypes.c_int, [_vp]),
    "lcsm_destroy": (None, [_vp]),
    "lcsm_graph_capture": (ctypes.c_int, [_vp, ctypes.c_int, ctypes.c_int, _vp, ctypes.c_size_t,
                                          ctypes.c_int, _vp, ctypes.c_size_t, ctypes.c_int,
                                          ctypes.c_int, ctypes.POINTER(_vp)]),
    "lcsm_graph_launch": (ctypes.c_int, [_vp]),
    "lcsm_graph_segments": (ctypes.c_int, [_vp, _c_int_p]),
    "lcsm_graph_destroy": (None, [_vp]),
    "lcsm_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "lcsm_last_error": (ctypes.c_char_p, [_vp]),
    # include/lcsm_base.h
    "lcsm_base_workspace_bytes": (ctypes.c_int, [ctypes.c_int] * 5 + [ctypes.POINTER(ctypes.c_size_t)]),
    "lcsm_base_init": (ctypes.c_int, [ctypes.POINTER(_vp), ctypes.c_int, _vp] + [ctypes.c_int] * 4
                       + [_vp, _vp, ctypes.c_size_t]),
    "lcsm_base_step": (ctypes.c_int, [_vp, _vp, _vp]),
    "lcsm_base_reset": (ctypes.c_int, [_vp]),
    "lcsm_base_position": (ctypes.c_int, [_vp, _c_int_p]),
    "lcsm_base_destroy": (None, [_vp]),
    "lcsm_base_last_error": (ctypes.c_char_p, [_vp]),
    # include/lcsm_dd.h
    "lcsm_dd_workspace_bytes": (ctypes.c_int, [ctypes.c_int] * 4
                                + [ctypes.POINTER(Options), ctypes.POINTER(ctypes.c_size_t)]),
    "lcsm_dd_init": (ctypes.c_int, [ctypes.POINTER(_vp)] + [ctypes.c_int] * 4
                     + [_vp, _vp, ctypes.c_size_t, ctypes.POINTER(Options)]),
    "lcsm_dd_step": (ctypes.c_int, [_vp, _vp, _vp, _vp]),
    "lcsm_dd_reset": (ctypes.c_int, [_vp]),
    "lcsm_dd_position": (ctypes.c_int, [_vp, _c_int_p]),
    "lcsm_dd_destroy": (None, [_vp]),
    "lcsm_dd_last_error": (ctypes.c_char_p, [_vp]),
    # include/lcsm_synth.h
    "lcsm_synth_init": (ctypes.c_int, [ctypes.POINTER(_vp)] + [_vp] * 5 + [ctypes.c_int] * 4
                        + [_vp, ctypes.POINTER(Options)]),
    "lcsm_synth_step": (ctypes.c_int, [_vp, _vp, _vp]),
    "lcsm_synth_reset": (ctypes.c_int, [_vp]),
    "lcsm_synth_position": (ctypes.c_int, [_vp, _c_int_p]),
    "lcsm_synth_destroy": (None, [_vp]),
    "lcsm_synth_last_error": (ctypes.c_char_p, [_vp]),
}

for _name, (_res, _args) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args

EXPORTED = tuple(_SIGS)


class LcsmError(RuntimeError):
    def __init__(self, code, where, detail=""):
        self.code = code
        msg = f"{where}: {_lib.lcsm_strerror(code).decode()} ({code})"
        if detail:
            msg += f": {detail}"
        super().__init__(msg)


def _opts(options):
    if options is None:
        return None
    if isinstance(options, Options):
        return ctypes.byref(options)
    o = Options()
    for k, v in dict(options).items():
        setattr(o, k, int(v))
    return ctypes.byref(o)


def strerror(code: int) -> str:
    return _lib.lcsm_strerror(code).decode()


def workspace_bytes(M, B, D, L, options=None) -> int:
    n = ctypes.c_size_t(0)
    r = _lib.lcsm_workspace_bytes(M, B, D, L, _opts(options), ctypes.byref(n))
    if r:
        raise LcsmError(r, "lcsm_workspace_bytes")
    return n.value


def plan_tile(M, B, D, L, t, options=None):
    """(i, U, dst_len, kind) of the gray tile queued after step t."""
    i, U, n, k = (ctypes.c_int() for _ in range(4))
    r = _lib.lcsm_plan_tile(M, B, D, L, _opts(options), t, ctypes.byref(i), ctypes.byref(U),
                            ctypes.byref(n), ctypes.byref(k))
    if r:
        raise LcsmError(r, "lcsm_plan_tile")
    return i.value, U.value, n.value, k.value


def raw():
    """The ctypes library handle (for tests of the raw ABI)."""
    return _lib


def _after_current(stream, device):
    """Order work queued next on ``stream`` after everything already queued on
    torch's current stream (where callers produce filters and inputs), when
    the two differ: the library's calls are asynchronous on their own stream."""
    import torch
    cur = torch.cuda.current_stream(device)
    if cur.cuda_stream != stream.cuda_stream:
        stream.wait_stream(cur)


class Lcsm:
    """One relaxed online convolution context.

    ``filters``: fp32 CUDA tensor [M, D, L] (h[m, d, k]).  ``B``: batch rows.
    The workspace is a torch uint8 tensor owned by this object; work runs on
    ``stream`` (a torch.cuda.Stream, default: the current stream).
    """

    def __init__(self, filters, B: int, options=None, stream=None):
        import torch
        if not (filters.is_cuda and filters.dtype == torch.float32 and filters.dim() == 3):
            raise ValueError("filters must be a CUDA fp32 tensor [M, D, L]")
        filters = filters.contiguous()
        self.M, self.D, self.L = (int(v) for v in filters.shape)
        self.B = int(B)
        self.device = filters.device
        self._opts_obj = None
        if options is not None and not isinstance(options, Options):
            o = Options()
            for k, v in dict(options).items():
                setattr(o, k, int(v))
            options = o
        self._opts_obj = options
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        nbytes = workspace_bytes(self.M, self.B, self.D, self.L, options)
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        self._ctx = _vp()
        _after_current(self.stream, self.device)
        r = _lib.lcsm_init(ctypes.byref(self._ctx), filters.data_ptr(), self.M, self.B, self.D,
                           self.L, self.stream.cuda_stream, self.workspace.data_ptr(), nbytes,
                           _opts(options))
        if r:
            raise LcsmError(r, "lcsm_init")
        self._filters_keepalive = filters
        self._graphs = weakref.WeakSet()  # recorded generations, released before the context

    # -- helpers
    def _check(self, r, where):
        if r:
            detail = _lib.lcsm_last_error(self._ctx).decode() if self._ctx else ""
            raise LcsmError(r, where, detail)

    def _slab(self, tensor, shape, name):
        import torch
        if not (tensor.is_cuda and tensor.dtype == torch.float32 and tensor.is_contiguous()
                and tuple(tensor.shape) == shape and tensor.device == self.device):
            raise ValueError(f"{name} must be a contiguous CUDA fp32 tensor of shape {shape}")
        return tensor.data_ptr()

    # -- ABI calls
    def step(self, y_t, z_t=None):
        """Emit z_t for all layers given y_t [M, B, D]; queues the gray tile."""
        import torch
        shape = (self.M, self.B, self.D)
        if z_t is None:
            z_t = torch.empty(shape, dtype=torch.float32, device=self.device)
        _after_current(self.stream, self.device)
        self._check(_lib.lcsm_step(self._ctx, self._slab(y_t, shape, "y_t"),
                                   self._slab(z_t, shape, "z_t")), "lcsm_step")
        return z_t

    def step_chain(self, x_t, z_t=None):
        """One position with the built-in tanh chain; x_t [M, B, D]."""
        import torch
        shape = (self.M, self.B, self.D)
        if z_t is None:
            z_t = torch.empty(shape, dtype=torch.float32, device=self.device)
        _after_current(self.stream, self.device)
        self._check(_lib.lcsm_step_chain(self._ctx, self._slab(x_t, shape, "x_t"),
                                         self._slab(z_t, shape, "z_t")), "lcsm_step_chain")
        return z_t

    def step_layer(self, layer, y, z=None):
        import torch
        shape = (self.B, self.D)
        if z is None:
            z = torch.empty(shape, dtype=torch.float32, device=self.device)
        _after_current(self.stream, self.device)
        self._check(_lib.lcsm_step_layer(self._ctx, int(layer), self._slab(y, shape, "y"),
                                         self._slab(z, shape, "z")), "lcsm_step_layer")
        return z

    def advance(self):
        self._check(_lib.lcsm_advance(self._ctx), "lcsm_advance")

    def run(self, y, z, n=None, t0=0):
        """Steps t0 .. t0+n-1 reading y[k] and writing z[k] ([n, M, B, D] tensors)."""
        shape = (self.M, self.B, self.D)
        n = y.shape[0] if n is None else n
        if y.shape[1:] != shape or z.shape[1:] != shape or y.shape[0] < n or z.shape[0] < n:
            raise ValueError("y and z must be [n, M, B, D]")
        if not (y.is_contiguous() and z.is_contiguous() and y.is_cuda and z.is_cuda):
            raise ValueError("y and z must be contiguous CUDA tensors")
        slab = self.M * self.B * self.D
        _after_current(self.stream, self.device)
        self._check(_lib.lcsm_run(self._ctx, int(n), y.data_ptr(), slab, z.data_ptr(), slab),
                    "lcsm_run")
        return z

    def run_chain(self, x, z, n=None):
        """n chained steps (lcsm_run_chain) reading x[k] and writing z[k] ([n, M, B, D])."""
        shape = (self.M, self.B, self.D)
        n = x.shape[0] if n is None else n
        if x.shape[1:] != shape or z.shape[1:] != shape or x.shape[0] < n or z.shape[0] < n:
            raise ValueError("x and z must be [n, M, B, D]")
        if not (x.is_contiguous() and z.is_contiguous() and x.is_cuda and z.is_cuda):
            raise ValueError("x and z must be contiguous CUDA tensors")
        slab = self.M * self.B * self.D
        _after_current(self.stream, self.device)
        self._check(_lib.lcsm_run_chain(self._ctx, int(n), x.data_ptr(), slab, z.data_ptr(), slab),
                    "lcsm_run_chain")
        return z

    def prefill(self, y, z, P=None):
        """Prompt prefill at position 0: y, z are [P, M, B, D] tensors (P a power
        of two, 2P <= L); z receives the prompt's outputs and the context moves
        to position P."""
        shape = (self.M, self.B, self.D)
        P = y.shape[0] if P is None else P
        if y.shape[1:] != shape or z.shape[1:] != shape or y.shape[0] < P or z.shape[0] < P:
            raise ValueError("y and z must be [P, M, B, D]")
        if not (y.is_contiguous() and z.is_contiguous() and y.is_cuda and z.is_cuda):
            raise ValueError("y and z must be contiguous CUDA tensors")
        slab = self.M * self.B * self.D
        _after_current(self.stream, self.device)
        self._check(_lib.lcsm_prefill(self._ctx, int(P), y.data_ptr(), slab, z.data_ptr(), slab),
                    "lcsm_prefill")
        return z

    def reset(self):
        self._check(_lib.lcsm_reset(self._ctx), "lcsm_reset")

    def capture(self, x, z, n=None, chain=False, seg=0):
        """Record lcsm_reset + n steps as a chain of HIP graphs (lcsm_graph_capture).
        x, z: [R, M, B, D] tensors used as rings (step k reads x[k % R], writes
        z[k % Rz]); chain: record lcsm_step_chain (x = additive inputs) instead of
        lcsm_step (x = y).  Returns a Graph; nothing runs until Graph.launch()."""
        shape = (self.M, self.B, self.D)
        n = self.L if n is None else int(n)
        if tuple(x.shape[1:]) != shape or tuple(z.shape[1:]) != shape:
            raise ValueError("x and z must be [R, M, B, D]")
        if not (x.is_contiguous() and z.is_contiguous() and x.is_cuda and z.is_cuda):
            raise ValueError("x and z must be contiguous CUDA tensors")
        slab = self.M * self.B * self.D
        g = _vp()
        self._check(_lib.lcsm_graph_capture(self._ctx, GRAPH_CHAIN if chain else 0, n,
                                            x.data_ptr(), slab, int(x.shape[0]), z.data_ptr(),
                                            slab, int(z.shape[0]), int(seg), ctypes.byref(g)),
                    "lcsm_graph_capture")
        graph = Graph(self, g, (x, z))
        self._graphs.add(graph)
        return graph

    @property
    def position(self) -> int:
        t = ctypes.c_int()
        self._check(_lib.lcsm_position(self._ctx, ctypes.byref(t)), "lcsm_position")
        return t.value

    def plan(self, t):
        return plan_tile(self.M, self.B, self.D, self.L, t, self._opts_obj)

    def tile(self, t):
        """(i, U, dst_len, kind) of the gray tile this context queues after step t."""
        i, U, n, k = (ctypes.c_int() for _ in range(4))
        self._check(_lib.lcsm_tile(self._ctx, int(t), ctypes.byref(i), ctypes.byref(U),
                                   ctypes.byref(n), ctypes.byref(k)), "lcsm_tile")
        return i.value, U.value, n.value, k.value

    def _ws_view(self, ptr, stride, rows, rowlen, what):
        """[rows, rowlen] fp32 view of the workspace at device address ptr,
        row k at ptr + k*stride floats (the library's buffers live in the
        workspace tensor this object owns)."""
        import torch
        base = self.workspace.data_ptr()
        off = ptr - base
        end = off + 4 * ((rows - 1) * stride + rowlen)
        if off < 0 or off % 4 or end > self.workspace.numel():
            raise LcsmError(LCSM_EINVAL, what, "view outside the workspace")
        flat = self.workspace.view(torch.float32)
        return flat.as_strided((rows, rowlen), (stride, 1), off // 4)

    def h0(self):
        """Lag-0 taps h[m, d, 0] as a [M, D] view of the library's filter copy."""
        p, st = _vp(), ctypes.c_size_t()
        self._check(_lib.lcsm_h0(self._ctx, ctypes.byref(p), ctypes.byref(st)), "lcsm_h0")
        return self._ws_view(p.value, st.value, self.M, self.D, "lcsm_h0")

    def pending(self):
        """Accumulators of the current position t as a [M, B, D] view of the
        state (valid for this position only); see lcsm_commit."""
        p, st = _vp(), ctypes.c_size_t()
        self._check(_lib.lcsm_pending(self._ctx, ctypes.byref(p), ctypes.byref(st)),
                    "lcsm_pending")
        v = self._ws_view(p.value, st.value, self.M, self.B * self.D, "lcsm_pending")
        return v.view(self.M, self.B, self.D)

    def commit(self):
        """After the caller's own red cells at t (z = fmaf(h0, y, acc), y
        written over the pending row): queue the gray tiles, advance t."""
        self._check(_lib.lcsm_commit(self._ctx), "lcsm_commit")

    def close(self):
        if self._ctx:
            for g in list(getattr(self, "_graphs", ())):
                g.close()
            _lib.lcsm_destroy(self._ctx)
            self._ctx = _vp()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Graph:
    """A recorded generation (``lcsm_graph``): ``launch()`` queues lcsm_reset +
    the recorded steps on the context's stream as a chain of HIP graphs."""

    def __init__(self, ctx, handle, keepalive):
        self._ctx = ctx
        self._g = handle
        self._keepalive = keepalive

    def launch(self):
        _after_current(self._ctx.stream, self._ctx.device)
        self._ctx._check(_lib.lcsm_graph_launch(self._g), "lcsm_graph_launch")

    @property
    def segments(self) -> int:
        n = ctypes.c_int()
        self._ctx._check(_lib.lcsm_graph_segments(self._g, ctypes.byref(n)), "lcsm_graph_segments")
        return n.value

    def close(self):
        if self._g:
            _lib.lcsm_graph_destroy(self._g)
            self._g = _vp()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def base_workspace_bytes(kind, M, B, D, L) -> int:
    n = ctypes.c_size_t(0)
    r = _lib.lcsm_base_workspace_bytes(int(kind), M, B, D, L, ctypes.byref(n))
    if r:
        raise LcsmError(r, "lcsm_base_workspace_bytes")
    return n.value


class Base:
    """A lazy or eager online convolution context (``include/lcsm_base.h``), the
    baselines of Sec. 3.1.1: ``kind`` is one of BASE_KINDS' names or codes.
    ``filters`` [M, D, L] fp32 CUDA tensor; the workspace is a torch uint8
    tensor owned by this object."""

    def __init__(self, kind, filters, B: int, stream=None):
        import torch
        if not (filters.is_cuda and filters.dtype == torch.float32 and filters.dim() == 3):
            raise ValueError("filters must be a CUDA fp32 tensor [M, D, L]")
        self.kind = BASE_KINDS[kind] if isinstance(kind, str) else int(kind)
        filters = filters.contiguous()
        self.M, self.D, self.L = (int(v) for v in filters.shape)
        self.B = int(B)
        self.device = filters.device
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        nbytes = base_workspace_bytes(self.kind, self.M, self.B, self.D, self.L)
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        self._ctx = _vp()
        _after_current(self.stream, self.device)
        r = _lib.lcsm_base_init(ctypes.byref(self._ctx), self.kind, filters.data_ptr(), self.M,
                                self.B, self.D, self.L, self.stream.cuda_stream,
                                self.workspace.data_ptr(), nbytes)
        if r:
            raise LcsmError(r, "lcsm_base_init")
        self._filters_keepalive = filters

    def _check(self, r, where):
        if r:
            detail = _lib.lcsm_base_last_error(self._ctx).decode() if self._ctx else ""
            raise LcsmError(r, where, detail)

    def step(self, y_t, z_t=None):
        import torch
        shape = (self.M, self.B, self.D)
        if z_t is None:
            z_t = torch.empty(shape, dtype=torch.float32, device=self.device)
        for t, name in ((y_t, "y_t"), (z_t, "z_t")):
            if not (t.is_cuda and t.dtype == torch.float32 and t.is_contiguous()
                    and tuple(t.shape) == shape):
                raise ValueError(f"{name} must be a contiguous CUDA fp32 tensor of shape {shape}")
        _after_current(self.stream, self.device)
        self._check(_lib.lcsm_base_step(self._ctx, y_t.data_ptr(), z_t.data_ptr()), "lcsm_base_step")
        return z_t

    def reset(self):
        self._check(_lib.lcsm_base_reset(self._ctx), "lcsm_base_reset")

    @property
    def position(self) -> int:
        t = ctypes.c_int()
        self._check(_lib.lcsm_base_position(self._ctx, ctypes.byref(t)), "lcsm_base_position")
        return t.value

    def close(self):
        if self._ctx:
            _lib.lcsm_base_destroy(self._ctx)
            self._ctx = _vp()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def dd_workspace_bytes(M, B, D, L, options=None) -> int:
    n = ctypes.c_size_t(0)
    r = _lib.lcsm_dd_workspace_bytes(M, B, D, L, _opts(options), ctypes.byref(n))
    if r:
        raise LcsmError(r, "lcsm_dd_workspace_bytes")
    return n.value


class Dd:
    """Relaxed online convolution with data-dependent filters
    (``include/lcsm_dd.h``): at step t both y_t and rho_t [M, B, D] arrive and
    z_t = sum_{j+k=t} y_j rho_k is returned.  The workspace is a torch uint8
    tensor owned by this object."""

    def __init__(self, M, B, D, L, options=None, stream=None, device="cuda:0"):
        import torch
        self.M, self.B, self.D, self.L = int(M), int(B), int(D), int(L)
        self.device = torch.device(device)
        if options is not None and not isinstance(options, Options):
            o = Options()
            for k, v in dict(options).items():
                setattr(o, k, int(v))
            options = o
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        nbytes = dd_workspace_bytes(self.M, self.B, self.D, self.L, options)
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        self._ctx = _vp()
        _after_current(self.stream, self.device)
        r = _lib.lcsm_dd_init(ctypes.byref(self._ctx), self.M, self.B, self.D, self.L,
                              self.stream.cuda_stream, self.workspace.data_ptr(), nbytes,
                              _opts(options))
        if r:
            raise LcsmError(r, "lcsm_dd_init")

    def _check(self, r, where):
        if r:
            detail = _lib.lcsm_dd_last_error(self._ctx).decode() if self._ctx else ""
            raise LcsmError(r, where, detail)

    def step(self, y_t, rho_t, z_t=None):
        import torch
        shape = (self.M, self.B, self.D)
        if z_t is None:
            z_t = torch.empty(shape, dtype=torch.float32, device=self.device)
        for t, name in ((y_t, "y_t"), (rho_t, "rho_t"), (z_t, "z_t")):
            if not (t.is_cuda and t.dtype == torch.float32 and t.is_contiguous()
                    and tuple(t.shape) == shape):
                raise ValueError(f"{name} must be a contiguous CUDA fp32 tensor of shape {shape}")
        _after_current(self.stream, self.device)
        self._check(_lib.lcsm_dd_step(self._ctx, y_t.data_ptr(), rho_t.data_ptr(), z_t.data_ptr()),
                    "lcsm_dd_step")
        return z_t

    def reset(self):
        self._check(_lib.lcsm_dd_reset(self._ctx), "lcsm_dd_reset")

    @property
    def position(self) -> int:
        t = ctypes.c_int()
        self._check(_lib.lcsm_dd_position(self._ctx, ctypes.byref(t)), "lcsm_dd_position")
        return t.value

    def close(self):
        if self._ctx:
            _lib.lcsm_dd_destroy(self._ctx)
            self._ctx = _vp()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Synth:
    """The synthetic end-to-end model (``include/lcsm_synth.h``): per layer the
    long-convolution mixer and an MLP block (hidden 2D, GELU); the next
    token's input is the last layer's output plus the noise handed to step.

    ``filters`` [M, D, L]; ``w_up`` [M, 2D, D], ``b_up`` [M, 2D], ``w_down``
    [M, D, 2D], ``b_down`` [M, D] (fp32 CUDA tensors, copied at init).
    """

    def __init__(self, filters, w_up, b_up, w_down, b_down, B: int, options=None, stream=None):
        import torch
        ts = (filters, w_up, b_up, w_down, b_down)
        if not all(t.is_cuda and t.dtype == torch.float32 for t in ts):
            raise ValueError("filters and weights must be CUDA fp32 tensors")
        filters, w_up, b_up, w_down, b_down = (t.contiguous() for t in ts)
        self.M, self.D, self.L = (int(v) for v in filters.shape)
        self.B = int(B)
        M, D = self.M, self.D
        shapes = {"w_up": (M, 2 * D, D), "b_up": (M, 2 * D), "w_down": (M, D, 2 * D),
                  "b_down": (M, D)}
        for name, t in zip(shapes, (w_up, b_up, w_down, b_down)):
            if tuple(t.shape) != shapes[name]:
                raise ValueError(f"{name} must have shape {shapes[name]}")
        self.device = filters.device
        if options is not None and not isinstance(options, Options):
            o = Options()
            for k, v in dict(options).items():
                setattr(o, k, int(v))
            options = o
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        self._ctx = _vp()
        _after_current(self.stream, self.device)
        r = _lib.lcsm_synth_init(ctypes.byref(self._ctx), filters.data_ptr(), w_up.data_ptr(),
                                 b_up.data_ptr(), w_down.data_ptr(), b_down.data_ptr(), M, self.B,
                                 D, self.L, self.stream.cuda_stream, _opts(options))
        if r:
            raise LcsmError(r, "lcsm_synth_init")
        # the copies are queued on the stream: keep the sources until it passes them
        self._keepalive = (filters, w_up, b_up, w_down, b_down)

    def _check(self, r, where):
        if r:
            detail = _lib.lcsm_synth_last_error(self._ctx).decode() if self._ctx else ""
            raise LcsmError(r, where, detail)

    def step(self, eps_t, act_t=None):
        """Position t: noise eps_t [B, D] in, block outputs of every layer
        act_t [M, B, D] out (act_t[M-1] is the model's output)."""
        import torch
        if act_t is None:
            act_t = torch.empty((self.M, self.B, self.D), dtype=torch.float32, device=self.device)
        for t, shape, name in ((eps_t, (self.B, self.D), "eps_t"),
                               (act_t, (self.M, self.B, self.D), "act_t")):
            if not (t.is_cuda and t.dtype == torch.float32 and t.is_contiguous()
                    and tuple(t.shape) == shape):
                raise ValueError(f"{name} must be a contiguous CUDA fp32 tensor of shape {shape}")
        _after_current(self.stream, self.device)
        self._check(_lib.lcsm_synth_step(self._ctx, eps_t.data_ptr(), act_t.data_ptr()),
                    "lcsm_synth_step")
        return act_t

    def reset(self):
        self._check(_lib.lcsm_synth_reset(self._ctx), "lcsm_synth_reset")

    @property
    def position(self) -> int:
        t = ctypes.c_int()
        self._check(_lib.lcsm_synth_position(self._ctx, ctypes.byref(t)), "lcsm_synth_position")
        return t.value

    def close(self):
        if self._ctx:
            _lib.lcsm_synth_destroy(self._ctx)
            self._ctx = _vp()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
