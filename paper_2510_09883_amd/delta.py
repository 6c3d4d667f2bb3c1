"""Python binding of libdelta_attn.so (ctypes; argument marshalling only).

Every function has the name and argument order of the C entry point declared in
include/delta_attn.h.  Tensors are passed by device pointer; the stream is torch's current
stream.  A non-zero status raises DeltaError.  Importing this module raises ImportError if
the library has not been built: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

import torch

# DELTA_ATTN_LIB selects another build of the same library (the debug or host-ASan build)
LIB_PATH = os.environ.get("DELTA_ATTN_LIB") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), "libdelta_attn.so")
if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                      "(python -m paper_2510_09883_amd.build)")
_lib = ctypes.CDLL(LIB_PATH)

DELTA_OK, DELTA_ERR_INVALID_ARG, DELTA_ERR_UNSUPPORTED, DELTA_ERR_WORKSPACE, DELTA_ERR_HIP = 0, -1, -2, -3, -4
DELTA_ERR_HOOK = -5
DELTA_ROLE_FULL, DELTA_ROLE_DELTA, DELTA_ROLE_SPARSE = 0, 1, 2
DELTA_AGG_MAX, DELTA_AGG_SUM = 0, 1
DELTA_PATH_AUTO, DELTA_PATH_SPLIT, DELTA_PATH_FUSED = 0, 1, 2

EXPORTED = ["delta_workspace_bytes", "delta_workspace_init", "delta_full_attn",
            "delta_delta_attn_select", "delta_sparse_attn", "delta_decode_step",
            "delta_kv_append", "delta_decode_step_hooked", "delta_delta_path",
            "delta_decode_step_noalloc", "delta_build_flags", "delta_status_string"]
DELTA_BUILD_DEBUG = 1
DELTA_DEBUG_PAGE, DELTA_DEBUG_SEQ_LEN, DELTA_DEBUG_SELECTION = 1, 2, 4
DELTA_NOALLOC_SCRATCH_BYTES = 160 << 20


class delta_shape_t(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("max_pages_per_seq", ctypes.c_int32),
                ("max_seq_len", ctypes.c_int32), ("sm_scale", ctypes.c_float)]


class delta_kv_t(ctypes.Structure):
    _fields_ = [("k_cache", ctypes.c_void_p), ("v_cache", ctypes.c_void_p),
                ("page_table", ctypes.c_void_p), ("seq_lens", ctypes.c_void_p),
                ("n_pages", ctypes.c_int64)]


class delta_select_t(ctypes.Structure):
    _fields_ = [("budget_tokens", ctypes.c_int32), ("recent_tokens", ctypes.c_int32),
                ("unit_tokens", ctypes.c_int32), ("agg", ctypes.c_int32),
                ("delta_path", ctypes.c_int32)]


_P = ctypes.POINTER
_vp = ctypes.c_void_p

# int (*)(int32_t layer, void* user, void* stream)
delta_layer_hook_t = ctypes.CFUNCTYPE(ctypes.c_int, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p)


class delta_hooks_t(ctypes.Structure):
    _fields_ = [("before_attn", delta_layer_hook_t), ("after_attn", delta_layer_hook_t),
                ("user", ctypes.c_void_p)]


def _bind(lib):
    """Declare the C signatures of include/delta_attn.h on a loaded library handle."""
    lib.delta_workspace_bytes.argtypes = [_P(delta_shape_t), _P(delta_select_t), _P(ctypes.c_size_t)]
    lib.delta_workspace_init.argtypes = [_vp, ctypes.c_size_t, _vp]
    lib.delta_full_attn.argtypes = [_P(delta_shape_t), _P(delta_kv_t), _vp, _vp, _vp, ctypes.c_size_t, _vp]
    lib.delta_delta_attn_select.argtypes = [_P(delta_shape_t), _P(delta_kv_t), _vp, _vp,
                                            _P(delta_select_t), _vp, _vp, _vp, _vp, _vp,
                                            ctypes.c_size_t, _vp]
    lib.delta_sparse_attn.argtypes = [_P(delta_shape_t), _P(delta_kv_t), _vp, _vp, _P(delta_select_t),
                                      _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]
    lib.delta_decode_step.argtypes = [_P(delta_shape_t), ctypes.c_int32, _P(ctypes.c_int32),
                                      _P(delta_kv_t), _P(_vp), _P(_vp), _P(delta_select_t),
                                      _vp, _vp, _vp, ctypes.c_size_t, _vp]
    lib.delta_kv_append.argtypes = [_P(delta_shape_t), _vp, _vp, _vp, _vp, _vp, _vp, _vp]
    lib.delta_decode_step_hooked.argtypes = [_P(delta_shape_t), ctypes.c_int32, _P(ctypes.c_int32),
                                             _P(delta_kv_t), _P(_vp), _P(_vp), _P(delta_select_t),
                                             _vp, _vp, _vp, ctypes.c_size_t, _vp, _P(delta_hooks_t)]
    lib.delta_decode_step_noalloc.argtypes = [_P(delta_shape_t), ctypes.c_int32, _P(ctypes.c_int32),
                                              _P(delta_kv_t), _P(_vp), _P(_vp), _P(delta_select_t),
                                              _vp, _vp, _vp]
    lib.delta_build_flags.argtypes = []
    lib.delta_hbm_read_probe.argtypes = [_vp, ctypes.c_size_t, _vp, ctypes.c_int32, ctypes.c_int32, _vp]
    lib.delta_hbm_read_probe.restype = ctypes.c_int
    lib.delta_hbm_gather_probe.argtypes = [_vp, ctypes.c_size_t, _vp, ctypes.c_int32, _vp,
                                           ctypes.c_int32, _vp]
    lib.delta_hbm_gather_probe.restype = ctypes.c_int
    lib.delta_status_string.argtypes = [ctypes.c_int]
    lib.delta_status_string.restype = ctypes.c_char_p
    for n in EXPORTED[:-1]:
        getattr(lib, n).restype = ctypes.c_int
    return lib


_lib = _bind(_lib)


class DeltaError(RuntimeError):
    def __init__(self, fn, status):
        super().__init__(f"{fn}: {delta_status_string(status)} ({status})")
        self.status = status


def delta_status_string(status: int) -> str:
    return _lib.delta_status_string(status).decode()


def _check(fn, status):
    if status != DELTA_OK:
        raise DeltaError(fn, status)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dev(name, t, dtype=None, shape=None, at_least=None):
    """The library reads and writes these buffers on the GPU: refuse, before any launch, a
    host tensor, a wrong element type, a non-contiguous view or a wrong shape (None entries of
    `shape` are free; `at_least` bounds the element count instead)."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch.Tensor, got {type(t).__name__}")
    if not t.is_cuda:
        raise ValueError(f"{name}: must be a GPU tensor (got device {t.device})")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name}: expected {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if shape is not None and (t.dim() != len(shape) or
                              any(w is not None and w != d for w, d in zip(shape, t.shape))):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")
    if at_least is not None and t.numel() < at_least:
        raise ValueError(f"{name}: needs at least {at_least} elements, has {t.numel()}")
    return t


def _check_kv(kv, shape):
    t = getattr(kv, "_tensors", None)
    if t is None:   # built by hand from raw pointers: nothing to check
        return
    k, v, pt, sl = t
    cache = (None, shape.n_kv_heads, shape.page_size, shape.head_dim)
    _dev("k_cache", k, torch.bfloat16, cache)
    _dev("v_cache", v, torch.bfloat16, cache)
    _dev("page_table", pt, torch.int32, (shape.batch, shape.max_pages_per_seq))
    _dev("seq_lens", sl, torch.int32, (shape.batch,))


def _check_qo(shape, q, out):
    qo = (shape.batch, shape.n_q_heads, shape.head_dim)
    _dev("q", q, torch.bfloat16, qo)
    _dev("out", out, torch.bfloat16, qo)


def _check_sel(shape, sel, sel_idx, sel_cnt, sel_phys=None):
    K = sel.budget_tokens // max(sel.unit_tokens, 1)
    _dev("sel_idx", sel_idx, torch.int32, (shape.batch, K))
    _dev("sel_cnt", sel_cnt, torch.int32, (shape.batch,))
    if sel_phys is not None:
        _dev("sel_phys", sel_phys, torch.int32, (shape.batch, K))


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def make_shape(batch, n_q_heads, n_kv_heads, head_dim, max_pages_per_seq, max_seq_len,
               sm_scale=0.0, page_size=16) -> delta_shape_t:
    return delta_shape_t(batch, n_q_heads, n_kv_heads, head_dim, page_size, max_pages_per_seq,
                         max_seq_len, sm_scale)


def make_select(budget_tokens, recent_tokens, unit_tokens=16, agg=DELTA_AGG_MAX,
                delta_path=DELTA_PATH_AUTO) -> delta_select_t:
    return delta_select_t(budget_tokens, recent_tokens, unit_tokens, agg, delta_path)


def make_kv(k_cache, v_cache, page_table, seq_lens) -> delta_kv_t:
    for name, t in (("k_cache", k_cache), ("v_cache", v_cache), ("page_table", page_table),
                    ("seq_lens", seq_lens)):
        _dev(name, t)
    if k_cache.dim() < 1 or v_cache.dim() < 1 or k_cache.shape[0] != v_cache.shape[0]:
        raise ValueError(f"k_cache and v_cache must hold the same number of pages "
                         f"(got {tuple(k_cache.shape)}, {tuple(v_cache.shape)})")
    kv = delta_kv_t(k_cache.data_ptr(), v_cache.data_ptr(), page_table.data_ptr(), seq_lens.data_ptr(),
                    k_cache.shape[0])
    kv._tensors = (k_cache, v_cache, page_table, seq_lens)   # checked against the shape per call
    return kv


def delta_build_flags() -> int:
    """DELTA_BUILD_DEBUG if the loaded library is the debug build."""
    return int(_lib.delta_build_flags())


def delta_delta_path(shape: delta_shape_t, sel: delta_select_t) -> bool:
    """Whether delta_delta_attn_select runs the fused kernel for this shape and selection
    (sel.delta_path) on the current device."""
    f = ctypes.c_int(0)
    _check("delta_delta_path", _lib.delta_delta_path(ctypes.byref(shape), ctypes.byref(sel),
                                                     ctypes.byref(f)))
    return bool(f.value)


def delta_workspace_bytes(shape: delta_shape_t, sel: delta_select_t | None = None) -> int:
    n = ctypes.c_size_t(0)
    _check("delta_workspace_bytes",
           _lib.delta_workspace_bytes(ctypes.byref(shape), ctypes.byref(sel) if sel else None,
                                      ctypes.byref(n)))
    return n.value


def delta_workspace_init(ws: torch.Tensor):
    _dev("ws", ws)
    _check("delta_workspace_init", _lib.delta_workspace_init(_ptr(ws), ws.numel() * ws.element_size(), _stream()))


def alloc_workspace(shape, sel=None, device="cuda") -> torch.Tensor:
    """A zero-filled workspace (uint8) large enough for every call with this shape/selection."""
    return torch.zeros(delta_workspace_bytes(shape, sel), dtype=torch.uint8, device=device)


def _nbytes(t):
    return t.numel() * t.element_size()


def delta_full_attn(shape, kv: delta_kv_t, q, out, ws):
    _check_kv(kv, shape)
    _check_qo(shape, q, out)
    _dev("ws", ws)
    _check("delta_full_attn", _lib.delta_full_attn(ctypes.byref(shape), ctypes.byref(kv), _ptr(q),
                                                   _ptr(out), _ptr(ws), _nbytes(ws), _stream()))


def delta_delta_attn_select(shape, kv: delta_kv_t, q, out, sel, sel_idx, sel_cnt, unit_scores, ws,
                            sel_phys=None):
    _check_kv(kv, shape)
    _check_qo(shape, q, out)
    _check_sel(shape, sel, sel_idx, sel_cnt, sel_phys)
    if unit_scores is not None:
        n_u = -(-shape.max_seq_len // max(sel.unit_tokens, 1))
        _dev("unit_scores", unit_scores, torch.float32, at_least=shape.batch * n_u)
    _dev("ws", ws)
    _check("delta_delta_attn_select",
           _lib.delta_delta_attn_select(ctypes.byref(shape), ctypes.byref(kv), _ptr(q), _ptr(out),
                                        ctypes.byref(sel), _ptr(sel_idx), _ptr(sel_cnt),
                                        _ptr(sel_phys), _ptr(unit_scores), _ptr(ws), _nbytes(ws),
                                        _stream()))


def delta_sparse_attn(shape, kv: delta_kv_t, q, out, sel, sel_idx, sel_cnt, ws, sel_phys=None):
    _check_kv(kv, shape)
    _check_qo(shape, q, out)
    _check_sel(shape, sel, sel_idx, sel_cnt, sel_phys)
    _dev("ws", ws)
    _check("delta_sparse_attn",
           _lib.delta_sparse_attn(ctypes.byref(shape), ctypes.byref(kv), _ptr(q), _ptr(out),
                                  ctypes.byref(sel), _ptr(sel_idx), _ptr(sel_cnt), _ptr(sel_phys),
                                  _ptr(ws), _nbytes(ws), _stream()))


class StepArgs:
    """Host-side argument arrays of delta_decode_step, built once and reused every step."""

    def __init__(self, shape, roles, kvs, qs, outs, sel, sel_idx, sel_cnt, ws):
        n = len(roles)
        if not (len(kvs) == len(qs) == len(outs) == n):
            raise ValueError(f"{n} roles need {n} kv, q and out entries "
                             f"(got {len(kvs)}, {len(qs)}, {len(outs)})")
        for kv, q, o in zip(kvs, qs, outs):
            _check_kv(kv, shape)
            _check_qo(shape, q, o)
        n_delta = sum(1 for r in roles if r == DELTA_ROLE_DELTA)
        if n_delta:
            K = sel.budget_tokens // max(sel.unit_tokens, 1)
            _dev("sel_idx", sel_idx, torch.int32, (None, shape.batch, K))
            _dev("sel_cnt", sel_cnt, torch.int32, (None, shape.batch))
            if sel_idx.shape[0] < n_delta or sel_cnt.shape[0] < n_delta:
                raise ValueError(f"sel_idx / sel_cnt need a slot for each of the {n_delta} Delta layers")
        if ws is not None:   # None: only for delta_decode_step_noalloc
            _dev("ws", ws)
        self.shape = shape
        self.n = n
        self.roles = (ctypes.c_int32 * n)(*roles)
        self.kvs = (delta_kv_t * n)(*kvs)
        self.qs = (_vp * n)(*[q.data_ptr() for q in qs])
        self.outs = (_vp * n)(*[o.data_ptr() for o in outs])
        self.sel = sel
        self.sel_idx, self.sel_cnt, self.ws = sel_idx, sel_cnt, ws
        self._keep = (qs, outs)


def delta_decode_step(args: StepArgs):
    a = args
    _check("delta_decode_step",
           _lib.delta_decode_step(ctypes.byref(a.shape), a.n, a.roles, a.kvs, a.qs, a.outs,
                                  ctypes.byref(a.sel) if a.sel is not None else None,
                                  _ptr(a.sel_idx), _ptr(a.sel_cnt), _ptr(a.ws), _nbytes(a.ws),
                                  _stream()))


def delta_decode_step_noalloc(args: StepArgs):
    """delta_decode_step on the library's own scratch memory (args.ws is not used)."""
    a = args
    _check("delta_decode_step_noalloc",
           _lib.delta_decode_step_noalloc(ctypes.byref(a.shape), a.n, a.roles, a.kvs, a.qs, a.outs,
                                          ctypes.byref(a.sel) if a.sel is not None else None,
                                          _ptr(a.sel_idx), _ptr(a.sel_cnt), _stream()))


def delta_kv_append(shape, k_cache, v_cache, page_table, seq_lens, k_new, v_new):
    _check_kv(make_kv(k_cache, v_cache, page_table, seq_lens), shape)
    row = (shape.batch, shape.n_kv_heads, shape.head_dim)
    _dev("k_new", k_new, torch.bfloat16, row)
    _dev("v_new", v_new, torch.bfloat16, row)
    _check("delta_kv_append",
           _lib.delta_kv_append(ctypes.byref(shape), _ptr(k_cache), _ptr(v_cache), _ptr(page_table),
                                _ptr(seq_lens), _ptr(k_new), _ptr(v_new), _stream()))


class LayerHooks:
    """Python callables before(layer) / after(layer), run around each layer's attention by
    delta_decode_step_hooked on the calling thread; they enqueue work on torch's current stream
    (the step's stream).  An exception in a hook stops the step and is re-raised."""

    def __init__(self, before=None, after=None):
        self.error = None

        def wrap(fn):
            if fn is None:
                return delta_layer_hook_t()

            def cb(layer, user, stream):
                try:
                    fn(int(layer))
                    return 0
                except BaseException as e:   # noqa: BLE001 - handed back to the caller
                    self.error = e
                    return 1
            return delta_layer_hook_t(cb)

        self._cbs = (wrap(before), wrap(after))
        self.c = delta_hooks_t(self._cbs[0], self._cbs[1], None)


def delta_decode_step_hooked(args: StepArgs, hooks: LayerHooks):
    a = args
    hooks.error = None
    status = _lib.delta_decode_step_hooked(ctypes.byref(a.shape), a.n, a.roles, a.kvs, a.qs, a.outs,
                                           ctypes.byref(a.sel) if a.sel is not None else None,
                                           _ptr(a.sel_idx), _ptr(a.sel_cnt), _ptr(a.ws), _nbytes(a.ws),
                                           _stream(), ctypes.byref(hooks.c))
    if hooks.error is not None:
        raise hooks.error
    _check("delta_decode_step_hooked", status)


def delta_hbm_read_probe(buf, sink, n_workgroups=2048, unroll=4):
    """Streaming read of `buf` (include/delta_probe.h); sink: int32/uint32 [n_workgroups]."""
    rc = _lib.delta_hbm_read_probe(_ptr(buf), _nbytes(buf), _ptr(sink), n_workgroups, unroll, _stream())
    if rc != 0:
        raise DeltaError("delta_hbm_read_probe", rc)


def delta_hbm_gather_probe(buf, chunks, sink, n_workgroups=256):
    """Gather of the 4 KB chunks `chunks` (int64, device) of `buf` (include/delta_probe.h);
    sink: int32/uint32 [n_workgroups * 256].  Every chunk index must lie inside `buf`: checked
    here (a device-to-host read) except while the stream is being captured into a graph, where
    the caller must have made the same call eagerly first."""
    n = _nbytes(buf) // 4096
    if not torch.cuda.is_current_stream_capturing() and chunks.numel() and \
            (int(chunks.min()) < 0 or int(chunks.max()) >= n):
        raise ValueError("gather probe: chunk index outside the buffer")
    rc = _lib.delta_hbm_gather_probe(_ptr(buf), _nbytes(buf), _ptr(chunks), chunks.numel(), _ptr(sink),
                                     n_workgroups, _stream())
    if rc != 0:
        raise DeltaError("delta_hbm_gather_probe", rc)
