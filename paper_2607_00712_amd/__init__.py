"""ISPA hot path on MI355X: thin ctypes binding over libispa.so.

Every computation runs in the HIP kernels of libispa; this module only checks
tensor dtypes/devices/layouts, allocates outputs with torch and passes raw
pointers plus the current HIP stream. There is no CPU fallback: importing
works without the library, but every call raises if it is not built.

    attn_chunk(q, k_cache, v_cache, cache_len, window, n_heads, sink_len=0,
               dual=False, segments=0) -> (out, lse) or (out, lse, out_local, lse_local)
    attn_ranges(q, k_cache, v_cache, ranges, n_heads) -> (out, lse)
    attn_merge(out_a, lse_a, out_b, lse_b) -> (out, lse)
    select_layers(eps, k) -> indices;  inject_modulation(weight, delta_w, transposed)
    LocalKV(k_cache, v_cache, cache_len, window, sink_len): evict, append, attend
    project(a, weight, out_dtype) -> a @ weight^T  (the L-Layer's output projection)
    Stats(d_in, d_out, max_rows).accum(x, y_full, y_local)
    Stats.solve(lam) -> (delta_w, eps)
"""

import ctypes
import os

import torch

__all__ = ["IspaError", "NotSPDError", "lib", "attn_chunk", "attn_chunk_noalloc", "attn_ranges", "attn_merge", "Stats", "StatsBatch",
           "status_string",
           "select_layers", "inject_modulation", "LocalKV", "project", "quantize_rows", "project_w8a8",
           "LIB_PATH", "ISPA_OK", "ISPA_ERR_INVALID_ARG", "ISPA_ERR_UNSUPPORTED",
           "ISPA_ERR_NOT_SPD", "ISPA_ERR_HIP", "ISPA_ERR_STATE", "ISPA_ERR_SCRATCH",
           "ISPA_STATIC_SCRATCH_BYTES"]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libispa.so")

ISPA_OK = 0
ISPA_ERR_INVALID_ARG = -1
ISPA_ERR_UNSUPPORTED = -2
ISPA_ERR_NOT_SPD = -3
ISPA_ERR_HIP = -4
ISPA_ERR_STATE = -5
ISPA_ERR_SCRATCH = -6
ISPA_STATIC_SCRATCH_BYTES = 160 << 20

DTYPE_BF16 = 0
DTYPE_F32 = 1

_c_i32, _c_i64, _c_f32, _c_p, _c_sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t

_SIGNATURES = {
    "ispa_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "ispa_abi_version": (ctypes.c_int, []),
    "ispa_solve_lookahead_check": (ctypes.c_int, [_c_i32, _c_i32]),
    "ispa_attn_chunk": (ctypes.c_int, [_c_p, _c_p, _c_p, _c_i64, _c_i64, _c_i64, _c_i32, _c_i32, _c_i32,
                                       _c_f32, _c_p, _c_p, _c_p, _c_p, _c_p]),
    "ispa_attn_chunk_ws": (ctypes.c_int, [_c_p, _c_p, _c_p, _c_i64, _c_i64, _c_i64, _c_i32, _c_i32, _c_i32,
                                          _c_f32, _c_p, _c_p, _c_p, _c_p, _c_i32, _c_p, _c_sz, _c_p]),
    "ispa_attn_workspace_bytes": (_c_sz, [_c_i64, _c_i64, _c_i64, _c_i32, _c_i32, _c_i32, _c_i32, _c_i32]),
    "ispa_attn_chunk_noalloc": (ctypes.c_int, [_c_p, _c_p, _c_p, _c_i64, _c_i64, _c_i64, _c_i32, _c_i32, _c_i32,
                                               _c_f32, _c_p, _c_p, _c_p, _c_p, _c_p]),
    "ispa_attn_ranges": (ctypes.c_int, [_c_p, _c_p, _c_p, ctypes.POINTER(_c_i64), _c_i32, _c_i32, _c_i32, _c_i32,
                                        _c_f32, _c_p, _c_p, _c_p]),
    "ispa_attn_merge": (ctypes.c_int, [_c_p, _c_p, _c_p, _c_p, _c_i32, _c_i32, _c_i32, _c_p, _c_p, _c_p]),
    "ispa_select_layers": (ctypes.c_int, [ctypes.POINTER(ctypes.c_double), _c_i32, _c_i32, ctypes.POINTER(_c_i32)]),
    "ispa_inject_modulation": (ctypes.c_int, [_c_p, _c_i32, _c_i32, _c_p, _c_i32, _c_i32, _c_p]),
    "ispa_kv_evict": (ctypes.c_int, [_c_p, _c_p, _c_i64, _c_i64, _c_i64, _c_i32, _c_p, _c_p, ctypes.POINTER(_c_i64),
                                     _c_p]),
    "ispa_kv_ring_append": (ctypes.c_int, [_c_p, _c_p, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_i64, _c_i32, _c_p]),
    "ispa_project": (ctypes.c_int, [_c_p, _c_p, _c_i64, _c_i32, _c_i32, _c_p, _c_i32, _c_p]),
    "ispa_quantize_rows": (ctypes.c_int, [_c_p, _c_i32, _c_i64, _c_i32, _c_p, _c_p, _c_p]),
    "ispa_project_w8a8": (ctypes.c_int, [_c_p, _c_p, _c_p, _c_p, _c_i64, _c_i32, _c_i32, _c_p, _c_i32, _c_p]),
    "ispa_stats_workspace_bytes": (_c_sz, [_c_i32, _c_i32, _c_i64]),
    "ispa_stats_create": (ctypes.c_int, [ctypes.POINTER(_c_p), _c_p, _c_sz, _c_i32, _c_i32, _c_i64, _c_p]),
    "ispa_stats_reset": (ctypes.c_int, [_c_p]),
    "ispa_stats_destroy": (ctypes.c_int, [_c_p]),
    "ispa_stats_views": (ctypes.c_int, [_c_p, ctypes.POINTER(_c_p), ctypes.POINTER(_c_p),
                                        ctypes.POINTER(_c_p), ctypes.POINTER(_c_i64)]),
    "ispa_accum_stats": (ctypes.c_int, [_c_p, _c_p, _c_i32, _c_p, _c_p, _c_i32, _c_i64]),
    "ispa_solve_modulation": (ctypes.c_int, [_c_p, _c_f32, _c_p, ctypes.POINTER(ctypes.c_double)]),
    "ispa_solve_modulation_async": (ctypes.c_int, [_c_p, _c_f32, _c_p, _c_p, _c_p]),
    "ispa_solve_modulation_batch": (ctypes.c_int, [ctypes.POINTER(_c_p), _c_i32, _c_f32, _c_p, _c_p, _c_p]),
}

_lib = None


class IspaError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} ({status})")


class NotSPDError(IspaError):
    pass


def lib():
    """The loaded libispa.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"libispa.so is not built ({LIB_PATH}); build it with python -m paper_2607_00712_amd.build")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def status_string(status):
    return lib().ispa_status_string(int(status)).decode()


def _check(status, where):
    if status != ISPA_OK:
        if status == ISPA_ERR_NOT_SPD:
            raise NotSPDError(status, where)
        raise IspaError(status, where)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _require(t, name, dtype, device=None, ndim=2):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on a HIP device")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if t.dim() != ndim or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous {ndim}-d tensor")


_workspaces = {}


def _workspace(device, nbytes):
    """A cached device workspace of at least nbytes (grown on demand)."""
    ws = _workspaces.get(device)
    if ws is None or ws.numel() < nbytes:
        ws = torch.empty(((nbytes + 255) // 256) * 256, dtype=torch.uint8, device=device)
        _workspaces[device] = ws
    return ws


def _qkv(q, k_cache, v_cache, n_heads):
    _require(q, "q", torch.bfloat16)
    dev = q.device
    _require(k_cache, "k_cache", torch.bfloat16, dev)
    _require(v_cache, "v_cache", torch.bfloat16, dev)
    n_q, hidden = q.shape
    if hidden % n_heads:
        raise ValueError("hidden size is not a multiple of n_heads")
    if k_cache.shape[1] != hidden or v_cache.shape[1] != hidden:
        raise ValueError("k/v hidden size differs from q")
    return dev, n_q, hidden, hidden // n_heads


def _outputs(dev, n_q, hidden, n_heads, pairs):
    for name, t, shape in pairs:
        if t is not None:
            _require(t, name, torch.float32, dev)
            if tuple(t.shape) != shape:
                raise ValueError(f"{name} must have shape {shape}")


def _chunk_outputs(q, k_cache, v_cache, cache_len, n_heads, dual, out, lse, out_local, lse_local, need_lse):
    dev, n_q, hidden, head_dim = _qkv(q, k_cache, v_cache, n_heads)
    if k_cache.shape[0] < cache_len or v_cache.shape[0] < cache_len:
        raise ValueError("cache tensors hold fewer than cache_len rows")
    if out is None:
        out = torch.empty((n_q, hidden), dtype=torch.float32, device=dev)
    if lse is None and need_lse:
        lse = torch.empty((n_heads, n_q), dtype=torch.float32, device=dev)
    if dual:
        if out_local is None:
            out_local = torch.empty((n_q, hidden), dtype=torch.float32, device=dev)
        if lse_local is None and need_lse:
            lse_local = torch.empty((n_heads, n_q), dtype=torch.float32, device=dev)
    _outputs(dev, n_q, hidden, n_heads,
             (("out", out, (n_q, hidden)), ("out_local", out_local, (n_q, hidden)),
              ("lse", lse, (n_heads, n_q)), ("lse_local", lse_local, (n_heads, n_q))))
    return dev, n_q, hidden, head_dim, out, lse, out_local, lse_local


def attn_chunk(q, k_cache, v_cache, cache_len, window, n_heads, sink_len=0, scale=0.0,
               dual=False, out=None, lse=None, out_local=None, lse_local=None, need_lse=True, segments=0):
    """Chunk attention (see ispa_attn_chunk / ispa_attn_chunk_ws in include/ispa.h).

    q [n_q, H*d] bf16; k_cache, v_cache [>= cache_len, H*d] bf16 on one device.
    Returns (out, lse), or (out, lse, out_local, lse_local) when dual: out is then
    the full-cache result and out_local the sink + window result. ``segments``:
    0 splits the work over the chip when whole work items fill it poorly, < 0
    never splits, > 0 forces that many runs (the workspace is cached per device).
    """
    L = lib()
    dev, n_q, hidden, head_dim, out, lse, out_local, lse_local = _chunk_outputs(
        q, k_cache, v_cache, cache_len, n_heads, dual, out, lse, out_local, lse_local, need_lse)
    with torch.cuda.device(dev):
        nbytes = L.ispa_attn_workspace_bytes(int(cache_len), int(window), int(sink_len), int(n_q), int(n_heads),
                                             int(head_dim), int(bool(dual)), int(segments))
    ws = _workspace(dev, nbytes) if nbytes > 0 else None
    st = L.ispa_attn_chunk_ws(_ptr(q), _ptr(k_cache), _ptr(v_cache), int(cache_len), int(window), int(sink_len),
                              int(n_q), int(n_heads), int(head_dim), float(scale), _ptr(out), _ptr(lse),
                              _ptr(out_local if dual else None), _ptr(lse_local if dual else None),
                              int(segments), _ptr(ws), int(ws.numel() if ws is not None else 0), _stream(dev))
    _check(st, "ispa_attn_chunk_ws")
    return (out, lse, out_local, lse_local) if dual else (out, lse)


def attn_chunk_noalloc(q, k_cache, v_cache, cache_len, window, n_heads, out, lse, out_local=None, lse_local=None,
                       sink_len=0, scale=0.0):
    """ispa_attn_chunk_noalloc: attn_chunk with the automatic split, its partial
    results in the library's fixed per-GPU device scratch. The caller passes the
    outputs (out_local given: the dual-stream form); nothing is allocated.
    Returns (out, lse[, out_local, lse_local])."""
    L = lib()
    dual = out_local is not None
    dev, n_q, hidden, head_dim, out, lse, out_local, lse_local = _chunk_outputs(
        q, k_cache, v_cache, cache_len, n_heads, dual, out, lse, out_local, lse_local, False)
    st = L.ispa_attn_chunk_noalloc(_ptr(q), _ptr(k_cache), _ptr(v_cache), int(cache_len), int(window),
                                   int(sink_len), int(n_q), int(n_heads), int(head_dim), float(scale), _ptr(out),
                                   _ptr(lse), _ptr(out_local), _ptr(lse_local), _stream(dev))
    _check(st, "ispa_attn_chunk_noalloc")
    return (out, lse, out_local, lse_local) if dual else (out, lse)


def attn_ranges(q, k_cache, v_cache, ranges, n_heads, scale=0.0, out=None, lse=None):
    """Attention over the union of key ranges [(begin, end), ...] (ispa_attn_ranges):
    one branch of the decomposable form (an empty list gives out = 0, lse = -inf)."""
    L = lib()
    dev, n_q, hidden, head_dim = _qkv(q, k_cache, v_cache, n_heads)
    ranges = [(int(b), int(e)) for b, e in ranges]
    if len(ranges) > 3:
        raise ValueError("at most 3 key ranges")
    for b, e in ranges:
        if not (0 <= b < e) or e > k_cache.shape[0] or e > v_cache.shape[0]:
            raise ValueError(f"key range {(b, e)} is empty or outside the cache tensors")
    if out is None:
        out = torch.empty((n_q, hidden), dtype=torch.float32, device=dev)
    if lse is None:
        lse = torch.empty((n_heads, n_q), dtype=torch.float32, device=dev)
    _outputs(dev, n_q, hidden, n_heads, (("out", out, (n_q, hidden)), ("lse", lse, (n_heads, n_q))))
    arr = (_c_i64 * max(1, 2 * len(ranges)))(*[v for r in ranges for v in r])
    st = L.ispa_attn_ranges(_ptr(q), _ptr(k_cache), _ptr(v_cache), arr, len(ranges), int(n_q), int(n_heads),
                            int(head_dim), float(scale), _ptr(out), _ptr(lse), _stream(dev))
    _check(st, "ispa_attn_ranges")
    return out, lse


def attn_merge(out_a, lse_a, out_b, lse_b, out=None, lse=None):
    """Eq. 11-12 LSE fusion of two branches over disjoint key sets (ispa_attn_merge)."""
    L = lib()
    _require(out_a, "out_a", torch.float32)
    dev = out_a.device
    n_q, hidden = out_a.shape
    _require(lse_a, "lse_a", torch.float32, dev)
    n_heads = lse_a.shape[0]
    if hidden % n_heads:
        raise ValueError("hidden size is not a multiple of n_heads")
    for name, t, shape in (("out_b", out_b, (n_q, hidden)), ("lse_a", lse_a, (n_heads, n_q)),
                           ("lse_b", lse_b, (n_heads, n_q))):
        _require(t, name, torch.float32, dev)
        if tuple(t.shape) != shape:
            raise ValueError(f"{name} must have shape {shape}")
    if out is None:
        out = torch.empty((n_q, hidden), dtype=torch.float32, device=dev)
    if lse is None:
        lse = torch.empty((n_heads, n_q), dtype=torch.float32, device=dev)
    _outputs(dev, n_q, hidden, n_heads, (("out", out, (n_q, hidden)), ("lse", lse, (n_heads, n_q))))
    st = L.ispa_attn_merge(_ptr(out_a), _ptr(lse_a), _ptr(out_b), _ptr(lse_b), int(n_q), int(n_heads),
                           int(hidden // n_heads), _ptr(out), _ptr(lse), _stream(dev))
    _check(st, "ispa_attn_merge")
    return out, lse


_DT = {torch.bfloat16: DTYPE_BF16, torch.float32: DTYPE_F32}


class Stats:
    """Warmup statistics of one layer and the closed-form solve (ispa_stats_*).

    The device workspace is a torch uint8 tensor owned by this object.
    """

    def __init__(self, d_in, d_out, max_rows=4680, device=None, workspace=None):
        """``workspace`` optionally supplies the device workspace: a 256-byte
        aligned uint8 tensor of at least ispa_stats_workspace_bytes (StatsBatch
        passes equal slices of one buffer); by default this object allocates it."""
        L = lib()
        dev = torch.device("cuda") if device is None else torch.device(device)
        if dev.type != "cuda":
            raise ValueError("Stats lives on a HIP device")
        self.device = dev if dev.index is not None else torch.device("cuda", torch.cuda.current_device())
        self.d_in, self.d_out, self.max_rows = int(d_in), int(d_out), int(max_rows)
        self._h = ctypes.c_void_p(0)
        nbytes = L.ispa_stats_workspace_bytes(self.d_in, self.d_out, self.max_rows)
        if nbytes == 0:
            raise IspaError(ISPA_ERR_INVALID_ARG, "ispa_stats_workspace_bytes")
        if workspace is None:
            self.workspace = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
            pad = (-self.workspace.data_ptr()) % 256
            self._ws = self.workspace[pad:pad + nbytes]
        else:
            _require(workspace, "workspace", torch.uint8, self.device, ndim=1)
            if workspace.numel() < nbytes or workspace.data_ptr() % 256:
                raise ValueError(f"workspace must be 256-byte aligned and hold {nbytes} bytes")
            self.workspace = workspace
            self._ws = workspace[:nbytes]
        _check(L.ispa_stats_create(ctypes.byref(self._h), _ptr(self._ws), nbytes, self.d_in, self.d_out,
                                   self.max_rows, _stream(self.device)), "ispa_stats_create")

    def _handle(self):
        if not self._h:
            raise IspaError(ISPA_ERR_STATE, "Stats (destroyed)")
        return self._h

    def reset(self):
        _check(lib().ispa_stats_reset(self._handle()), "ispa_stats_reset")

    def accum(self, x, y_full, y_local):
        """Add rows: x [n, d_in] (bf16 or fp32); y_full, y_local [n, d_out] (same dtype)."""
        for name, t, cols in (("x", x, self.d_in), ("y_full", y_full, self.d_out), ("y_local", y_local, self.d_out)):
            if t.dtype not in _DT:
                raise TypeError(f"{name} must be bf16 or fp32")
            _require(t, name, t.dtype, self.device)
            if t.shape[1] != cols:
                raise ValueError(f"{name} must have {cols} columns")
        if y_full.dtype != y_local.dtype:
            raise TypeError("y_full and y_local must share a dtype")
        n = x.shape[0]
        if y_full.shape[0] != n or y_local.shape[0] != n:
            raise ValueError("row counts differ")
        _check(lib().ispa_accum_stats(self._handle(), _ptr(x), _DT[x.dtype], _ptr(y_full), _ptr(y_local),
                                      _DT[y_full.dtype], int(n)), "ispa_accum_stats")

    def views(self):
        """(G, C, s, n): G [d_in, d_in] (lower block triangle valid), C [d_in, d_out]
        fp32 views of the workspace, s a 1-element fp64 view, n the row count."""
        g, c, s = ctypes.c_void_p(), ctypes.c_void_p(), ctypes.c_void_p()
        n = ctypes.c_int64()
        _check(lib().ispa_stats_views(self._handle(), ctypes.byref(g), ctypes.byref(c), ctypes.byref(s),
                                      ctypes.byref(n)), "ispa_stats_views")
        base = self._ws.data_ptr()

        def view(ptr, count, dtype, shape):
            off = ptr - base
            size = torch.tensor([], dtype=dtype).element_size()
            return self._ws[off:off + count * size].view(dtype).view(*shape)

        G = view(g.value, self.d_in * self.d_in, torch.float32, (self.d_in, self.d_in))
        C = view(c.value, self.d_in * self.d_out, torch.float32, (self.d_in, self.d_out))
        S = view(s.value, 1, torch.float64, (1,))
        return G, C, S, n.value

    def solve(self, lam=1e-3, delta_w=None):
        """dW = (G + lam I)^-1 C and eps (Eq. 5-6). Synchronises the stream."""
        if delta_w is None:
            delta_w = torch.empty((self.d_in, self.d_out), dtype=torch.float32, device=self.device)
        _require(delta_w, "delta_w", torch.float32, self.device)
        eps = ctypes.c_double()
        _check(lib().ispa_solve_modulation(self._handle(), float(lam), _ptr(delta_w), ctypes.byref(eps)),
               "ispa_solve_modulation")
        return delta_w, eps.value

    def solve_async(self, lam=1e-3, delta_w=None, eps=None, status=None):
        """The same solve without waiting (ispa_solve_modulation_async): returns
        (delta_w, eps, status) with eps a device fp64 [1] and status a device
        int32 [1] (0, or 1 when G + lam I was not positive definite), valid once
        the handle's stream has run the work."""
        if delta_w is None:
            delta_w = torch.empty((self.d_in, self.d_out), dtype=torch.float32, device=self.device)
        if eps is None:
            eps = torch.empty((1,), dtype=torch.float64, device=self.device)
        if status is None:
            status = torch.empty((1,), dtype=torch.int32, device=self.device)
        _require(delta_w, "delta_w", torch.float32, self.device)
        _require(eps, "eps", torch.float64, self.device, ndim=1)
        _require(status, "status", torch.int32, self.device, ndim=1)
        _check(lib().ispa_solve_modulation_async(self._handle(), float(lam), _ptr(delta_w), _ptr(eps), _ptr(status)),
               "ispa_solve_modulation_async")
        return delta_w, eps, status

    def close(self):
        if self._h:
            lib().ispa_stats_destroy(self._h)
            self._h = ctypes.c_void_p(0)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class StatsBatch:
    """The warmup statistics of several layers on one workspace (equal
    256-byte-aligned slices, one statistics handle per layer), solved together
    by ispa_solve_modulation_batch. ``layers[i]`` is a Stats of layer i."""

    def __init__(self, n_layers, d_in, d_out, max_rows=4680, device=None):
        L = lib()
        dev = torch.device("cuda") if device is None else torch.device(device)
        if dev.type != "cuda":
            raise ValueError("StatsBatch lives on a HIP device")
        self.device = dev if dev.index is not None else torch.device("cuda", torch.cuda.current_device())
        self.n_layers = int(n_layers)
        self.d_in, self.d_out, self.max_rows = int(d_in), int(d_out), int(max_rows)
        if self.n_layers < 1:
            raise ValueError("n_layers must be positive")
        nbytes = L.ispa_stats_workspace_bytes(self.d_in, self.d_out, self.max_rows)
        if nbytes == 0:
            raise IspaError(ISPA_ERR_INVALID_ARG, "ispa_stats_workspace_bytes")
        self.stride = (nbytes + 255) // 256 * 256
        self.workspace = torch.empty(self.stride * self.n_layers + 256, dtype=torch.uint8, device=self.device)
        pad = (-self.workspace.data_ptr()) % 256
        self.layers = [Stats(self.d_in, self.d_out, self.max_rows, self.device,
                             workspace=self.workspace[pad + i * self.stride: pad + (i + 1) * self.stride])
                       for i in range(self.n_layers)]

    def solve(self, lam=1e-3, delta_w=None, eps=None, status=None):
        """dW, eps and the status word of every layer (ispa_solve_modulation_batch),
        without waiting: delta_w [n_layers, d_in, d_out] fp32, eps fp64 [n_layers],
        status int32 [n_layers] (0, or 1 when that layer's G + lam I was not
        positive definite), valid once the stream has run the work."""
        n = self.n_layers
        if delta_w is None:
            delta_w = torch.empty((n, self.d_in, self.d_out), dtype=torch.float32, device=self.device)
        if eps is None:
            eps = torch.empty((n,), dtype=torch.float64, device=self.device)
        if status is None:
            status = torch.empty((n,), dtype=torch.int32, device=self.device)
        _require(delta_w, "delta_w", torch.float32, self.device, ndim=3)
        if tuple(delta_w.shape) != (n, self.d_in, self.d_out):
            raise ValueError(f"delta_w must have shape {(n, self.d_in, self.d_out)}")
        _require(eps, "eps", torch.float64, self.device, ndim=1)
        _require(status, "status", torch.int32, self.device, ndim=1)
        if eps.shape[0] < n or status.shape[0] < n:
            raise ValueError("eps and status need n_layers entries")
        hs = (_c_p * n)(*[st._handle() for st in self.layers])
        _check(lib().ispa_solve_modulation_batch(hs, n, float(lam), _ptr(delta_w), _ptr(eps), _ptr(status)),
               "ispa_solve_modulation_batch")
        return delta_w, eps, status

    def close(self):
        for st in self.layers:
            st.close()


def select_layers(eps, k):
    """Indices of the k layers with the lowest eps (ispa_select_layers, Sec. 3.3)."""
    L = lib()
    vals = [float(e) for e in eps]
    arr = (ctypes.c_double * max(1, len(vals)))(*vals)
    out = (_c_i32 * max(1, int(k)))()
    _check(L.ispa_select_layers(arr, len(vals), int(k), out), "ispa_select_layers")
    return [int(out[i]) for i in range(int(k))]


def inject_modulation(weight, delta_w, transposed=False):
    """In-place W += dW (or dW^T for a [d_out, d_in] linear weight); ispa_inject_modulation."""
    L = lib()
    if weight.dtype not in _DT:
        raise TypeError("weight must be bf16 or fp32")
    _require(weight, "weight", weight.dtype)
    _require(delta_w, "delta_w", torch.float32, weight.device)
    d_in, d_out = delta_w.shape
    want = (d_out, d_in) if transposed else (d_in, d_out)
    if tuple(weight.shape) != want:
        raise ValueError(f"weight must have shape {want}")
    st = L.ispa_inject_modulation(_ptr(weight), _DT[weight.dtype], int(bool(transposed)), _ptr(delta_w), int(d_in),
                                  int(d_out), _stream(weight.device))
    _check(st, "ispa_inject_modulation")
    return weight


class LocalKV:
    """An L-Layer's KV cache after the permanent eviction (ispa_kv_evict /
    ispa_kv_ring_append): the sink rows and a ring of the `window` most recent
    keys, attended as one contiguous set of rows."""

    def __init__(self, k_cache, v_cache, cache_len, window, sink_len=0, ring=None):
        """``ring`` optionally supplies the (k, v) ring tensors, each at least
        [min(sink_len, cache_len) + window, hidden] bf16 (reused instead of allocated)."""
        L = lib()
        _require(k_cache, "k_cache", torch.bfloat16)
        dev = k_cache.device
        _require(v_cache, "v_cache", torch.bfloat16, dev)
        if k_cache.shape != v_cache.shape or k_cache.shape[0] < cache_len:
            raise ValueError("k/v caches must have the same shape and hold cache_len rows")
        self.hidden = int(k_cache.shape[1])
        self.window = int(window)
        self.sink = int(min(sink_len, cache_len))
        shape = (self.sink + self.window, self.hidden)
        if ring is None:
            self.k = torch.empty(shape, dtype=torch.bfloat16, device=dev)
            self.v = torch.empty_like(self.k)
        else:
            self.k, self.v = ring
            for name, t in (("ring k", self.k), ("ring v", self.v)):
                _require(t, name, torch.bfloat16, dev)
                if t.shape[0] < shape[0] or t.shape[1] != shape[1]:
                    raise ValueError(f"{name} must be at least {shape}")
        rows = _c_i64(0)
        st = L.ispa_kv_evict(_ptr(k_cache), _ptr(v_cache), int(cache_len), self.window, int(sink_len), self.hidden,
                             _ptr(self.k), _ptr(self.v), ctypes.byref(rows), _stream(dev))
        _check(st, "ispa_kv_evict")
        self.head = int(rows.value) - self.sink

    @property
    def rows(self):
        """Filled ring rows (sink + window keys held)."""
        return self.sink + min(self.head, self.window)

    def append(self, k_new, v_new):
        L = lib()
        _require(k_new, "k_new", torch.bfloat16, self.k.device)
        _require(v_new, "v_new", torch.bfloat16, self.k.device)
        if k_new.shape != v_new.shape or k_new.shape[1] != self.hidden:
            raise ValueError("new keys/values must be [n, hidden] of the cache's hidden size")
        st = L.ispa_kv_ring_append(_ptr(self.k), _ptr(self.v), self.sink, self.window, self.head, _ptr(k_new),
                                   _ptr(v_new), int(k_new.shape[0]), self.hidden, _stream(self.k.device))
        _check(st, "ispa_kv_ring_append")
        self.head += int(k_new.shape[0])

    def attend(self, q, n_heads, **kw):
        """Attention of q over every key the L-Layer holds (append the current
        chunk first: the keys of the current chunk are part of its local set)."""
        n = self.rows
        return attn_chunk(q, self.k, self.v, n, n, n_heads, **kw)


def project(a, weight, out=None, out_dtype=torch.float32):
    """y = a weight^T with weight in the linear-layer layout [d_out, d_in] (ispa_project)."""
    L = lib()
    _require(a, "a", torch.bfloat16)
    _require(weight, "weight", torch.bfloat16, a.device)
    n, d_in = a.shape
    d_out, k = weight.shape
    if k != d_in:
        raise ValueError("weight must be [d_out, d_in] with the d_in of a")
    if out is None:
        out = torch.empty((n, d_out), dtype=out_dtype, device=a.device)
    if out.dtype not in _DT:
        raise TypeError("out must be fp32 or bf16")
    _require(out, "out", out.dtype, a.device)
    if tuple(out.shape) != (n, d_out):
        raise ValueError(f"out must have shape {(n, d_out)}")
    st = L.ispa_project(_ptr(a), _ptr(weight), int(n), int(d_in), int(d_out), _ptr(out), _DT[out.dtype],
                        _stream(a.device))
    _check(st, "ispa_project")
    return out


def quantize_rows(x, q=None, scale=None):
    """Symmetric per-row int8 codes and fp32 scales of x [rows, cols], bf16 or
    fp32 (ispa_quantize_rows). Returns (q, scale)."""
    L = lib()
    if not isinstance(x, torch.Tensor) or x.dtype not in _DT:
        raise TypeError("x must be a bf16 or fp32 torch.Tensor")
    _require(x, "x", x.dtype)
    rows, cols = x.shape
    if q is None:
        q = torch.empty((rows, cols), dtype=torch.int8, device=x.device)
    if scale is None:
        scale = torch.empty((rows,), dtype=torch.float32, device=x.device)
    _require(q, "q", torch.int8, x.device)
    _require(scale, "scale", torch.float32, x.device, ndim=1)
    if tuple(q.shape) != (rows, cols) or scale.shape[0] != rows:
        raise ValueError("q must be [rows, cols] and scale [rows]")
    st = L.ispa_quantize_rows(_ptr(x), _DT[x.dtype], int(rows), int(cols), _ptr(q), _ptr(scale), _stream(x.device))
    _check(st, "ispa_quantize_rows")
    return q, scale


def project_w8a8(q_a, scale_a, q_w, scale_w, out=None, out_dtype=torch.float32):
    """y = (q_a q_w^T) * scale_a[row] * scale_w[col] (ispa_project_w8a8): the
    W8A8 form of project, with the codes of quantize_rows."""
    L = lib()
    _require(q_a, "q_a", torch.int8)
    dev = q_a.device
    _require(q_w, "q_w", torch.int8, dev)
    _require(scale_a, "scale_a", torch.float32, dev, ndim=1)
    _require(scale_w, "scale_w", torch.float32, dev, ndim=1)
    n, d_in = q_a.shape
    d_out, k = q_w.shape
    if k != d_in or scale_a.shape[0] != n or scale_w.shape[0] != d_out:
        raise ValueError("q_w must be [d_out, d_in], scale_a [n] and scale_w [d_out]")
    if out is None:
        out = torch.empty((n, d_out), dtype=out_dtype, device=dev)
    if out.dtype not in _DT:
        raise TypeError("out must be fp32 or bf16")
    _require(out, "out", out.dtype, dev)
    if tuple(out.shape) != (n, d_out):
        raise ValueError(f"out must have shape {(n, d_out)}")
    st = L.ispa_project_w8a8(_ptr(q_a), _ptr(scale_a), _ptr(q_w), _ptr(scale_w), int(n), int(d_in), int(d_out),
                             _ptr(out), _DT[out.dtype], _stream(dev))
    _check(st, "ispa_project_w8a8")
    return out
