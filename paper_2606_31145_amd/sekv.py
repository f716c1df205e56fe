"""ctypes binding of libsekv.so (the C ABI declared in include/sekv.h).

Argument marshalling only: torch allocates device memory and provides the stream;
every step of the decode path runs in the library's HIP kernels.  Importing this
module loads the library and raises if it has not been built.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
# SEKV_LIB=trace selects the diagnostic phase-trace build of the same sources
LIB_PATH = os.path.join(_PKG, "libsekv_trace.so" if os.environ.get("SEKV_LIB") == "trace"
                        else "libsekv.so")

SEKV_OK, SEKV_ERR_INVALID_ARG, SEKV_ERR_UNSUPPORTED, SEKV_ERR_WORKSPACE, SEKV_ERR_HIP = range(5)
SEKV_F32, SEKV_BF16 = 0, 1
SEKV_ZOOM_DEFAULT, SEKV_ZOOM_FACTORED = 0, 1
SEKV_TIER_GATHER, SEKV_TIER_MEMCPY = 0, 1
TIER_MODES = {"gather": SEKV_TIER_GATHER, "memcpy": SEKV_TIER_MEMCPY}
DTYPE_CODES = {"f32": SEKV_F32, "bf16": SEKV_BF16}

EXPORTED = ("sekv_status_string", "sekv_last_error", "sekv_phase_trace", "sekv_check_dims",
            "sekv_workspace_size",
            "sekv_workspace_init", "sekv_workspace_status", "sekv_route_topk",
            "sekv_zoom_attend", "sekv_decode_step", "sekv_graph_create", "sekv_graph_launch",
            "sekv_graph_destroy", "sekv_tier_create", "sekv_tier_destroy",
            "sekv_tier_staging_size", "sekv_tier_last_copy", "sekv_decode_step_tiered",
            "sekv_validate_cache", "sekv_decode_step_noalloc", "sekv_route_gated",
            "sekv_decode_step_gated", "sekv_segment_workspace_size", "sekv_segment",
            "sekv_build_layout", "sekv_build_cache", "sekv_decode_layers_tiered",
            "sekv_tier_layer_stats")


class SekvError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_status_name(status)}: {message}")
        self.status = status


class Dims(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("rank", ctypes.c_int32), ("top_k", ctypes.c_int32),
                ("max_anchors", ctypes.c_int32), ("max_spans", ctypes.c_int32),
                ("max_span_len", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("out_dtype", ctypes.c_int32), ("flags", ctypes.c_int32),
                ("softmax_scale", ctypes.c_double)]


class CacheStruct(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("anchor_k", ctypes.c_void_p),
                ("anchor_v", ctypes.c_void_p), ("n_anchors", ctypes.c_void_p),
                ("sum_k", ctypes.c_void_p), ("sum_v", ctypes.c_void_p),
                ("n_spans", ctypes.c_void_p), ("span_len", ctypes.c_void_p),
                ("span_logsize", ctypes.c_void_p), ("factors", ctypes.c_void_p),
                ("factors_bytes", ctypes.c_int64), ("block_off", ctypes.c_void_p),
                ("block_rank", ctypes.c_void_p)]


class HostFactorsStruct(ctypes.Structure):
    _fields_ = [("arena", ctypes.c_void_p), ("arena_bytes", ctypes.c_int64),
                ("block_off", ctypes.c_void_p), ("span_len", ctypes.c_void_p),
                ("block_rank", ctypes.c_void_p)]


class GateStruct(ctypes.Structure):
    _fields_ = [("route_dim", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("budget_tokens", ctypes.c_int64), ("proj", ctypes.c_void_p),
                ("sum_route", ctypes.c_void_p), ("thresholds", ctypes.c_void_p)]


class BuildDims(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("max_tokens", ctypes.c_int32),
                ("rank", ctypes.c_int32), ("sketch", ctypes.c_int32),
                ("min_span", ctypes.c_int32), ("window", ctypes.c_int32),
                ("sweeps", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("power", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("alpha", ctypes.c_double)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
    lib = ctypes.CDLL(LIB_PATH)
    P, VP, SZ, I32P = ctypes.POINTER, ctypes.c_void_p, ctypes.c_size_t, ctypes.POINTER(ctypes.c_int32)
    lib.sekv_status_string.restype = ctypes.c_char_p
    lib.sekv_status_string.argtypes = [ctypes.c_int]
    lib.sekv_last_error.restype = ctypes.c_char_p
    lib.sekv_last_error.argtypes = []
    lib.sekv_phase_trace.restype = ctypes.c_int
    lib.sekv_phase_trace.argtypes = [VP, SZ]
    lib.sekv_check_dims.restype = ctypes.c_int
    lib.sekv_check_dims.argtypes = [P(Dims)]
    lib.sekv_workspace_size.restype = SZ
    lib.sekv_workspace_size.argtypes = [P(Dims)]
    lib.sekv_workspace_init.restype = ctypes.c_int
    lib.sekv_workspace_init.argtypes = [VP, SZ, VP]
    lib.sekv_workspace_status.restype = ctypes.c_int
    lib.sekv_workspace_status.argtypes = [VP, SZ, VP, I32P]
    lib.sekv_route_topk.restype = ctypes.c_int
    lib.sekv_route_topk.argtypes = [P(Dims), P(CacheStruct), VP, VP, VP, SZ, VP]
    lib.sekv_zoom_attend.restype = ctypes.c_int
    lib.sekv_zoom_attend.argtypes = [P(Dims), P(CacheStruct), VP, VP, VP, VP, SZ, VP]
    lib.sekv_decode_step.restype = ctypes.c_int
    lib.sekv_decode_step.argtypes = [P(Dims), P(CacheStruct), VP, VP, VP, SZ, VP]
    lib.sekv_graph_create.restype = ctypes.c_int
    lib.sekv_graph_create.argtypes = [P(Dims), P(CacheStruct), ctypes.c_int32, VP, VP, VP, SZ,
                                      P(VP)]
    lib.sekv_graph_launch.restype = ctypes.c_int
    lib.sekv_graph_launch.argtypes = [VP, VP]
    lib.sekv_graph_destroy.restype = ctypes.c_int
    lib.sekv_graph_destroy.argtypes = [VP]
    lib.sekv_tier_create.restype = ctypes.c_int
    lib.sekv_tier_create.argtypes = [P(Dims), ctypes.c_int32, P(VP)]
    lib.sekv_tier_destroy.restype = ctypes.c_int
    lib.sekv_tier_destroy.argtypes = [VP]
    lib.sekv_tier_staging_size.restype = SZ
    lib.sekv_tier_staging_size.argtypes = [VP]
    lib.sekv_tier_last_copy.restype = ctypes.c_int
    lib.sekv_tier_last_copy.argtypes = [VP, P(ctypes.c_int64), I32P, P(ctypes.c_float)]
    lib.sekv_decode_step_tiered.restype = ctypes.c_int
    lib.sekv_decode_step_tiered.argtypes = [P(Dims), P(CacheStruct), P(HostFactorsStruct), VP, VP,
                                            VP, VP, SZ, VP, VP]
    lib.sekv_decode_step_noalloc.restype = ctypes.c_int
    lib.sekv_decode_step_noalloc.argtypes = [P(Dims), P(CacheStruct), VP, VP, VP]
    lib.sekv_route_gated.restype = ctypes.c_int
    lib.sekv_route_gated.argtypes = [P(Dims), P(CacheStruct), P(GateStruct), VP, VP, VP, SZ, VP]
    lib.sekv_decode_step_gated.restype = ctypes.c_int
    lib.sekv_decode_step_gated.argtypes = [P(Dims), P(CacheStruct), P(GateStruct), VP, VP, VP, SZ, VP]
    lib.sekv_validate_cache.restype = ctypes.c_int
    lib.sekv_validate_cache.argtypes = [P(Dims), P(CacheStruct)]
    lib.sekv_decode_layers_tiered.restype = ctypes.c_int
    lib.sekv_decode_layers_tiered.argtypes = [P(Dims), P(CacheStruct), P(HostFactorsStruct), ctypes.c_int32,
                                              ctypes.c_int32, VP, VP, VP, VP, SZ, VP, VP]
    lib.sekv_tier_layer_stats.restype = ctypes.c_int
    lib.sekv_tier_layer_stats.argtypes = [VP, P(ctypes.c_int64)]
    lib.sekv_segment_workspace_size.restype = ctypes.c_size_t
    lib.sekv_segment_workspace_size.argtypes = [P(BuildDims)]
    lib.sekv_segment.restype = ctypes.c_int
    lib.sekv_segment.argtypes = [P(BuildDims), VP, VP, VP, VP, VP, VP, VP, VP, SZ, VP]
    lib.sekv_build_layout.restype = ctypes.c_int64
    lib.sekv_build_layout.argtypes = [P(BuildDims), ctypes.c_int32, VP, VP, VP, VP]
    lib.sekv_build_cache.restype = ctypes.c_int
    lib.sekv_build_cache.argtypes = [P(BuildDims), VP, VP, VP, VP, VP, VP, VP, VP, VP, VP,
                                     ctypes.c_int32, ctypes.c_int32, VP, VP, VP, VP, VP, VP, VP,
                                     ctypes.c_int64, VP, VP, SZ, VP]
    return lib


LIB = _load()


def _status_name(status: int) -> str:
    try:
        return LIB.sekv_status_string(int(status)).decode()
    except Exception:
        return f"status {status}"


def _check(status: int):
    if status != SEKV_OK:
        raise SekvError(status, LIB.sekv_last_error().decode())


def _ptr(t) -> int | None:
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("expected a torch tensor")
    if not t.is_contiguous():
        raise ValueError("tensors passed to the library must be contiguous")
    return t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def make_dims(*, batch, n_q_heads, n_kv_heads, head_dim, rank, top_k, max_anchors, max_spans,
              max_span_len, dtype, softmax_scale, out_dtype=None, zoom=SEKV_ZOOM_DEFAULT) -> Dims:
    dt = DTYPE_CODES[dtype] if isinstance(dtype, str) else int(dtype)
    if out_dtype is None:
        odt = dt
    else:
        odt = DTYPE_CODES[out_dtype] if isinstance(out_dtype, str) else int(out_dtype)
    return Dims(batch, n_q_heads, n_kv_heads, head_dim, rank, top_k, max_anchors, max_spans,
                max_span_len, dt, odt, int(zoom), float(softmax_scale))


def phase_trace(buf=None):
    """sekv_phase_trace: attach a device int64 buffer (or detach with None)."""
    if buf is None:
        _check(LIB.sekv_phase_trace(None, 0))
    else:
        _check(LIB.sekv_phase_trace(_ptr(buf), buf.numel() * buf.element_size()))


def check_dims(dims: Dims):
    _check(LIB.sekv_check_dims(ctypes.byref(dims)))


def workspace_size(dims: Dims) -> int:
    return int(LIB.sekv_workspace_size(ctypes.byref(dims)))


class Workspace:
    """A zero-initialised device workspace for a dims (256-byte aligned view of a torch buffer)."""

    def __init__(self, dims: Dims, device="cuda", stream=None, nbytes: int | None = None):
        need = workspace_size(dims) if nbytes is None else int(nbytes)
        if need == 0:
            check_dims(dims)
        need = (need + 15) // 16 * 16
        self._buf = torch.empty(need + 256, dtype=torch.uint8, device=device)
        off = (-self._buf.data_ptr()) % 256
        self.tensor = self._buf[off:off + need]
        self.nbytes = need
        _check(LIB.sekv_workspace_init(self.tensor.data_ptr(), need, _stream(stream)))

    @property
    def ptr(self) -> int:
        return self.tensor.data_ptr()

    def status(self, stream=None) -> int:
        bits = ctypes.c_int32(0)
        _check(LIB.sekv_workspace_status(self.ptr, self.nbytes, _stream(stream), ctypes.byref(bits)))
        return int(bits.value)


_TORCH_STORAGE = {"f32": torch.float32, "bf16": torch.bfloat16}


def _to_device(arr: np.ndarray, dtype: str | None, device) -> torch.Tensor:
    a = np.ascontiguousarray(arr)
    if dtype == "bf16":
        t = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(a)
    return t.to(device)


class DeviceCache:
    """Device tensors of one layer's stored cache, laid out as sekv_cache describes."""

    FIELDS = ("q", "anchor_k", "anchor_v", "n_anchors", "sum_k", "sum_v", "n_spans", "span_len",
              "span_logsize", "factors", "block_off")

    def __init__(self, tensors: dict, dtype: str):
        missing = [f for f in self.FIELDS if f not in tensors]
        if missing:
            raise ValueError(f"missing cache fields: {missing}")
        self.t = dict(tensors)
        self.dtype = dtype
        self._struct = None

    @classmethod
    def from_arrays(cls, arrays: dict, dtype: str, device="cuda", factors_device=None):
        """Upload numpy arrays (storage-typed; bf16 as uint16 bit patterns)."""
        t = {}
        for f in ("q", "anchor_k", "anchor_v", "sum_k", "sum_v"):
            t[f] = _to_device(arrays[f], dtype, device)
        for f in ("n_anchors", "n_spans", "span_len"):
            t[f] = torch.from_numpy(np.ascontiguousarray(arrays[f], dtype=np.int32)).to(device)
        t["span_logsize"] = torch.from_numpy(np.ascontiguousarray(arrays["span_logsize"],
                                                                  dtype=np.float64)).to(device)
        t["block_off"] = torch.from_numpy(np.ascontiguousarray(arrays["block_off"],
                                                               dtype=np.int64)).to(device)
        t["factors"] = torch.from_numpy(np.ascontiguousarray(arrays["factors"],
                                                             dtype=np.uint8)).to(
            factors_device or device)
        if arrays.get("block_rank") is not None:
            t["block_rank"] = torch.from_numpy(np.ascontiguousarray(arrays["block_rank"],
                                                                    dtype=np.int32)).to(device)
        return cls(t, dtype)

    def struct(self) -> CacheStruct:
        t = self.t
        return CacheStruct(_ptr(t["q"]), _ptr(t["anchor_k"]), _ptr(t["anchor_v"]),
                           _ptr(t["n_anchors"]), _ptr(t["sum_k"]), _ptr(t["sum_v"]),
                           _ptr(t["n_spans"]), _ptr(t["span_len"]), _ptr(t["span_logsize"]),
                           _ptr(t["factors"]), int(t["factors"].numel()), _ptr(t["block_off"]),
                           _ptr(t.get("block_rank")))


def _alloc(shape, dtype, device):
    return torch.empty(shape, dtype=dtype, device=device)


def route_topk(dims: Dims, cache: DeviceCache, ws: Workspace, sel=None, logits=None,
               want_logits: bool = True, stream=None):
    """sekv_route_topk: returns (sel int32 [B][Hkv][k], logits float [B][Hq][M_max] or None)."""
    dev = cache.t["q"].device
    if sel is None:
        sel = _alloc((dims.batch, dims.n_kv_heads, max(dims.top_k, 0)), torch.int32, dev)
    if logits is None and want_logits:
        logits = _alloc((dims.batch, dims.n_q_heads, dims.max_spans), torch.float32, dev)
    cs = cache.struct()
    _check(LIB.sekv_route_topk(ctypes.byref(dims), ctypes.byref(cs), _ptr(sel), _ptr(logits),
                               ws.ptr, ws.nbytes, _stream(stream)))
    return sel, logits


def _out_tensor(dims: Dims, dev):
    dt = torch.float32 if dims.out_dtype == SEKV_F32 else torch.bfloat16
    return _alloc((dims.batch, dims.n_q_heads, dims.head_dim), dt, dev)


def zoom_attend(dims: Dims, cache: DeviceCache, sel, logits, ws: Workspace, out=None, stream=None):
    """sekv_zoom_attend: returns out [B][Hq][d] in out_dtype."""
    if out is None:
        out = _out_tensor(dims, cache.t["q"].device)
    cs = cache.struct()
    _check(LIB.sekv_zoom_attend(ctypes.byref(dims), ctypes.byref(cs), _ptr(sel), _ptr(logits),
                                _ptr(out), ws.ptr, ws.nbytes, _stream(stream)))
    return out


def decode_step(dims: Dims, cache: DeviceCache, ws: Workspace, sel=None, out=None, stream=None):
    """sekv_decode_step: returns (sel, out)."""
    dev = cache.t["q"].device
    if sel is None:
        sel = _alloc((dims.batch, dims.n_kv_heads, max(dims.top_k, 0)), torch.int32, dev)
    if out is None:
        out = _out_tensor(dims, dev)
    cs = cache.struct()
    _check(LIB.sekv_decode_step(ctypes.byref(dims), ctypes.byref(cs), _ptr(sel), _ptr(out),
                                ws.ptr, ws.nbytes, _stream(stream)))
    return sel, out


class DeviceGate:
    """Device tensors of the learned-routing parameters, laid out as sekv_gate describes."""

    def __init__(self, route_dim: int, proj, sum_route, thresholds, budget_tokens: int):
        self.route_dim = int(route_dim)
        self.proj, self.sum_route, self.thresholds = proj, sum_route, thresholds
        self.budget_tokens = int(budget_tokens)

    @classmethod
    def from_arrays(cls, route_dim, proj, sum_route, thresholds, budget_tokens, dtype: str,
                    device="cuda"):
        """Upload storage-typed numpy arrays (bf16 as uint16 bit patterns)."""
        thr = torch.from_numpy(np.ascontiguousarray(thresholds, dtype=np.float64)).to(device)
        return cls(route_dim, _to_device(proj, dtype, device), _to_device(sum_route, dtype, device),
                   thr, budget_tokens)

    def struct(self, budget_tokens=None) -> GateStruct:
        bt = self.budget_tokens if budget_tokens is None else int(budget_tokens)
        return GateStruct(self.route_dim, 0, bt, _ptr(self.proj), _ptr(self.sum_route),
                          _ptr(self.thresholds))


def route_gated(dims: Dims, cache: DeviceCache, gate: DeviceGate, ws: Workspace, sel=None,
                gate_logits=None, want_logits: bool = False, stream=None):
    """sekv_route_gated: returns (sel int32 [B][Hkv][k], gate logits float64 [B][Hq][M_max] or None)."""
    dev = cache.t["q"].device
    if sel is None:
        sel = _alloc((dims.batch, dims.n_kv_heads, max(dims.top_k, 0)), torch.int32, dev)
    if gate_logits is None and want_logits:
        gate_logits = _alloc((dims.batch, dims.n_q_heads, dims.max_spans), torch.float64, dev)
    cs, gs = cache.struct(), gate.struct()
    _check(LIB.sekv_route_gated(ctypes.byref(dims), ctypes.byref(cs), ctypes.byref(gs), _ptr(sel),
                                _ptr(gate_logits), ws.ptr, ws.nbytes, _stream(stream)))
    return sel, gate_logits


def decode_step_gated(dims: Dims, cache: DeviceCache, gate: DeviceGate, ws: Workspace, sel=None,
                      out=None, stream=None):
    """sekv_decode_step_gated: returns (sel, out)."""
    dev = cache.t["q"].device
    if sel is None:
        sel = _alloc((dims.batch, dims.n_kv_heads, max(dims.top_k, 0)), torch.int32, dev)
    if out is None:
        out = _out_tensor(dims, dev)
    cs, gs = cache.struct(), gate.struct()
    _check(LIB.sekv_decode_step_gated(ctypes.byref(dims), ctypes.byref(cs), ctypes.byref(gs),
                                      _ptr(sel), _ptr(out), ws.ptr, ws.nbytes, _stream(stream)))
    return sel, out


NOALLOC_MAX_WORKSPACE = 16 << 20


def decode_step_noalloc(dims: Dims, cache: DeviceCache, sel=None, out=None, stream=None):
    """sekv_decode_step_noalloc (the library's static device workspace): returns (sel, out)."""
    dev = cache.t["q"].device
    if sel is None:
        sel = _alloc((dims.batch, dims.n_kv_heads, max(dims.top_k, 0)), torch.int32, dev)
    if out is None:
        out = _out_tensor(dims, dev)
    cs = cache.struct()
    _check(LIB.sekv_decode_step_noalloc(ctypes.byref(dims), ctypes.byref(cs), _ptr(sel), _ptr(out),
                                        _stream(stream)))
    return sel, out


class LayerGraph:
    """sekv_graph_*: one decode step over several layers, captured once as a HIP graph.

    caches: one DeviceCache per layer (same shapes).  sel [L][B][Hkv][k] and out
    [L][B][Hq][d] are allocated here unless given.  The graph holds raw pointers, so this
    object keeps every tensor it was built from alive.
    """

    def __init__(self, dims: Dims, caches, ws: Workspace, sel=None, out=None):
        caches = list(caches)
        if not caches:
            raise ValueError("need at least one layer")
        L = len(caches)
        dev = caches[0].t["q"].device
        if sel is None:
            sel = _alloc((L, dims.batch, dims.n_kv_heads, max(dims.top_k, 0)), torch.int32, dev)
        if out is None:
            dt = torch.float32 if dims.out_dtype == SEKV_F32 else torch.bfloat16
            out = _alloc((L, dims.batch, dims.n_q_heads, dims.head_dim), dt, dev)
        self.dims, self.caches, self.ws, self.sel, self.out = dims, caches, ws, sel, out
        self._structs = (CacheStruct * L)(*[c.struct() for c in caches])
        h = ctypes.c_void_p(0)
        _check(LIB.sekv_graph_create(ctypes.byref(dims), self._structs, L, _ptr(sel), _ptr(out),
                                     ws.ptr, ws.nbytes, ctypes.byref(h)))
        self._h = h

    def launch(self, stream=None):
        if not self._h:
            raise RuntimeError("graph destroyed")
        _check(LIB.sekv_graph_launch(self._h, _stream(stream)))
        return self.sel, self.out

    def destroy(self):
        if self._h:
            h, self._h = self._h, ctypes.c_void_p(0)
            _check(LIB.sekv_graph_destroy(h))

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


class HostFactors:
    """The factor arena in pinned host memory plus host copies of block_off, span_len and
    (for per-block ranks) block_rank."""

    def __init__(self, factors: np.ndarray, block_off: np.ndarray, span_len: np.ndarray,
                 block_rank: np.ndarray | None = None):
        a = np.ascontiguousarray(factors, dtype=np.uint8)
        self.arena = torch.empty(a.nbytes, dtype=torch.uint8, pin_memory=True)
        self.arena.numpy()[:] = a
        self.block_off = np.ascontiguousarray(block_off, dtype=np.int64)
        self.span_len = np.ascontiguousarray(span_len, dtype=np.int32)
        self.block_rank = None if block_rank is None else np.ascontiguousarray(block_rank, dtype=np.int32)

    def struct(self) -> HostFactorsStruct:
        return HostFactorsStruct(self.arena.data_ptr(), int(self.arena.numel()),
                                 self.block_off.ctypes.data, self.span_len.ctypes.data,
                                 None if self.block_rank is None else self.block_rank.ctypes.data)


class Tier:
    """sekv_tier_*: pinned mirrors, device staging and events for tiered steps.

    mode "gather" (device-planned gather kernel, no host wait) or "memcpy" (host-planned
    hipMemcpyAsync per run of neighbouring blocks)."""

    def __init__(self, dims: Dims, mode: str = "gather"):
        h = ctypes.c_void_p(0)
        _check(LIB.sekv_tier_create(ctypes.byref(dims), TIER_MODES[mode], ctypes.byref(h)))
        self._h = h
        self.dims = dims
        self.mode = mode

    @property
    def staging_bytes(self) -> int:
        return int(LIB.sekv_tier_staging_size(self._h))

    def layer_stats(self):
        """Counters of the last layered call: (critical bytes, critical blocks, prefetched
        bytes, prefetched blocks)."""
        st = (ctypes.c_int64 * 4)()
        _check(LIB.sekv_tier_layer_stats(self._h, st))
        return tuple(int(x) for x in st)

    def last_copy(self):
        """(bytes, copies, milliseconds) of the last step's host-to-device copies."""
        nb, nc, ms = ctypes.c_int64(0), ctypes.c_int32(0), ctypes.c_float(0)
        _check(LIB.sekv_tier_last_copy(self._h, ctypes.byref(nb), ctypes.byref(nc), ctypes.byref(ms)))
        return int(nb.value), int(nc.value), float(ms.value)

    def destroy(self):
        if self._h:
            h, self._h = self._h, ctypes.c_void_p(0)
            _check(LIB.sekv_tier_destroy(h))

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def decode_layers_tiered(dims: Dims, caches, hosts, tier: Tier, ws: Workspace, prefetch: bool = True,
                         sel=None, out=None, stream=None, side=None):
    """sekv_decode_layers_tiered over len(caches) layers: returns (sel [L][B][Hkv][k],
    out [L][B][Hq][d]).  `side` is the copy stream."""
    if side is None:
        raise ValueError("a side stream is needed for the copies")
    L = len(caches)
    if len(hosts) != L:
        raise ValueError("one host arena per layer")
    dev = caches[0].t["q"].device
    if sel is None:
        sel = _alloc((L, dims.batch, dims.n_kv_heads, max(dims.top_k, 0)), torch.int32, dev)
    if out is None:
        o = _out_tensor(dims, dev)
        out = _alloc((L,) + tuple(o.shape), o.dtype, dev)
    cs = (CacheStruct * L)(*[c.struct() for c in caches])
    hs = (HostFactorsStruct * L)(*[h.struct() for h in hosts])
    _check(LIB.sekv_decode_layers_tiered(ctypes.byref(dims), cs, hs, L, int(bool(prefetch)), tier._h,
                                         _ptr(sel), _ptr(out), ws.ptr, ws.nbytes, _stream(stream),
                                         _stream(side)))
    return sel, out


def validate_cache(dims: Dims, arrays: dict):
    """sekv_validate_cache on host copies (numpy arrays, storage-typed as for
    DeviceCache.from_arrays).  Raises SekvError with the first violation."""
    keep = {}
    for f in ("q", "anchor_k", "anchor_v", "sum_k", "sum_v"):
        keep[f] = np.ascontiguousarray(arrays[f])
    keep["n_anchors"] = np.ascontiguousarray(arrays["n_anchors"], dtype=np.int32)
    keep["n_spans"] = np.ascontiguousarray(arrays["n_spans"], dtype=np.int32)
    keep["span_len"] = np.ascontiguousarray(arrays["span_len"], dtype=np.int32)
    keep["span_logsize"] = np.ascontiguousarray(arrays["span_logsize"], dtype=np.float64)
    keep["block_off"] = np.ascontiguousarray(arrays["block_off"], dtype=np.int64)
    keep["factors"] = np.ascontiguousarray(arrays["factors"], dtype=np.uint8)
    if arrays.get("block_rank") is not None:
        keep["block_rank"] = np.ascontiguousarray(arrays["block_rank"], dtype=np.int32)
    c = lambda f: keep[f].ctypes.data if f in keep and keep[f].size else None  # noqa: E731
    cs = CacheStruct(c("q"), c("anchor_k"), c("anchor_v"), c("n_anchors"), c("sum_k"), c("sum_v"),
                     c("n_spans"), c("span_len"), c("span_logsize"), c("factors"),
                     int(keep["factors"].nbytes), c("block_off"), c("block_rank"))
    _check(LIB.sekv_validate_cache(ctypes.byref(dims), ctypes.byref(cs)))


def decode_step_tiered(dims: Dims, cache: DeviceCache, host: HostFactors, tier: Tier,
                       ws: Workspace, sel=None, out=None, stream=None, side=None):
    """sekv_decode_step_tiered: returns (sel, out).  `side` is the copy stream."""
    dev = cache.t["q"].device
    if sel is None:
        sel = _alloc((dims.batch, dims.n_kv_heads, max(dims.top_k, 0)), torch.int32, dev)
    if out is None:
        out = _out_tensor(dims, dev)
    if side is None:
        raise ValueError("a side stream is needed for the copies")
    cs = cache.struct()
    hs = host.struct()
    _check(LIB.sekv_decode_step_tiered(ctypes.byref(dims), ctypes.byref(cs), ctypes.byref(hs),
                                       tier._h, _ptr(sel), _ptr(out), ws.ptr, ws.nbytes,
                                       _stream(stream), _stream(side)))
    return sel, out


# ---------------------------------------------------------------------------
# prefill-side builder
# ---------------------------------------------------------------------------

def make_build_dims(*, batch, n_kv_heads, head_dim, max_tokens, rank, sketch, min_span, window,
                    dtype, alpha=1.0, sweeps=8, power=1) -> BuildDims:
    dt = DTYPE_CODES[dtype] if isinstance(dtype, str) else int(dtype)
    return BuildDims(batch, n_kv_heads, head_dim, max_tokens, rank, sketch, min_span, window,
                     sweeps, dt, power, 0, float(alpha))


def segment(bd: BuildDims, surprisal, n_tokens, stream=None) -> dict:
    """sekv_segment: surprisal float32 [B][N_max] and n_tokens int32 [B] on the device.
    Returns device tensors n_anchors, anchor_idx, n_spans, span_start, span_len."""
    dev = surprisal.device
    B, N = bd.batch, bd.max_tokens
    ws_bytes = int(LIB.sekv_segment_workspace_size(ctypes.byref(bd)))
    if ws_bytes == 0 and B > 0:
        _check(LIB.sekv_segment(ctypes.byref(bd), None, None, None, None, None, None, None,
                                None, 0, None))
    out = {"n_anchors": _alloc((B,), torch.int32, dev), "anchor_idx": _alloc((B, N), torch.int32, dev),
           "n_spans": _alloc((B,), torch.int32, dev), "span_start": _alloc((B, N), torch.int32, dev),
           "span_len": _alloc((B, N), torch.int32, dev)}
    ws = _alloc((max(ws_bytes, 16),), torch.uint8, dev)
    _check(LIB.sekv_segment(ctypes.byref(bd), _ptr(surprisal), _ptr(n_tokens), _ptr(out["n_anchors"]),
                            _ptr(out["anchor_idx"]), _ptr(out["n_spans"]), _ptr(out["span_start"]),
                            _ptr(out["span_len"]), _ptr(ws), ws_bytes, _stream(stream)))
    out["_ws"] = ws
    return out


def build_layout(bd: BuildDims, max_spans: int, n_spans, span_len):
    """sekv_build_layout on host arrays: (block_off int64, block_rank int32, arena bytes)."""
    ns = np.ascontiguousarray(n_spans, dtype=np.int32)
    sl = np.ascontiguousarray(span_len, dtype=np.int32)
    shape = (bd.batch, bd.n_kv_heads, max(int(max_spans), 1))
    off = np.zeros(shape, dtype=np.int64)
    rank = np.zeros(shape, dtype=np.int32)
    nbytes = LIB.sekv_build_layout(ctypes.byref(bd), int(max_spans), ns.ctypes.data, sl.ctypes.data,
                                   off.ctypes.data, rank.ctypes.data)
    if nbytes < 0:
        raise SekvError(SEKV_ERR_INVALID_ARG, LIB.sekv_last_error().decode())
    return off, rank, int(nbytes)


def build_cache(bd: BuildDims, keys, values, surprisal, n_tokens, seg: dict, omega, max_anchors: int,
                max_spans: int, block_off, factors_bytes: int, ws: Workspace, out: dict | None = None,
                stream=None) -> dict:
    """sekv_build_cache: returns the device tensors of the stored cache (anchor_k/v, sum_k/v,
    span_len, span_logsize, factors); `out` may hold them preallocated."""
    dev = keys.device
    B, Hkv, d = bd.batch, bd.n_kv_heads, bd.head_dim
    st = keys.dtype
    if out is None:
        out = {"anchor_k": torch.zeros((B, Hkv, max_anchors, d), dtype=st, device=dev),
               "anchor_v": torch.zeros((B, Hkv, max_anchors, d), dtype=st, device=dev),
               "sum_k": torch.zeros((B, Hkv, max_spans, d), dtype=st, device=dev),
               "sum_v": torch.zeros((B, Hkv, max_spans, d), dtype=st, device=dev),
               "span_len": torch.ones((B, max_spans), dtype=torch.int32, device=dev),
               "span_logsize": torch.zeros((B, max_spans), dtype=torch.float64, device=dev),
               "factors": torch.zeros((int(factors_bytes),), dtype=torch.uint8, device=dev)}
    _check(LIB.sekv_build_cache(
        ctypes.byref(bd), _ptr(keys), _ptr(values), _ptr(surprisal), _ptr(n_tokens),
        _ptr(seg["n_anchors"]), _ptr(seg["anchor_idx"]), _ptr(seg["n_spans"]), _ptr(seg["span_start"]),
        _ptr(seg["span_len"]), _ptr(omega), int(max_anchors), int(max_spans), _ptr(out["anchor_k"]),
        _ptr(out["anchor_v"]), _ptr(out["sum_k"]), _ptr(out["sum_v"]), _ptr(out["span_len"]),
        _ptr(out["span_logsize"]), _ptr(out["factors"]), int(out["factors"].numel()), _ptr(block_off),
        ws.ptr, ws.nbytes, _stream(stream)))
    return out


def build_layer(bd: BuildDims, keys, values, surprisal, n_tokens, omega, ws: Workspace, stream=None):
    """Segment, lay out and build one layer's cache.  The layout needs the span tables on
    the host, so the stream is synchronised once between segmentation and the build.
    Returns (cache tensors, segmentation tensors, host layout dict)."""
    seg = segment(bd, surprisal, n_tokens, stream)
    (stream if stream is not None else torch.cuda.current_stream()).synchronize()
    ns = seg["n_spans"].cpu().numpy()
    na = seg["n_anchors"].cpu().numpy()
    span_len = seg["span_len"].cpu().numpy()
    max_spans = max(int(ns.max(initial=0)), 1)
    max_anchors = max(int(na.max(initial=0)), 1)
    off, rank, nbytes = build_layout(bd, max_spans, ns, span_len)
    dev = keys.device
    block_off = torch.from_numpy(off).to(dev)
    cache = build_cache(bd, keys, values, surprisal, n_tokens, seg, omega, max_anchors, max_spans,
                        block_off, nbytes, ws, stream=stream)
    cache["block_off"] = block_off
    cache["block_rank"] = torch.from_numpy(rank).to(dev)
    cache["n_anchors"] = seg["n_anchors"]
    cache["n_spans"] = seg["n_spans"]
    layout = {"n_spans": ns, "n_anchors": na, "max_spans": max_spans, "max_anchors": max_anchors,
              "block_off": off, "block_rank": rank, "factors_bytes": nbytes,
              "max_span_len": max([int(span_len[b, :ns[b]].max(initial=1)) for b in range(bd.batch)],
                                  default=1)}
    return cache, seg, layout
