"""Thin ctypes binding of libppas.so (C ABI in include/ppas.h).

Argument marshalling only: every step of the computation runs in the library's
HIP kernels. Device buffers are torch tensors (data pointers are passed through),
descriptors and block-table host copies are NumPy int32 arrays. Importing this
module fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes
import math
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libppas.so")
if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_15171_amd.build`")

# PyTorch wheels carry their own HIP runtime. Import torch first so that the
# library's libamdhip64.so.7 dependency binds to the runtime torch already
# loaded (same SONAME): device pointers and streams are then shared by one HIP
# runtime. Without torch, the system ROCm runtime is used.
try:
    import torch  # noqa: F401
except ImportError:
    torch = None
_lib = ctypes.CDLL(LIB_PATH)


def _hip_runtimes() -> set:
    paths = set()
    with open("/proc/self/maps") as f:
        for line in f:
            path = line.split()[-1] if len(line.split()) >= 6 else ""
            if os.path.basename(path).startswith("libamdhip64.so"):
                paths.add(os.path.realpath(path))
    return paths


if len(_hip_runtimes()) > 1:
    raise ImportError(f"two HIP runtimes are loaded in this process ({sorted(_hip_runtimes())}); "
                      "import torch before loading libppas.so")

PPAS_OK, PPAS_EINVAL, PPAS_ERANGE, PPAS_ENOSPACE, PPAS_EHIP, PPAS_EUNSUPPORTED = 0, -1, -2, -3, -4, -5


class Shape(ctypes.Structure):
    _fields_ = [("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("num_pages", ctypes.c_int32), ("scale", ctypes.c_float)]


class PPASError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} ({status})")


class PlanOpts(ctypes.Structure):
    """Planning choices of one call (0 = automatic): see ppas_plan_opts in include/ppas.h."""
    _fields_ = [("prefill_split", ctypes.c_int32), ("decode_split", ctypes.c_int32),
                ("tile_positions", ctypes.c_int32), ("num_cus", ctypes.c_int32)]


class Events(ctypes.Structure):
    """hipEvent_t handles a call's launches record (None = not recorded): see ppas_events."""
    _fields_ = [("start", ctypes.c_void_p), ("stop", ctypes.c_void_p),
                ("merge_start", ctypes.c_void_p), ("merge_stop", ctypes.c_void_p)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("n_items", ctypes.c_int32), ("n_merge", ctypes.c_int32), ("tile_positions", ctypes.c_int32),
                ("n_append", ctypes.c_int32), ("workspace_bytes", ctypes.c_uint64)]


_vp, _i32, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
_P = ctypes.POINTER(Shape)
_O = ctypes.POINTER(PlanOpts)
_E = ctypes.POINTER(Events)
_lib.ppas_status_string.restype = ctypes.c_char_p
_lib.ppas_status_string.argtypes = [ctypes.c_int]
_lib.ppas_validate_step.restype = ctypes.c_int
_lib.ppas_validate_step.argtypes = [_P, _vp, _i32, _vp, _i32]
_lib.ppas_kv_append.restype = ctypes.c_int
_lib.ppas_kv_append.argtypes = [_P, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _i32, _vp, _vp]
_lib.ppas_rope_kv_append.restype = ctypes.c_int
_lib.ppas_rope_kv_append.argtypes = [_P, ctypes.c_float, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _i32, _vp, _vp]
_lib.ppas_attn_workspace_bytes.restype = _sz
_lib.ppas_attn_workspace_bytes.argtypes = [_P, _vp, _i32]
_lib.ppas_attn_step.restype = ctypes.c_int
_lib.ppas_attn_step.argtypes = [_P, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _i32, _vp, _vp, _sz, _vp]
_lib.ppas_attn_step_noalloc.restype = ctypes.c_int
_lib.ppas_attn_step_noalloc.argtypes = [_P, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _i32, _vp, _vp]
_lib.ppas_gateup_proj.restype = ctypes.c_int
_lib.ppas_gateup_proj.argtypes = [_vp, _vp, _vp, _i32, _i32, _i32, _vp, _sz, _E, _vp]
_lib.ppas_gateup_workspace_bytes.restype = _sz
_lib.ppas_gateup_workspace_bytes.argtypes = [_i32, _i32, _i32]
_lib.ppas_gateup_act.restype = ctypes.c_int
_lib.ppas_gateup_act.argtypes = [_vp, _vp, _vp, _i32, _i32, _i32, _vp, _sz, _E, _vp]
_lib.ppas_gateup_act_workspace_bytes.restype = _sz
_lib.ppas_gateup_act_workspace_bytes.argtypes = [_i32, _i32, _i32]
_lib.ppas_stream_read.restype = ctypes.c_int
_lib.ppas_stream_read.argtypes = [_vp, _sz, _vp, _E, _vp]
_lib.ppas_plan_items.restype = _i32
_lib.ppas_plan_items.argtypes = [_P, _vp, _i32, _O, _vp, _i32]
_lib.ppas_step_plan_create.restype = ctypes.c_int
_lib.ppas_step_plan_create.argtypes = [_P, _vp, _i32, _vp, _i32, _O, ctypes.POINTER(ctypes.c_void_p)]
_lib.ppas_step_plan_info.restype = ctypes.c_int
_lib.ppas_step_plan_info.argtypes = [_vp, ctypes.POINTER(PlanInfo)]
_lib.ppas_step_plan_destroy.restype = None
_lib.ppas_step_plan_destroy.argtypes = [_vp]
_lib.ppas_kv_append_planned.restype = ctypes.c_int
_lib.ppas_kv_append_planned.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _E, _vp]
_lib.ppas_rope_kv_append_planned.restype = ctypes.c_int
_lib.ppas_rope_kv_append_planned.argtypes = [_vp, ctypes.c_float, _vp, _vp, _vp, _vp, _vp, _vp, _E, _vp]
_lib.ppas_attn_step_planned.restype = ctypes.c_int
_lib.ppas_attn_step_planned.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _E, _vp]


def status_string(status: int) -> str:
    return _lib.ppas_status_string(int(status)).decode()


def make_shape(n_q_heads: int = 16, n_kv_heads: int = 2, num_pages: int = 1, scale: float | None = None,
               head_dim: int = 128, page_size: int = 16) -> Shape:
    if scale is None:
        scale = 1.0 / math.sqrt(head_dim)
    return Shape(n_q_heads, n_kv_heads, head_dim, page_size, num_pages, scale)


def _desc(desc) -> np.ndarray:
    d = np.ascontiguousarray(desc, dtype=np.int32)
    if d.ndim != 2 or d.shape[1] != 3:
        raise ValueError("descriptors must be int32 [S, 3] (query_start, n_query, cached_len)")
    return d


def _host_ptr(a):
    return None if a is None else a.ctypes.data


def _bt_host(bt_host, bt_dev=None):
    """The host copy of the block table as int32; when the device table is given, the
    two must have the same shape (the library reads the host copy with the device
    table's row stride)."""
    if bt_host is None:
        return None
    bt = np.ascontiguousarray(bt_host, dtype=np.int32)
    if bt.ndim != 2:
        raise ValueError("the host block table must be int32 [n_seqs, stride]")
    if bt_dev is not None and tuple(bt.shape) != tuple(bt_dev.shape):
        raise ValueError(f"host block table {tuple(bt.shape)} and device block table {tuple(bt_dev.shape)} differ")
    return bt


def _dev(t, name):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _rows(d) -> int:
    return int(d[:, 1].astype(np.int64).clip(min=0).sum()) if len(d) else 0


def _need(t, name, nbytes: int, elem: int | None = 2):
    """Refuse a device buffer smaller than the call will touch (or of the wrong
    element size), so a bad argument raises here instead of reaching a kernel."""
    if t is None:
        return
    if elem is not None and t.element_size() != elem:
        raise ValueError(f"{name} must have {elem}-byte elements (bf16 bit patterns), got {t.dtype}")
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{name} holds {have} bytes; this call needs {nbytes}")


def _check_buffers(shape: Shape, d, q=None, out=None, k_new=None, v_new=None, k_pages=None, v_pages=None,
                   bt_dev=None):
    if len(d) == 0:
        return                      # an empty step touches no buffer
    T, D = _rows(d), shape.head_dim
    _need(q, "q", T * shape.n_q_heads * D * 2)
    _need(out, "out", T * shape.n_q_heads * D * 2)
    _need(k_new, "k_new", T * shape.n_kv_heads * D * 2)
    _need(v_new, "v_new", T * shape.n_kv_heads * D * 2)
    pool = int(shape.num_pages) * shape.n_kv_heads * shape.page_size * D * 2
    _need(k_pages, "k_pages", pool)
    _need(v_pages, "v_pages", pool)
    if bt_dev is not None:
        if bt_dev.element_size() != 4 or bt_dev.dim() != 2:
            raise ValueError("block_table must be an int32 [n_seqs, stride] device tensor")
        if bt_dev.shape[0] < len(d):
            raise ValueError(f"block_table has {bt_dev.shape[0]} rows for {len(d)} requests")


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def _check(st: int, what: str):
    if st != PPAS_OK:
        raise PPASError(st, what)


def validate_step(shape: Shape, desc, bt_host=None, bt_stride: int | None = None) -> int:
    d = _desc(desc)
    bt = _bt_host(bt_host)
    stride = bt_stride if bt_stride is not None else (bt.shape[1] if bt is not None else 1)
    return _lib.ppas_validate_step(ctypes.byref(shape), _host_ptr(d), len(d), _host_ptr(bt), stride)


def kv_append(shape: Shape, k_pages, v_pages, k_new, v_new, desc, bt_dev, bt_host=None, stream=None) -> None:
    d = _desc(desc)
    bt = _bt_host(bt_host, bt_dev)
    _check_buffers(shape, d, k_new=k_new, v_new=v_new, k_pages=k_pages, v_pages=v_pages, bt_dev=bt_dev)
    st = _lib.ppas_kv_append(ctypes.byref(shape), _dev(k_pages, "k_pages"), _dev(v_pages, "v_pages"),
                             _dev(k_new, "k_new"), _dev(v_new, "v_new"), _host_ptr(d), len(d),
                             _dev(bt_dev, "block_table"), bt_dev.shape[1], _host_ptr(bt), _stream(stream))
    _check(st, "ppas_kv_append")


def rope_kv_append(shape: Shape, theta: float, q, k_pages, v_pages, k_new, v_new, desc, bt_dev, bt_host=None,
                   stream=None) -> None:
    """Rotate q in place and k_new into the pages at each row's position; copy v_new."""
    d = _desc(desc)
    bt = _bt_host(bt_host, bt_dev)
    _check_buffers(shape, d, q=q, k_new=k_new, v_new=v_new, k_pages=k_pages, v_pages=v_pages, bt_dev=bt_dev)
    st = _lib.ppas_rope_kv_append(ctypes.byref(shape), float(theta), _dev(q, "q"), _dev(k_pages, "k_pages"),
                                  _dev(v_pages, "v_pages"), _dev(k_new, "k_new"), _dev(v_new, "v_new"),
                                  _host_ptr(d), len(d), _dev(bt_dev, "block_table"), bt_dev.shape[1],
                                  _host_ptr(bt), _stream(stream))
    _check(st, "ppas_rope_kv_append")


def attn_workspace_bytes(shape: Shape, desc) -> int:
    d = _desc(desc)
    return int(_lib.ppas_attn_workspace_bytes(ctypes.byref(shape), _host_ptr(d), len(d)))


def attn_step(shape: Shape, out, q, k_pages, v_pages, desc, bt_dev, workspace, bt_host=None, stream=None) -> None:
    d = _desc(desc)
    bt = _bt_host(bt_host, bt_dev)
    _check_buffers(shape, d, q=q, out=out, k_pages=k_pages, v_pages=v_pages, bt_dev=bt_dev)
    st = _lib.ppas_attn_step(ctypes.byref(shape), _dev(out, "out"), _dev(q, "q"), _dev(k_pages, "k_pages"),
                             _dev(v_pages, "v_pages"), _host_ptr(d), len(d), _dev(bt_dev, "block_table"),
                             bt_dev.shape[1], _host_ptr(bt), _dev(workspace, "workspace"),
                             workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "ppas_attn_step")


def attn_step_noalloc(shape: Shape, out, q, k_pages, v_pages, desc, bt_dev, bt_host=None, stream=None) -> None:
    """ppas_attn_step without a workspace: the library's fixed device array holds the work list
    and the split partials (PPAS_ENOSPACE when the step does not fit it)."""
    d = _desc(desc)
    bt = _bt_host(bt_host, bt_dev)
    _check_buffers(shape, d, q=q, out=out, k_pages=k_pages, v_pages=v_pages, bt_dev=bt_dev)
    st = _lib.ppas_attn_step_noalloc(ctypes.byref(shape), _dev(out, "out"), _dev(q, "q"), _dev(k_pages, "k_pages"),
                                     _dev(v_pages, "v_pages"), _host_ptr(d), len(d), _dev(bt_dev, "block_table"),
                                     bt_dev.shape[1], _host_ptr(bt), _stream(stream))
    _check(st, "ppas_attn_step_noalloc")


def gateup_workspace_bytes(n_tokens: int, hidden: int, n_out: int) -> int:
    return int(_lib.ppas_gateup_workspace_bytes(int(n_tokens), int(hidden), int(n_out)))


def gateup_proj(x, w, y, workspace=None, events: Events | None = None, stream=None) -> None:
    """y = x w^T: the fused gate-up projection (x [T, H], w [N, H], y [T, N], bf16 device tensors).
    workspace: a device buffer for split reductions (see gateup_workspace_bytes), or None."""
    for t, name in ((x, "x"), (w, "w"), (y, "y")):
        if t.dim() != 2 or t.element_size() != 2:
            raise ValueError(f"{name} must be a 2-D bf16 tensor")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    T, H = x.shape
    N = w.shape[0]
    if w.shape[1] != H or tuple(y.shape) != (T, N):
        raise ValueError(f"shapes x {tuple(x.shape)}, w {tuple(w.shape)}, y {tuple(y.shape)} do not match")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = _lib.ppas_gateup_proj(_dev(x, "x"), _dev(w, "w"), _dev(y, "y"), T, H, N, _dev(workspace, "workspace"),
                               ws_bytes, None if events is None else ctypes.byref(events), _stream(stream))
    _check(st, "ppas_gateup_proj")


def gateup_act_workspace_bytes(n_tokens: int, hidden: int, n_inter: int) -> int:
    return int(_lib.ppas_gateup_act_workspace_bytes(int(n_tokens), int(hidden), int(n_inter)))


def gateup_act(x, w, y, workspace=None, events: Events | None = None, stream=None) -> None:
    """y = silu(x w_gate^T) * (x w_up^T): the gate-up projection with the gated activation
    (x [T, H], w [2I, H] with the gate rows over the up rows, y [T, I], bf16 device tensors).
    workspace: a device buffer for split reductions (see gateup_act_workspace_bytes), or None."""
    for t, name in ((x, "x"), (w, "w"), (y, "y")):
        if t.dim() != 2 or t.element_size() != 2:
            raise ValueError(f"{name} must be a 2-D bf16 tensor")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    T, H = x.shape
    N = w.shape[0]
    if N % 2 or w.shape[1] != H or tuple(y.shape) != (T, N // 2):
        raise ValueError(f"shapes x {tuple(x.shape)}, w {tuple(w.shape)}, y {tuple(y.shape)} do not match")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = _lib.ppas_gateup_act(_dev(x, "x"), _dev(w, "w"), _dev(y, "y"), T, H, N // 2, _dev(workspace, "workspace"),
                              ws_bytes, None if events is None else ctypes.byref(events), _stream(stream))
    _check(st, "ppas_gateup_act")


def stream_read(buf, sink, events: Events | None = None, stream=None) -> None:
    """A plain streaming read of the whole of `buf` (a contiguous device tensor, a multiple of
    16 bytes): the XOR of its 16-byte words, as four 32-bit lanes, is XORed into `sink` (a
    device tensor of 16 bytes). The measured HBM read ceiling of the device."""
    nbytes = buf.numel() * buf.element_size()
    if sink.numel() * sink.element_size() != 16:
        raise ValueError("sink must hold 16 bytes")
    st = _lib.ppas_stream_read(_dev(buf, "buf"), nbytes, _dev(sink, "sink"),
                               None if events is None else ctypes.byref(events), _stream(stream))
    _check(st, "ppas_stream_read")


def plan_opts(prefill_split: int = 0, decode_split: int = 0, tile_positions: int = 0, num_cus: int = 0) -> PlanOpts:
    return PlanOpts(int(prefill_split), int(decode_split), int(tile_positions), int(num_cus))


def events(start=None, stop=None, merge_start=None, merge_stop=None) -> Events:
    return Events(start, stop, merge_start, merge_stop)


def _opts_ptr(opts):
    return None if opts is None else ctypes.byref(opts)


def plan_items(shape: Shape, desc, num_cus: int = 256, opts: PlanOpts | None = None) -> np.ndarray:
    """The planned work list as int32 [n, 8]: kind, seq, kv_head, row0, pos0, npos, key_lo, key_hi."""
    d = _desc(desc)
    o = PlanOpts() if opts is None else PlanOpts(opts.prefill_split, opts.decode_split, opts.tile_positions,
                                                 opts.num_cus)
    if o.num_cus == 0:
        o.num_cus = int(num_cus)
    n = _lib.ppas_plan_items(ctypes.byref(shape), _host_ptr(d), len(d), ctypes.byref(o), None, 0)
    if n < 0:
        raise PPASError(n, "ppas_plan_items")
    out = np.zeros((max(n, 1), 8), dtype=np.int32)
    _lib.ppas_plan_items(ctypes.byref(shape), _host_ptr(d), len(d), ctypes.byref(o), out.ctypes.data, n)
    return out[:n]


class StepPlan:
    """A step's validated descriptors, attention work list and page-write list, made once
    (ppas_step_plan_create) and used by any number of planned calls, e.g. one per layer."""

    def __init__(self, shape: Shape, desc, bt_host=None, bt_stride: int | None = None, opts: PlanOpts | None = None):
        self.shape = Shape(shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.page_size, shape.num_pages,
                           shape.scale)
        self.desc = _desc(desc)
        bt = _bt_host(bt_host)
        self.bt_stride = int(bt_stride if bt_stride is not None else (bt.shape[1] if bt is not None else 1))
        if bt is not None and bt.shape[1] != self.bt_stride:
            raise ValueError("bt_stride differs from the host block table's row length")
        h = ctypes.c_void_p()
        st = _lib.ppas_step_plan_create(ctypes.byref(self.shape), _host_ptr(self.desc), len(self.desc),
                                        _host_ptr(bt), self.bt_stride, _opts_ptr(opts), ctypes.byref(h))
        _check(st, "ppas_step_plan_create")
        self._h = h.value
        self.info = PlanInfo()
        _check(_lib.ppas_step_plan_info(self._h, ctypes.byref(self.info)), "ppas_step_plan_info")

    @property
    def workspace_bytes(self) -> int:
        return int(self.info.workspace_bytes)

    def _bt(self, bt_dev):
        if bt_dev is None:
            raise ValueError("block_table is required")
        if bt_dev.dim() != 2 or bt_dev.shape[1] != self.bt_stride:
            raise ValueError(f"block_table must have rows of {self.bt_stride} entries, got {tuple(bt_dev.shape)}")
        return bt_dev

    def kv_append(self, k_pages, v_pages, k_new, v_new, bt_dev, events: Events | None = None, stream=None) -> None:
        _check_buffers(self.shape, self.desc, k_new=k_new, v_new=v_new, k_pages=k_pages, v_pages=v_pages,
                       bt_dev=self._bt(bt_dev))
        st = _lib.ppas_kv_append_planned(self._h, _dev(k_pages, "k_pages"), _dev(v_pages, "v_pages"),
                                         _dev(k_new, "k_new"), _dev(v_new, "v_new"), _dev(bt_dev, "block_table"),
                                         None if events is None else ctypes.byref(events), _stream(stream))
        _check(st, "ppas_kv_append_planned")

    def rope_kv_append(self, theta: float, q, k_pages, v_pages, k_new, v_new, bt_dev, events: Events | None = None,
                       stream=None) -> None:
        _check_buffers(self.shape, self.desc, q=q, k_new=k_new, v_new=v_new, k_pages=k_pages, v_pages=v_pages,
                       bt_dev=self._bt(bt_dev))
        st = _lib.ppas_rope_kv_append_planned(self._h, float(theta), _dev(q, "q"), _dev(k_pages, "k_pages"),
                                              _dev(v_pages, "v_pages"), _dev(k_new, "k_new"), _dev(v_new, "v_new"),
                                              _dev(bt_dev, "block_table"),
                                              None if events is None else ctypes.byref(events), _stream(stream))
        _check(st, "ppas_rope_kv_append_planned")

    def attn_step(self, out, q, k_pages, v_pages, bt_dev, workspace, events: Events | None = None,
                  stream=None) -> None:
        _check_buffers(self.shape, self.desc, q=q, out=out, k_pages=k_pages, v_pages=v_pages,
                       bt_dev=self._bt(bt_dev))
        st = _lib.ppas_attn_step_planned(self._h, _dev(out, "out"), _dev(q, "q"), _dev(k_pages, "k_pages"),
                                         _dev(v_pages, "v_pages"), _dev(bt_dev, "block_table"),
                                         _dev(workspace, "workspace"), workspace.numel() * workspace.element_size(),
                                         None if events is None else ctypes.byref(events), _stream(stream))
        _check(st, "ppas_attn_step_planned")

    def close(self) -> None:
        h, self._h = getattr(self, "_h", None), None
        if h and _lib is not None:
            _lib.ppas_step_plan_destroy(h)

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        self.close()
