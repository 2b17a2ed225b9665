"""Python binding of liboc, the MI355X octree-CNN hot path (O-CNN, arXiv 1712.01537).

Argument marshalling only: every step runs in the HIP kernels of ``liboc.so``
(built from ``csrc/`` by ``build.py``).  torch provides device memory (the
octree's arrays are carved from torch tensors through the allocator callback
of ``oc_build``) and the stream every call is enqueued on (torch's current
stream).  The functions carry the C ABI's names; see ``include/oc.h`` for the
contract of each.

If ``liboc.so`` is missing or cannot be loaded, every entry point raises
:class:`OcError`; there is no other implementation to fall back to.
"""
from __future__ import annotations

import ctypes as C
import os

import torch

__all__ = [
    "OcError",
    "Octree",
    "lib_path",
    "load",
    "oc_build",
    "oc_build_async",
    "BuildJob",
    "oc_conv_fwd",
    "oc_conv_fwd_noalloc",
    "oc_conv_pool_fwd",
    "oc_conv_kernel",
    "oc_profile_next",
    "CallProfile",
    "oc_conv_bwd",
    "oc_sum_partials",
    "oc_round_bf16",
    "oc_conv_bwd_pool",
    "oc_deconv_fwd",
    "oc_deconv_bwd",
    "oc_pool_fwd",
    "oc_pool_bwd",
    "oc_unpool_fwd",
    "oc_unpool_bwd",
    "oc_gpool_fwd",
    "oc_gpool_bwd",
    "OC_FUSE_RELU",
    "OC_DEFER_DW",
    "OC_POOL_MAX",
    "OC_POOL_AVG",
    "oc_bn_fwd",
    "oc_bn_pool_fwd",
    "oc_bn_bwd",
    "oc_fc_fwd",
    "oc_fc_bwd",
    "oc_dropout",
    "oc_softmax_ce",
    "oc_sgd",
    "EXPORTS",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
OC_FUSE_RELU = 1
OC_DEFER_DW = 2
OC_POOL_MAX, OC_POOL_AVG = 0, 1
OC_F32, OC_BF16 = 0, 1
STATUS = {0: "OC_OK", 1: "OC_ERR_ARG", 2: "OC_ERR_RANGE", 3: "OC_ERR_NOMEM", 4: "OC_ERR_DEVICE",
          5: "OC_ERR_UNSUPPORTED"}

# Every symbol include/oc.h declares.
EXPORTS = (
    "oc_build", "oc_build_async", "oc_build_finish", "oc_build_cancel",
    "oc_octree_level", "oc_octree_info", "oc_octree_signal", "oc_octree_free",
    "oc_conv_fwd", "oc_conv_kernel", "oc_conv_fwd_workspace", "oc_conv_bwd_workspace", "oc_conv_bwd", "oc_pool_fwd", "oc_pool_bwd",
    "oc_unpool_fwd", "oc_unpool_bwd", "oc_status_str", "oc_last_error", "oc_profile_next",
    "oc_deconv_fwd", "oc_deconv_fwd_workspace", "oc_deconv_bwd", "oc_deconv_bwd_workspace",
    "oc_gpool_fwd", "oc_gpool_bwd", "oc_profile_calls", "oc_conv_fwd_noalloc",
    "oc_bn_workspace", "oc_bn_fwd", "oc_bn_bwd", "oc_fc_fwd", "oc_fc_bwd", "oc_dropout",
    "oc_softmax_ce_workspace", "oc_softmax_ce", "oc_sgd", "oc_conv_pool_fwd",
    "oc_conv_pool_fwd_workspace", "oc_bn_pool_fwd", "oc_conv_bwd_pool_workspace",
    "oc_conv_bwd_pool", "oc_conv_dw_partials", "oc_sum_partials", "oc_round_bf16",
)


class OcError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = code


def lib_path() -> str:
    return os.path.join(_HERE, "liboc.so")


class _Level(C.Structure):
    _fields_ = [
        ("depth", C.c_int32),
        ("num_octants", C.c_int64),
        ("num_nonempty", C.c_int64),
        ("keys", C.c_void_p),
        ("labels", C.c_void_p),
        ("rows_of_label", C.c_void_p),
        ("nbr", C.c_void_p),
    ]


_ALLOC_FN = C.CFUNCTYPE(C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p)
_FREE_FN = C.CFUNCTYPE(None, C.c_void_p, C.c_void_p, C.c_void_p)


class _Allocator(C.Structure):
    _fields_ = [("alloc", _ALLOC_FN), ("free", _FREE_FN), ("ctx", C.c_void_p)]


# Live device allocations made for the library: data_ptr -> backing tensor,
# and the stream each was allocated on.
_live: dict[int, torch.Tensor] = {}
_live_stream: dict[int, int] = {}


def _torch_alloc(ctx, nbytes, stream):
    # the wrappers make `stream` torch's current stream during the call
    try:
        t = torch.empty(int(nbytes), dtype=torch.uint8, device="cuda")
    except Exception:  # out of memory -> NULL -> OC_ERR_NOMEM
        return None
    _live[t.data_ptr()] = t
    _live_stream[t.data_ptr()] = int(stream or 0)
    return t.data_ptr()


def _torch_free(ctx, ptr, stream):
    # released in stream order on `stream`: when that is not the allocation
    # stream, torch keeps the block until the work queued there is done
    t = _live.pop(int(ptr), None)
    s0 = _live_stream.pop(int(ptr), 0)
    if t is not None and int(stream or 0) != s0:
        t.record_stream(torch.cuda.ExternalStream(int(stream or 0)))


_alloc_cb = _ALLOC_FN(_torch_alloc)
_free_cb = _FREE_FN(_torch_free)
_allocator = _Allocator(_alloc_cb, _free_cb, None)

_lib = None


def load():
    """Load liboc.so (built in-tree by build.py); raise OcError if it is absent."""
    global _lib
    if _lib is not None:
        return _lib
    path = lib_path()
    if not os.path.exists(path):
        raise OcError(-1, f"{path} is missing: run paper_1712_01537_amd/build.py (hipcc, gfx950)")
    L = C.CDLL(path)
    p, i32, i64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
    sigs = {
        "oc_build": ([p, p, p, i32, i32, i32, p, p, C.POINTER(p)], C.c_int),
        "oc_build_async": ([p, p, p, i32, i32, i32, p, p, C.POINTER(p)], C.c_int),
        "oc_build_finish": ([p, p, C.POINTER(p)], C.c_int),
        "oc_build_cancel": ([p], None),
        "oc_octree_level": ([p, i32, C.POINTER(_Level)], C.c_int),
        "oc_octree_info": ([p, p, p, p], C.c_int),
        "oc_octree_signal": ([p], p),
        "oc_octree_free": ([p], None),
        "oc_conv_fwd": ([p, i32, i32, i32, C.c_int, p, i32, p, i32, p, p, sz, i32, p], C.c_int),
        "oc_conv_fwd_workspace": ([p, i32, i32, i32, C.c_int, i32, i32], sz),
        "oc_conv_pool_fwd_workspace": ([p, i32, i32, C.c_int, i32, i32], sz),
        "oc_conv_pool_fwd": ([p, i32, i32, C.c_int, p, i32, p, i32, p, p, p, sz, i32, p],
                             C.c_int),
        "oc_conv_fwd_noalloc": ([p, i32, i32, i32, C.c_int, p, i32, p, i32, p, i32, p],
                                C.c_int),
        "oc_conv_kernel": ([p, i32, i32, i32, C.c_int, i32, i32, i32], C.c_char_p),
        "oc_conv_bwd_workspace": ([p, i32, i32, i32, C.c_int, i32, i32], sz),
        "oc_conv_bwd": ([p, i32, i32, i32, C.c_int, p, i32, p, i32, p, p, p, p, p, sz, i32, p],
                        C.c_int),
        "oc_conv_bwd_pool_workspace": ([p, i32, i32, i32, i32], sz),
        "oc_conv_dw_partials": ([p, i32, i32, i32, C.c_int, i32, i32, p, p, p], C.c_int),
        "oc_sum_partials": ([i32, p, p, p, p, p], C.c_int),
        "oc_round_bf16": ([i64, p, p, p], C.c_int),
        "oc_conv_bwd_pool": ([p, i32, i32, p, i32, i32, p, p, p, p, p, p, p, sz, i32, p],
                             C.c_int),
        "oc_deconv_fwd": ([p, i32, i32, i32, C.c_int, p, i32, p, i32, p, p, sz, i32, p],
                          C.c_int),
        "oc_deconv_fwd_workspace": ([p, i32, i32, i32, C.c_int, i32, i32], sz),
        "oc_deconv_bwd_workspace": ([p, i32, i32, i32, C.c_int, i32, i32], sz),
        "oc_deconv_bwd": ([p, i32, i32, i32, C.c_int, p, i32, p, i32, p, p, p, p, sz, i32, p],
                          C.c_int),
        "oc_gpool_fwd": ([p, i32, i32, i32, i32, p, i32, p, p, p], C.c_int),
        "oc_gpool_bwd": ([p, i32, i32, i32, i32, p, p, i32, p, p], C.c_int),
        "oc_pool_fwd": ([p, i32, p, i32, p, p, p], C.c_int),
        "oc_pool_bwd": ([p, i32, p, p, i32, p, p, p], C.c_int),
        "oc_unpool_fwd": ([p, i32, p, p, i32, p, p], C.c_int),
        "oc_unpool_bwd": ([p, i32, p, p, i32, p, p], C.c_int),
        "oc_status_str": ([C.c_int], C.c_char_p),
        "oc_last_error": ([], C.c_char_p),
        "oc_profile_next": ([p, p], C.c_int),
        "oc_profile_calls": ([p, p, i32, p], C.c_int),
        "oc_bn_workspace": ([i64, i32], sz),
        "oc_bn_fwd": ([i64, i32, p, p, p, C.c_float, i32, p, p, p, p, sz, p], C.c_int),
        "oc_bn_bwd": ([i64, i32, p, p, p, p, p, p, p, p, p, sz, p], C.c_int),
        "oc_bn_pool_fwd": ([p, i32, i32, p, p, p, C.c_float, i32, p, p, p, p, p, sz, p], C.c_int),
        "oc_fc_fwd": ([i32, i32, i32, p, p, p, p, p], C.c_int),
        "oc_fc_bwd": ([i32, i32, i32, p, p, p, p, p, p, p], C.c_int),
        "oc_dropout": ([i64, p, p, C.c_float, p, p], C.c_int),
        "oc_softmax_ce_workspace": ([i32], sz),
        "oc_softmax_ce": ([i32, i32, p, p, p, p, p, sz, p], C.c_int),
        "oc_sgd": ([i64, p, p, p, C.c_float, C.c_float, C.c_float, p], C.c_int),
    }
    for name, (args, res) in sigs.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = res
    _lib = L
    return L


def _check(rc: int):
    if rc != 0:
        raise OcError(rc, load().oc_last_error().decode())


_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


def _stream():
    """The current stream of the current device, as a raw handle (torch's
    C-level accessor when present: the Python one costs several
    microseconds per call, which adds up over the dozens of calls a step
    makes)."""
    if _raw_stream is not None:
        return _raw_stream(torch._C._cuda_getDevice())
    return torch.cuda.current_stream().cuda_stream


def _dev(t: torch.Tensor, name: str, dtype=None, shape=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise OcError(1, f"{name} must be a CUDA (HIP) tensor")
    if not t.is_contiguous():
        raise OcError(1, f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise OcError(1, f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise OcError(1, f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return C.c_void_p(t.data_ptr())


class Octree:
    """A built super-octree; its arrays live in torch-owned device memory."""

    def __init__(self, handle: C.c_void_p):
        self._h = handle
        d, fd, b = C.c_int32(), C.c_int32(), C.c_int32()
        _check(load().oc_octree_info(handle, C.byref(d), C.byref(fd), C.byref(b)))
        self.depth, self.full_depth, self.batch = d.value, fd.value, b.value
        self._lv = []
        for l in range(self.depth + 1):
            lv = _Level()
            _check(load().oc_octree_level(handle, l, C.byref(lv)))
            self._lv.append(lv)

    @property
    def handle(self):
        return self._h

    def num(self, l: int) -> int:
        return int(self._lv[l].num_octants)

    def nonempty(self, l: int) -> int:
        return int(self._lv[l].num_nonempty)

    def _view(self, ptr, count, dtype, shape):
        if count == 0 or not ptr:
            return torch.empty(shape, dtype=dtype, device="cuda")
        esz = torch.empty((), dtype=dtype).element_size()
        for base, t in _live.items():
            if base <= ptr < base + t.numel():
                off = ptr - base
                return t[off:off + count * esz].view(dtype).view(shape)
        raise OcError(1, "octree array not found among live allocations")

    def keys(self, l):
        return self._view(self._lv[l].keys, self.num(l), torch.int32, (self.num(l),))

    def labels(self, l):
        return self._view(self._lv[l].labels, self.num(l), torch.int32, (self.num(l),))

    def rows(self, l):
        return self._view(self._lv[l].rows_of_label, self.nonempty(l), torch.int32, (self.nonempty(l),))

    def nbr(self, l):
        m = self.nonempty(l - 1)
        return self._view(self._lv[l].nbr, 27 * m, torch.int32, (m, 27))

    def signal(self):
        n = self.num(self.depth)
        return self._view(load().oc_octree_signal(self._h), 3 * n, torch.float32, (n, 3))

    def record_stream(self, stream) -> None:
        """Mark the octree's arrays as used on `stream` (torch's caching
        allocator then keeps them until that stream's pending work is done)."""
        for ptr in self._blocks():
            _live[ptr].record_stream(stream)

    def _blocks(self):
        ptrs = set()
        for lv in self._lv:
            for p in (lv.keys, lv.labels, lv.rows_of_label, lv.nbr):
                if p:
                    ptrs.update(b for b, t in _live.items() if b <= p < b + t.numel())
        return ptrs

    def free(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            load().oc_octree_free(self._h)
            self._h = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def oc_build(points: torch.Tensor, normals: torch.Tensor, shape_offsets, depth: int,
             full_depth: int = 2) -> Octree:
    """Build the super-octree of a batch of point clouds (dev f32 [P][3] each)."""
    L = load()
    offs = torch.as_tensor(shape_offsets, dtype=torch.int32).cpu().contiguous()
    P = int(offs[-1])
    if points.numel() != 3 * P or normals.numel() != 3 * P:
        raise OcError(1, f"points/normals must hold {P} x 3 values")
    pp = _dev(points, "points", torch.float32)
    nn = _dev(normals, "normals", torch.float32)
    h = C.c_void_p()
    _check(L.oc_build(pp, nn, C.c_void_p(offs.data_ptr()), len(offs) - 1, depth, full_depth,
                      C.byref(_allocator), _stream(), C.byref(h)))
    return Octree(h)


class BuildJob:
    """The first half of a build (oc_build_async), enqueued on the stream
    that was current; finish() completes it into an Octree."""

    def __init__(self, handle: C.c_void_p, keep):
        self._h = handle
        self._keep = keep  # points and normals stay alive until finish()

    def finish(self, stream=None) -> Octree:
        """Wait for the counts and enqueue the rest of the build on `stream`
        (a torch stream; the current one when None)."""
        if self._h is None:
            raise OcError(1, "build job already finished or cancelled")
        h, self._h = self._h, None
        st = stream if stream is not None else torch.cuda.current_stream()
        out = C.c_void_p()
        with torch.cuda.stream(st):
            _check(load().oc_build_finish(h, C.c_void_p(st.cuda_stream), C.byref(out)))
        return Octree(out)

    def cancel(self) -> None:
        if self._h is not None:
            h, self._h = self._h, None
            load().oc_build_cancel(h)

    def __del__(self):
        try:
            self.cancel()
        except Exception:
            pass


def oc_build_async(points: torch.Tensor, normals: torch.Tensor, shape_offsets, depth: int,
                   full_depth: int = 2) -> BuildJob:
    """Enqueue the first half of a build on the current stream (oc_build_async)."""
    L = load()
    offs = torch.as_tensor(shape_offsets, dtype=torch.int32).cpu().contiguous()
    P = int(offs[-1])
    if points.numel() != 3 * P or normals.numel() != 3 * P:
        raise OcError(1, f"points/normals must hold {P} x 3 values")
    pp = _dev(points, "points", torch.float32)
    nn = _dev(normals, "normals", torch.float32)
    h = C.c_void_p()
    _check(L.oc_build_async(pp, nn, C.c_void_p(offs.data_ptr()), len(offs) - 1, depth,
                            full_depth, C.byref(_allocator), _stream(), C.byref(h)))
    return BuildJob(h, (points, normals))


def _dtype_code(x: torch.Tensor):
    if x.dtype == torch.float32:
        return OC_F32
    if x.dtype == torch.bfloat16:
        return OC_BF16
    raise OcError(1, f"unsupported dtype {x.dtype}")


def _conv_dims(tree: Octree, depth: int, stride: int, x, w):
    if not 1 <= depth <= tree.depth:
        raise OcError(1, f"depth {depth} not in 1..{tree.depth}")
    K3, cin, cout = w.shape
    n_in = tree.num(depth)
    r = int(stride).bit_length() - 1  # stride 2^r
    if not 0 <= r <= depth:
        raise OcError(1, f"stride {stride} needs depth >= {r}")
    n_out = tree.num(depth - r)
    if x is not None and tuple(x.shape) != (n_in, cin):
        raise OcError(1, f"x has shape {tuple(x.shape)}, expected {(n_in, cin)}")
    return K3, cin, cout, n_in, n_out


def oc_profile_next(start, stop) -> None:
    """Bracket the next conv-pass kernel launch of this thread with two
    torch.cuda.Event objects (created with enable_timing=True and recorded at
    least once, so that they exist)."""
    _check(load().oc_profile_next(C.c_void_p(start.cuda_event) if start is not None else None,
                                  C.c_void_p(stop.cuda_event) if stop is not None else None))


class CallProfile:
    """Brackets every kernel the library launches from this thread between
    arm() and disarm() with a pair of torch.cuda events (oc_profile_calls);
    kernel_ms() is the sum of their durations once the work is done."""

    def __init__(self, cap: int = 64):
        self.cap = cap
        self.start = [torch.cuda.Event(enable_timing=True) for _ in range(cap)]
        self.stop = [torch.cuda.Event(enable_timing=True) for _ in range(cap)]
        for e in self.start + self.stop:
            e.record()  # instantiates the events
        self._a = (C.c_void_p * cap)(*[e.cuda_event for e in self.start])
        self._b = (C.c_void_p * cap)(*[e.cuda_event for e in self.stop])
        self._used = C.c_int32(0)

    def arm(self) -> None:
        _check(load().oc_profile_calls(self._a, self._b, self.cap, C.byref(self._used)))

    def disarm(self) -> None:
        _check(load().oc_profile_calls(None, None, 0, None))

    @property
    def used(self) -> int:
        return min(int(self._used.value), self.cap)

    def kernel_ms(self) -> float:
        return sum(self.start[i].elapsed_time(self.stop[i]) for i in range(self.used))


def oc_conv_kernel(tree: Octree, depth: int, ksize: int, stride: int, cin: int, cout: int,
                   pass_: int, dtype=torch.float32) -> str:
    """Name of the kernel doing pass 0 (fwd), 1 (input grad) or 2 (weight grad)."""
    dt = OC_F32 if dtype == torch.float32 else OC_BF16
    name = load().oc_conv_kernel(tree.handle, depth, ksize, stride, dt, cin, cout, pass_)
    if not name:
        raise OcError(1, load().oc_last_error().decode())
    return name.decode()


def oc_conv_fwd(tree: Octree, depth: int, ksize: int, stride: int, x: torch.Tensor,
                w: torch.Tensor, relu: bool = False, y: torch.Tensor | None = None) -> torch.Tensor:
    K3, cin, cout, n_in, n_out = _conv_dims(tree, depth, stride, x, w)
    if K3 != ksize ** 3:
        raise OcError(1, f"w has {K3} taps, expected {ksize ** 3}")
    dt = _dtype_code(x)
    if w.dtype != x.dtype:
        raise OcError(1, "x and w must share a dtype")
    if y is None:
        y = torch.empty((n_out, cout), dtype=torch.float32, device=x.device)
    L = load()
    ws_bytes = int(L.oc_conv_fwd_workspace(tree.handle, depth, ksize, stride, dt, cin, cout))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=x.device) if ws_bytes else None
    _check(L.oc_conv_fwd(tree.handle, depth, ksize, stride, dt, _dev(x, "x"), cin,
                         _dev(w, "w"), cout, _dev(y, "y", torch.float32, (n_out, cout)),
                         _dev(ws, "ws") if ws is not None else None, ws_bytes,
                         OC_FUSE_RELU if relu else 0, _stream()))
    return y


def oc_conv_pool_fwd(tree: Octree, depth: int, ksize: int, x: torch.Tensor, w: torch.Tensor,
                     relu: bool = True):
    """Stride-1 convolution at depth, optional ReLU and the 2x2x2 max-pool to
    depth - 1 in one call: (pooled [N_{l-1}][cout], switches [M_{l-1}][cout])."""
    K3, cin, cout, n_in, n_out = _conv_dims(tree, depth, 1, x, w)
    if K3 != ksize ** 3:
        raise OcError(1, f"w has {K3} taps, expected {ksize ** 3}")
    dt = _dtype_code(x)
    if w.dtype != x.dtype:
        raise OcError(1, "x and w must share a dtype")
    n_p, m = tree.num(depth - 1), tree.nonempty(depth - 1)
    y = torch.empty((n_p, cout), dtype=torch.float32, device=x.device)
    sw = torch.empty((m, cout), dtype=torch.uint8, device=x.device)
    L = load()
    ws_bytes = int(L.oc_conv_pool_fwd_workspace(tree.handle, depth, ksize, dt, cin, cout))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=x.device) if ws_bytes else None
    _check(L.oc_conv_pool_fwd(tree.handle, depth, ksize, dt, _dev(x, "x"), cin, _dev(w, "w"),
                              cout, _dev(y, "y"), _dev(sw, "sw"),
                              _dev(ws, "ws") if ws is not None else None, ws_bytes,
                              OC_FUSE_RELU if relu else 0, _stream()))
    return y, sw


def oc_conv_fwd_noalloc(tree: Octree, depth: int, ksize: int, stride: int, x: torch.Tensor,
                        w: torch.Tensor, y: torch.Tensor, relu: bool = False) -> torch.Tensor:
    """oc_conv_fwd with the library's static workspace (no allocation by the
    library; y is the caller's)."""
    K3, cin, cout, n_in, n_out = _conv_dims(tree, depth, stride, x, w)
    if K3 != ksize ** 3:
        raise OcError(1, f"w has {K3} taps, expected {ksize ** 3}")
    dt = _dtype_code(x)
    if w.dtype != x.dtype:
        raise OcError(1, "x and w must share a dtype")
    _check(load().oc_conv_fwd_noalloc(tree.handle, depth, ksize, stride, dt, _dev(x, "x"), cin,
                                      _dev(w, "w"), cout,
                                      _dev(y, "y", torch.float32, (n_out, cout)),
                                      OC_FUSE_RELU if relu else 0, _stream()))
    return y


def oc_conv_bwd(tree: Octree, depth: int, ksize: int, stride: int, x: torch.Tensor,
                w: torch.Tensor, dy: torch.Tensor, y: torch.Tensor | None = None,
                relu: bool = False, need_dx: bool = True, need_dw: bool = True,
                dw_out: torch.Tensor | None = None, defer: list | None = None):
    """(dx or None, dw or None); dw_out: a caller tensor to write dw into.
    defer: a list; when the layer's weight gradient has a deferred form
    (oc_conv_dw_partials), its partial sums stay in this call's workspace, a
    record is appended to the list, and dw is written by oc_sum_partials(defer)."""
    K3, cin, cout, n_in, n_out = _conv_dims(tree, depth, stride, x, w)
    if K3 != ksize ** 3:
        raise OcError(1, f"w has {K3} taps, expected {ksize ** 3}")
    dt = _dtype_code(w)
    L = load()
    dx = torch.empty((n_in, cin), dtype=torch.float32, device=w.device) if need_dx else None
    dw = None
    if need_dw:
        dw = (dw_out.view(K3, cin, cout) if dw_out is not None else
              torch.empty((K3, cin, cout), dtype=torch.float32, device=w.device))
    ws_bytes = L.oc_conv_bwd_workspace(tree.handle, depth, ksize, stride, dt, cin, cout)
    ws = torch.empty(max(int(ws_bytes), 1), dtype=torch.uint8, device=w.device)
    yp = _dev(y, "y", torch.float32, (n_out, cout)) if relu else None
    flags = OC_FUSE_RELU if relu else 0
    rec = None
    if defer is not None and need_dw:
        off, npart, cnt = C.c_size_t(0), C.c_int32(0), C.c_int64(0)
        _check(L.oc_conv_dw_partials(tree.handle, depth, ksize, stride, dt, cin, cout,
                                     C.byref(off), C.byref(npart), C.byref(cnt)))
        if npart.value > 0:
            flags |= OC_DEFER_DW
            rec = (ws, off.value, npart.value, cnt.value, dw)
    _check(L.oc_conv_bwd(tree.handle, depth, ksize, stride, dt, _dev(x, "x") if x is not None else None,
                         cin, _dev(w, "w"), cout, yp,
                         _dev(dy, "dy", torch.float32, (n_out, cout)),
                         _dev(dx, "dx") if dx is not None else None,
                         _dev(dw, "dw") if dw is not None else None,
                         _dev(ws, "ws"), ws.numel(), flags, _stream()))
    if rec is not None:
        defer.append(rec)
    return dx, dw


def oc_sum_partials(defer: list) -> None:
    """Write the weight gradients of the oc_conv_bwd calls recorded in defer
    (their partial sums, one launch per eight layers) and empty the list."""
    if not defer:
        return
    L = load()
    n = len(defer)
    parts = (C.c_void_p * n)(*[r[0].data_ptr() + r[1] for r in defer])
    nparts = (C.c_int32 * n)(*[r[2] for r in defer])
    counts = (C.c_int64 * n)(*[r[3] for r in defer])
    outs = (C.c_void_p * n)(*[_dev(r[4], "dw") for r in defer])
    _check(L.oc_sum_partials(n, parts, nparts, counts, outs, _stream()))
    defer.clear()


def oc_round_bf16(x: torch.Tensor) -> torch.Tensor:
    """x (f32, any shape) rounded to a bf16 tensor of the same shape: the
    operand of a bf16 layer after a layer with f32 output."""
    y = torch.empty(x.shape, dtype=torch.bfloat16, device=x.device)
    _check(load().oc_round_bf16(x.numel(), _dev(x, "x", torch.float32), _dev(y, "y"),
                                _stream()))
    return y


def oc_conv_bwd_pool(tree: Octree, depth: int, ksize: int, w: torch.Tensor, dy: torch.Tensor,
                     sw: torch.Tensor, xp: torch.Tensor | None = None,
                     y: torch.Tensor | None = None, relu: bool = False,
                     dym: torch.Tensor | None = None) -> torch.Tensor:
    """Input gradient of the stride-1 fp32 convolution at depth (input: the
    2x2x2 max-pool of depth + 1 with switches sw), routed on through that
    pooling: [N_{depth+1}][cin].  xp: the pooled values (the convolution's
    input), masking the gradient as oc_pool_bwd's y; relu with y: the
    convolution's own ReLU applied to dy first, the masked dy also written
    to dym when given."""
    K3, cin, cout = w.shape
    if K3 != ksize ** 3:
        raise OcError(1, f"w has {K3} taps, expected {ksize ** 3}")
    if not 1 <= depth < tree.depth:
        raise OcError(1, f"depth {depth} not in 1..{tree.depth - 1}")
    n_l, n_f, m = tree.num(depth), tree.num(depth + 1), tree.nonempty(depth)
    L = load()
    dxf = torch.empty((n_f, cin), dtype=torch.float32, device=w.device)
    ws_bytes = int(L.oc_conv_bwd_pool_workspace(tree.handle, depth, ksize, cin, cout))
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=w.device)
    _check(L.oc_conv_bwd_pool(tree.handle, depth, ksize, _dev(w, "w", torch.float32), cin, cout,
                              _dev(y, "y", torch.float32, (n_l, cout)) if relu else None,
                              _dev(dy, "dy", torch.float32, (n_l, cout)),
                              _dev(xp, "xp", torch.float32, (n_l, cin)) if xp is not None else None,
                              _dev(sw, "sw", torch.uint8, (m, cin)), _dev(dxf, "dxf"),
                              _dev(dym, "dym", torch.float32, (n_l, cout))
                              if dym is not None and relu else None,
                              _dev(ws, "ws"), ws.numel(), OC_FUSE_RELU if relu else 0, _stream()))
    return dxf


def _deconv_dims(tree: Octree, depth: int, stride: int, x, w):
    """Rows of the input and output of a deconvolution to depth `depth`, and
    its channels (w is [K^3][cout][cin])."""
    if not 1 <= depth <= tree.depth:
        raise OcError(1, f"depth {depth} not in 1..{tree.depth}")
    K3, cout, cin = w.shape
    r = int(stride).bit_length() - 1  # stride 2^r
    if not 0 <= r <= depth:
        raise OcError(1, f"stride {stride} needs depth >= {r}")
    n_out = tree.num(depth)
    n_in = tree.num(depth - r)
    if x is not None and tuple(x.shape) != (n_in, cin):
        raise OcError(1, f"x has shape {tuple(x.shape)}, expected {(n_in, cin)}")
    return K3, cin, cout, n_in, n_out


def oc_deconv_fwd(tree: Octree, depth: int, ksize: int, stride: int, x: torch.Tensor,
                  w: torch.Tensor, y: torch.Tensor | None = None) -> torch.Tensor:
    """Deconvolution to depth `depth` (Sec. 3.2); w [K^3][cout][cin] is the
    weight of the convolution cout -> cin it transposes."""
    K3, cin, cout, n_in, n_out = _deconv_dims(tree, depth, stride, x, w)
    if K3 != ksize ** 3:
        raise OcError(1, f"w has {K3} taps, expected {ksize ** 3}")
    dt = _dtype_code(x)
    if w.dtype != x.dtype:
        raise OcError(1, "x and w must share a dtype")
    if y is None:
        y = torch.empty((n_out, cout), dtype=torch.float32, device=x.device)
    L = load()
    ws_bytes = int(L.oc_deconv_fwd_workspace(tree.handle, depth, ksize, stride, dt, cin, cout))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=x.device) if ws_bytes else None
    _check(L.oc_deconv_fwd(tree.handle, depth, ksize, stride, dt, _dev(x, "x"), cin,
                           _dev(w, "w"), cout,
                           _dev(y, "y", torch.float32, (n_out, cout)),
                           _dev(ws, "ws") if ws is not None else None, ws_bytes, 0, _stream()))
    return y


def oc_deconv_bwd(tree: Octree, depth: int, ksize: int, stride: int, x: torch.Tensor,
                  w: torch.Tensor, dy: torch.Tensor, need_dx: bool = True,
                  need_dw: bool = True):
    """Input and weight gradients of oc_deconv_fwd: (dx or None, dw or None)."""
    K3, cin, cout, n_in, n_out = _deconv_dims(tree, depth, stride, x, w)
    if K3 != ksize ** 3:
        raise OcError(1, f"w has {K3} taps, expected {ksize ** 3}")
    dt = _dtype_code(w)
    L = load()
    dx = torch.empty((n_in, cin), dtype=torch.float32, device=w.device) if need_dx else None
    dw = torch.empty((K3, cout, cin), dtype=torch.float32, device=w.device) if need_dw else None
    ws_bytes = int(L.oc_deconv_bwd_workspace(tree.handle, depth, ksize, stride, dt, cin, cout))
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=w.device)
    _check(L.oc_deconv_bwd(tree.handle, depth, ksize, stride, dt,
                           _dev(x, "x") if x is not None else None, cin, _dev(w, "w"), cout,
                           _dev(dy, "dy", torch.float32, (n_out, cout)),
                           _dev(dx, "dx") if dx is not None else None,
                           _dev(dw, "dw") if dw is not None else None,
                           _dev(ws, "ws"), ws.numel(), 0, _stream()))
    return dx, dw


def oc_pool_fwd(tree: Octree, depth: int, x: torch.Tensor):
    c = x.shape[1]
    n_in, n_out, m = tree.num(depth), tree.num(depth - 1), tree.nonempty(depth - 1)
    y = torch.empty((n_out, c), dtype=torch.float32, device=x.device)
    sw = torch.empty((m, c), dtype=torch.uint8, device=x.device)
    _check(load().oc_pool_fwd(tree.handle, depth, _dev(x, "x", torch.float32, (n_in, c)), c,
                              _dev(y, "y"), _dev(sw, "sw"), _stream()))
    return y, sw


def oc_pool_bwd(tree: Octree, depth: int, dy: torch.Tensor, sw: torch.Tensor,
                y: torch.Tensor | None = None) -> torch.Tensor:
    """y: the pooled output, when a ReLU came before the pooling: its backward
    is then applied too (entries with y <= 0 get no gradient)."""
    c = dy.shape[1]
    n_in, n_out, m = tree.num(depth), tree.num(depth - 1), tree.nonempty(depth - 1)
    dx = torch.empty((n_in, c), dtype=torch.float32, device=dy.device)
    yp = _dev(y, "y", torch.float32, (n_out, c)) if y is not None else None
    _check(load().oc_pool_bwd(tree.handle, depth, _dev(dy, "dy", torch.float32, (n_out, c)),
                              _dev(sw, "sw", torch.uint8, (m, c)), c, yp, _dev(dx, "dx"),
                              _stream()))
    return dx


def oc_unpool_fwd(tree: Octree, depth: int, x: torch.Tensor, sw: torch.Tensor) -> torch.Tensor:
    c = x.shape[1]
    n_l, n_p, m = tree.num(depth), tree.num(depth - 1), tree.nonempty(depth - 1)
    y = torch.empty((n_l, c), dtype=torch.float32, device=x.device)
    _check(load().oc_unpool_fwd(tree.handle, depth, _dev(x, "x", torch.float32, (n_p, c)),
                                _dev(sw, "sw", torch.uint8, (m, c)), c, _dev(y, "y"), _stream()))
    return y


def oc_unpool_bwd(tree: Octree, depth: int, dy: torch.Tensor, sw: torch.Tensor) -> torch.Tensor:
    c = dy.shape[1]
    n_l, n_p, m = tree.num(depth), tree.num(depth - 1), tree.nonempty(depth - 1)
    dx = torch.empty((n_p, c), dtype=torch.float32, device=dy.device)
    _check(load().oc_unpool_bwd(tree.handle, depth, _dev(dy, "dy", torch.float32, (n_l, c)),
                                _dev(sw, "sw", torch.uint8, (m, c)), c, _dev(dx, "dx"), _stream()))
    return dx


def oc_gpool_fwd(tree: Octree, depth: int, ksize: int, mode: int, x: torch.Tensor,
                 stride: int = 1):
    """General pooling over the K^3 neighbourhood (Sec. 3.2), stride 1 or 2^r:
    (y, sw) for OC_POOL_MAX, (y, None) for OC_POOL_AVG."""
    r = int(stride).bit_length() - 1
    n_in, n = tree.num(depth), tree.num(depth - r)
    c = x.shape[1]
    y = torch.empty((n, c), dtype=torch.float32, device=x.device)
    sw = (torch.empty((n, c), dtype=torch.uint8, device=x.device) if mode == OC_POOL_MAX
          else None)
    _check(load().oc_gpool_fwd(tree.handle, depth, ksize, stride, mode,
                               _dev(x, "x", torch.float32, (n_in, c)), c, _dev(y, "y"),
                               _dev(sw, "sw") if sw is not None else None, _stream()))
    return y, sw


def oc_gpool_bwd(tree: Octree, depth: int, ksize: int, mode: int, dy: torch.Tensor,
                 sw: torch.Tensor | None, stride: int = 1) -> torch.Tensor:
    r = int(stride).bit_length() - 1
    n_in, n = tree.num(depth), tree.num(depth - r)
    c = dy.shape[1]
    dx = torch.empty((n_in, c), dtype=torch.float32, device=dy.device)
    _check(load().oc_gpool_bwd(tree.handle, depth, ksize, stride, mode,
                               _dev(dy, "dy", torch.float32, (n, c)),
                               _dev(sw, "sw", torch.uint8, (n, c)) if sw is not None else None,
                               c, _dev(dx, "dx"), _stream()))
    return dx


# --- the rest of the O-CNN(d) training iteration --------------------------


def _opt(t, name, **kw):
    return _dev(t, name, **kw) if t is not None else None


def oc_bn_fwd(x: torch.Tensor, gamma: torch.Tensor, beta: torch.Tensor, eps: float = 1e-5,
              relu: bool = False):
    """Batch normalisation over the rows of x [n][c] (training mode):
    (y, mean, invstd)."""
    n, c = x.shape
    y = torch.empty_like(x)
    mean = torch.empty(c, dtype=torch.float32, device=x.device)
    invstd = torch.empty(c, dtype=torch.float32, device=x.device)
    L = load()
    ws = torch.empty(max(int(L.oc_bn_workspace(n, c)), 1), dtype=torch.uint8, device=x.device)
    _check(L.oc_bn_fwd(n, c, _dev(x, "x", torch.float32), _dev(gamma, "gamma", torch.float32),
                       _dev(beta, "beta", torch.float32), eps, OC_FUSE_RELU if relu else 0,
                       _dev(y, "y"), _dev(mean, "mean"), _dev(invstd, "invstd"), _dev(ws, "ws"),
                       ws.numel(), _stream()))
    return y, mean, invstd


def oc_bn_pool_fwd(tree: Octree, depth: int, z: torch.Tensor, gamma: torch.Tensor,
                   beta: torch.Tensor, eps: float = 1e-5, relu: bool = True):
    """Batch normalisation of z [N_l][c] (training mode), optional ReLU and
    the 2x2x2 max-pool to depth - 1 in one call: (pooled, switches, mean,
    invstd)."""
    n, c = z.shape
    if n != tree.num(depth):
        raise OcError(1, f"z has {n} rows, depth {depth} has {tree.num(depth)}")
    n_p, m = tree.num(depth - 1), tree.nonempty(depth - 1)
    y = torch.empty((n_p, c), dtype=torch.float32, device=z.device)
    sw = torch.empty((m, c), dtype=torch.uint8, device=z.device)
    mean = torch.empty(c, dtype=torch.float32, device=z.device)
    invstd = torch.empty(c, dtype=torch.float32, device=z.device)
    L = load()
    ws = torch.empty(max(int(L.oc_bn_workspace(n, c)), 1), dtype=torch.uint8, device=z.device)
    _check(L.oc_bn_pool_fwd(tree.handle, depth, c, _dev(z, "z", torch.float32),
                            _dev(gamma, "gamma", torch.float32), _dev(beta, "beta", torch.float32),
                            eps, OC_FUSE_RELU if relu else 0, _dev(y, "y"), _dev(sw, "sw"),
                            _dev(mean, "mean"), _dev(invstd, "invstd"), _dev(ws, "ws"),
                            ws.numel(), _stream()))
    return y, sw, mean, invstd


def oc_bn_bwd(x, dy, gamma, mean, invstd, dgamma=None, dbeta=None):
    """(dx, dgamma, dbeta) of oc_bn_fwd (without its ReLU); dgamma, dbeta:
    optional caller tensors to write into."""
    n, c = x.shape
    dx = torch.empty_like(x)
    dg = dgamma if dgamma is not None else torch.empty(c, dtype=torch.float32, device=x.device)
    db = dbeta if dbeta is not None else torch.empty(c, dtype=torch.float32, device=x.device)
    L = load()
    ws = torch.empty(max(int(L.oc_bn_workspace(n, c)), 1), dtype=torch.uint8, device=x.device)
    _check(L.oc_bn_bwd(n, c, _dev(x, "x", torch.float32), _dev(dy, "dy", torch.float32, (n, c)),
                       _dev(gamma, "gamma", torch.float32), _dev(mean, "mean"),
                       _dev(invstd, "invstd"), _dev(dx, "dx"), _dev(dg, "dgamma"),
                       _dev(db, "dbeta"), _dev(ws, "ws"), ws.numel(), _stream()))
    return dx, dg, db


def oc_fc_fwd(x, w, b=None):
    B, cin = x.shape
    cout = w.shape[1]
    y = torch.empty((B, cout), dtype=torch.float32, device=x.device)
    _check(load().oc_fc_fwd(B, cin, cout, _dev(x, "x", torch.float32),
                            _dev(w, "w", torch.float32, (cin, cout)), _opt(b, "b"), _dev(y, "y"),
                            _stream()))
    return y


def oc_fc_bwd(x, w, dy, need_dx=True, dw=None, db=None):
    """(dx or None, dw, db); dw, db: optional caller tensors to write into."""
    B, cin = x.shape
    cout = w.shape[1]
    dx = torch.empty_like(x) if need_dx else None
    dw = dw if dw is not None else torch.empty_like(w)
    db = db if db is not None else torch.empty(cout, dtype=torch.float32, device=x.device)
    _check(load().oc_fc_bwd(B, cin, cout, _dev(x, "x", torch.float32), _dev(w, "w"),
                            _dev(dy, "dy", torch.float32, (B, cout)), _opt(dx, "dx"),
                            _dev(dw, "dw"), _dev(db, "db"), _stream()))
    return dx, dw, db


def oc_dropout(x, keep, p):
    y = torch.empty_like(x)
    _check(load().oc_dropout(x.numel(), _dev(x, "x", torch.float32),
                             _dev(keep, "keep", torch.uint8, tuple(x.shape)), p, _dev(y, "y"),
                             _stream()))
    return y


def oc_softmax_ce(z, labels):
    """(loss as a 0-d device tensor, dz)."""
    B, nc = z.shape
    loss = torch.empty((), dtype=torch.float32, device=z.device)
    dz = torch.empty_like(z)
    L = load()
    ws = torch.empty(max(int(L.oc_softmax_ce_workspace(B)), 1), dtype=torch.uint8,
                     device=z.device)
    _check(L.oc_softmax_ce(B, nc, _dev(z, "z", torch.float32),
                           _dev(labels, "labels", torch.int32, (B,)), _dev(loss, "loss"),
                           _dev(dz, "dz"), _dev(ws, "ws"), ws.numel(), _stream()))
    return loss, dz


def oc_sgd(w, g, v, lr, momentum, decay):
    """In place: v = momentum v + lr (g + decay w), w -= v."""
    _check(load().oc_sgd(w.numel(), _dev(w, "w", torch.float32),
                         _dev(g, "g", torch.float32, tuple(w.shape)),
                         _dev(v, "v", torch.float32, tuple(w.shape)), lr, momentum, decay,
                         _stream()))
