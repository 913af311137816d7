"""ctypes binding of libmemfine.so, the MI355X chunked MoE expert layer.

Argument marshalling only: every function here turns torch tensors into raw
pointers and sizes, checks on the host that they match the shape the kernels
will assume (so that no kernel is launched on a mismatched buffer), and calls
the C entry point of the same name declared in include/memfine.h.  There is
no fallback: if the library is not built, loading it raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmemfine.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_BUDGET, ERR_OOM, ERR_HIP = 0, -1, -2, -3, -4, -5
ERR_SCRATCH = -6
NOALLOC_SCRATCH_BYTES = 64 << 20
BF16, F32 = 0, 1
PASS_FWD, PASS_BWD = 0, 1

KERNELS = ["count", "dispatch", "fc1", "fc2", "combine", "fc1_recompute", "fc2_dgrad",
           "fc2_wgrad", "fc1_wgrad", "fc1_dgrad", "unpermute", "fc1_dgrad_wgrad",
           "router_fwd", "router_bwd_dx", "router_wgrad", "router_reduce"]


class MemfineError(RuntimeError):
    def __init__(self, code: int, where: str):
        super().__init__(f"{where}: {status_str(code)} ({code})")
        self.code = code


class Shape(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int64), ("h", ctypes.c_int32), ("F", ctypes.c_int32),
                ("E", ctypes.c_int32), ("k", ctypes.c_int32), ("dtype", ctypes.c_int32)]


ALLOC_FN = ctypes.CFUNCTYPE(ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p)
RELEASE_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                              ctypes.c_void_p)


class Allocator(ctypes.Structure):
    _fields_ = [("alloc", ALLOC_FN), ("release", RELEASE_FN), ("ctx", ctypes.c_void_p)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("s_recv", ctypes.c_int64), ("beta", ctypes.c_int64), ("avail", ctypes.c_int64),
                ("s_max", ctypes.c_double), ("c_theory", ctypes.c_int64),
                ("chunks", ctypes.c_int32), ("fits", ctypes.c_int32),
                ("paper_peak_bytes", ctypes.c_int64), ("beta_paper", ctypes.c_int64),
                ("beta_impl", ctypes.c_int64), ("workspace_bytes", ctypes.c_int64),
                ("paper_chunks", ctypes.c_int32), ("reserved", ctypes.c_int32)]


TILE_AUTO, TILE_128, TILE_256, TILE_256_REG = 0, 1, 2, 3
CHUNK_TOKENS, CHUNK_EXPERTS = 0, 1


class LaunchOptions(ctypes.Structure):
    """memfine_launch_options: GEMM tile shape, tile order, split tail, paired
    FC1 backward launch, side streams (all bit-identical), chunk order."""
    _fields_ = [("tile", ctypes.c_int32), ("raster", ctypes.c_int32),
                ("split_tail", ctypes.c_int32), ("pair", ctypes.c_int32),
                ("streams", ctypes.c_int32), ("chunk_order", ctypes.c_int32)]


class Model(ctypes.Structure):
    """memfine_model: the memory model's configuration (notation-table symbols)."""
    _fields_ = [("b", ctypes.c_int64), ("s", ctypes.c_int64), ("h", ctypes.c_int64),
                ("a", ctypes.c_int64), ("h_d", ctypes.c_int64), ("k_a", ctypes.c_int64),
                ("e_n", ctypes.c_int64), ("g_e", ctypes.c_int64), ("t", ctypes.c_int32),
                ("c", ctypes.c_int32), ("v", ctypes.c_int32), ("p", ctypes.c_int32),
                ("D_t", ctypes.c_int32), ("full_recompute", ctypes.c_int32)]


class KernelStat(ctypes.Structure):
    _fields_ = [("launches", ctypes.c_int64), ("total_ms", ctypes.c_double),
                ("flops", ctypes.c_double), ("bytes", ctypes.c_double)]


_LIB = None
P = ctypes.c_void_p
I32P = ctypes.POINTER(ctypes.c_int32)
I64P = ctypes.POINTER(ctypes.c_int64)
SHP = ctypes.POINTER(Shape)
ALP = ctypes.POINTER(Allocator)

_SIGS = {
    "memfine_count": (ctypes.c_int, [SHP, P, P, I64P, P]),
    "memfine_dispatch": (ctypes.c_int, [SHP, P, ctypes.c_int64, ctypes.c_int64, P, P, P, P, ALP, P]),
    "memfine_plan": (ctypes.c_int, [SHP, I64P, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                    I32P, ctypes.c_int32, I32P, ctypes.POINTER(PlanInfo)]),
    "memfine_workspace_bytes": (ctypes.c_int64, [SHP, ctypes.c_int32, ctypes.c_int32]),
    "memfine_workspace_held": (ctypes.c_int, [P, I64P]),
    "memfine_workspace_trim": (ctypes.c_int, [P, ctypes.c_int64]),
    "memfine_pool_high_water": (ctypes.c_int, [I64P, ctypes.c_int32]),
    "memfine_set_launch_options": (ctypes.c_int, [ctypes.POINTER(LaunchOptions)]),
    "memfine_get_launch_options": (ctypes.c_int, [ctypes.POINTER(LaunchOptions)]),
    "memfine_moe_fwd": (ctypes.c_int, [SHP, ctypes.c_int32, P, P, P, P, P, P, ALP, P]),
    "memfine_moe_fwd_noalloc": (ctypes.c_int, [SHP, ctypes.c_int32, P, P, P, P, P, P, P]),
    "memfine_moe_bwd": (ctypes.c_int, [SHP, ctypes.c_int32, P, P, P, P, P, P, P, P, P, P,
                                       ctypes.c_int32, ALP, P]),
    "memfine_static_memory": (ctypes.c_int, [I64P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                             ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, I64P]),
    "memfine_activation_memory": (ctypes.c_int, [ctypes.POINTER(Model), ctypes.c_int32,
                                                 ctypes.c_int64, I64P]),
    "memfine_mact_thresholds": (ctypes.c_int, [ctypes.POINTER(Model), ctypes.c_int32, ctypes.c_int64,
                                               ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, I32P,
                                               ctypes.c_int32, I64P]),
    "memfine_mact_select": (ctypes.c_int, [I32P, I64P, ctypes.c_int32, ctypes.c_int64, I32P]),
    "memfine_router_fwd": (ctypes.c_int, [SHP, P, P, P, P, P, P]),
    "memfine_router_bwd": (ctypes.c_int, [SHP, P, P, P, P, P, P, P, ctypes.c_int32,
                                          ctypes.c_int32, ALP, P]),
    "memfine_status_str": (ctypes.c_char_p, [ctypes.c_int]),
    "memfine_profile_begin": (ctypes.c_int, [ctypes.c_uint32]),
    "memfine_profile_end": (ctypes.c_int, [ctypes.POINTER(KernelStat)]),
}


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2511_21431_amd.build` (there is no fallback)")
        # torch first, when it is installed: the library then binds to the HIP
        # runtime torch has loaded.  Loaded before torch, it would bring in the
        # system's runtime, and torch would load its own beside it; two runtimes
        # in one process share neither device memory nor streams, and the
        # library's first launch on torch's tensors fails.
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = L
    return _LIB


def status_str(code: int) -> str:
    return lib().memfine_status_str(int(code)).decode()


def _check(code: int, where: str, allow=(OK,)) -> int:
    if code not in allow:
        raise MemfineError(code, where)
    return code


def make_shape(T: int, h: int, F: int, E: int, k: int, dtype: int) -> Shape:
    return Shape(int(T), int(h), int(F), int(E), int(k), int(dtype))


# ----------------------------------------------------------- tensor checks
def _torch():
    import torch
    return torch


def _dt(shape: Shape):
    torch = _torch()
    return torch.bfloat16 if shape.dtype == BF16 else torch.float32


def _ptr(t, shape_tuple, dtype, name):
    if t is None:
        raise ValueError(f"{name} is required")
    if tuple(t.shape) != tuple(shape_tuple):
        raise ValueError(f"{name}: shape {tuple(t.shape)} != expected {tuple(shape_tuple)}")
    if t.dtype != dtype:
        raise ValueError(f"{name}: dtype {t.dtype} != expected {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if not t.is_cuda and t.numel() > 0:
        raise ValueError(f"{name} must be a device tensor")
    return ctypes.c_void_p(t.data_ptr() if t.numel() > 0 else 0)


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        torch = _torch()
        stream = torch.cuda.current_stream()
    if hasattr(stream, "cuda_stream"):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


class TorchAllocator:
    """Serves the layer's per-chunk buffers from torch's caching allocator,
    so that torch.cuda.max_memory_allocated sees the layer's true peak.

    The library asks for and hands back each buffer in order on the stream of
    its call: a buffer is allocated on that stream (torch then reuses it only
    in that stream's order), and released with record_stream on it, so torch
    never hands the memory to other work before the library's kernels that
    use it have run."""

    def __init__(self, device=None):
        torch = _torch()
        self.device = torch.device("cuda", torch.cuda.current_device()) if device is None else device
        self.live: Dict[int, object] = {}
        self.live_bytes = 0
        self.high_water = 0                    # most bytes held at once
        self.calls = 0
        self.fail_at: Optional[int] = None     # for tests: fail the n-th allocation
        self._alloc = ALLOC_FN(self._do_alloc)
        self._release = RELEASE_FN(self._do_release)
        self.struct = Allocator(self._alloc, self._release, None)

    def _stream(self, stream):
        """The torch stream object for the library's stream handle."""
        torch = _torch()
        ptr = int(stream or 0)
        for cand in (torch.cuda.current_stream(self.device), torch.cuda.default_stream(self.device)):
            if cand.cuda_stream == ptr:
                return cand
        return torch.cuda.ExternalStream(ptr, device=self.device)

    def _do_alloc(self, nbytes, stream, ctx):
        torch = _torch()
        self.calls += 1
        if self.fail_at is not None and self.calls >= self.fail_at:
            return None
        with torch.cuda.stream(self._stream(stream)):
            t = torch.empty(int(nbytes), dtype=torch.uint8, device=self.device)
        p = t.data_ptr()
        self.live[p] = t
        self.live_bytes += int(nbytes)
        self.high_water = max(self.high_water, self.live_bytes)
        return p

    def _do_release(self, ptr, nbytes, stream, ctx):
        t = self.live.pop(int(ptr), None)
        if t is not None:
            t.record_stream(self._stream(stream))
            self.live_bytes -= int(nbytes)


def _alloc_arg(allocator):
    if allocator is None:
        return None
    if isinstance(allocator, TorchAllocator):
        return ctypes.byref(allocator.struct)
    return ctypes.byref(allocator)


# --------------------------------------------------------------- entry points
def memfine_count(shape: Shape, idx, work, stream=None) -> np.ndarray:
    torch = _torch()
    out = np.zeros(shape.E, dtype=np.int64)
    rc = lib().memfine_count(ctypes.byref(shape), _ptr(idx, (shape.T, shape.k), torch.int32, "idx"),
                             _ptr(work, (shape.E + 1,), torch.int32, "work"),
                             out.ctypes.data_as(I64P), _stream(stream))
    _check(rc, "memfine_count")
    return out


def memfine_dispatch(shape: Shape, idx, t0: int, t1: int, counts, offsets, sorted_slot,
                     row_of_slot, allocator=None, stream=None) -> None:
    torch = _torch()
    n = (t1 - t0) * shape.k
    rc = lib().memfine_dispatch(
        ctypes.byref(shape), _ptr(idx, (shape.T, shape.k), torch.int32, "idx"), int(t0), int(t1),
        _ptr(counts, (shape.E,), torch.int32, "counts"),
        _ptr(offsets, (shape.E + 1,), torch.int32, "offsets"),
        _ptr(sorted_slot, (n,), torch.int32, "sorted_slot"),
        _ptr(row_of_slot, (n,), torch.int32, "row_of_slot"), _alloc_arg(allocator),
        _stream(stream))
    _check(rc, "memfine_dispatch")


def memfine_plan(shape: Shape, counts: Sequence[int], budget_bytes: int, bins=(1, 2, 4, 8),
                 fixed_bytes: int = 0, beta_bytes: int = 0):
    """Returns (status, chunks, info dict); status is OK or ERR_BUDGET."""
    c = np.ascontiguousarray(np.asarray(counts, dtype=np.int64))
    b = np.ascontiguousarray(np.asarray(bins, dtype=np.int32))
    if c.size != shape.E:
        raise ValueError("counts must have E entries")
    out = ctypes.c_int32(0)
    info = PlanInfo()
    rc = lib().memfine_plan(ctypes.byref(shape), c.ctypes.data_as(I64P), int(budget_bytes),
                            int(fixed_bytes), int(beta_bytes), b.ctypes.data_as(I32P), int(b.size),
                            ctypes.byref(out), ctypes.byref(info))
    _check(rc, "memfine_plan", allow=(OK, ERR_BUDGET))
    return rc, int(out.value), {f: getattr(info, f) for f, _ in PlanInfo._fields_}


def make_model(**kw) -> Model:
    """memfine_model from keyword fields (b, s, h, a, h_d, k_a, e_n, g_e, t, c, v, p,
    D_t, full_recompute); unspecified fields default to 0 except the parallel
    sizes and b (1), D_t (2) and full_recompute (1)."""
    d = dict(b=1, t=1, c=1, v=1, p=1, D_t=2, full_recompute=1)
    d.update(kw)
    m = Model()
    for f, _ in Model._fields_:
        setattr(m, f, int(d.get(f, 0)))
    return m


def memfine_static_memory(S_para: Sequence[int], v: int, l: int, D_para: int = 2,
                          D_grad: int = 2, D_opt: int = 4) -> int:
    a = np.ascontiguousarray(np.asarray(list(S_para), dtype=np.int64))
    out = ctypes.c_int64(0)
    rc = lib().memfine_static_memory(a.ctypes.data_as(I64P), int(a.size), int(v), int(l),
                                     int(D_para), int(D_grad), int(D_opt), ctypes.byref(out))
    _check(rc, "memfine_static_memory")
    return int(out.value)


def memfine_activation_memory(model: Model, r_pp: int, s_recv: int) -> int:
    out = ctypes.c_int64(0)
    rc = lib().memfine_activation_memory(ctypes.byref(model), int(r_pp), int(s_recv),
                                         ctypes.byref(out))
    _check(rc, "memfine_activation_memory")
    return int(out.value)


def memfine_mact_thresholds(model: Model, r_pp: int, M_gpu: int, alpha_num: int, alpha_den: int,
                            M_sta: int, bins=(1, 2, 4, 8)) -> list:
    b = np.ascontiguousarray(np.asarray(bins, dtype=np.int32))
    out = np.zeros(b.size, dtype=np.int64)
    rc = lib().memfine_mact_thresholds(ctypes.byref(model), int(r_pp), int(M_gpu), int(alpha_num),
                                       int(alpha_den), int(M_sta), b.ctypes.data_as(I32P),
                                       int(b.size), out.ctypes.data_as(I64P))
    _check(rc, "memfine_mact_thresholds")
    return [int(x) for x in out]


def memfine_mact_select(bins: Sequence[int], thresholds: Sequence[int], s_recv: int):
    """Returns (status, chunks); status is OK or ERR_BUDGET."""
    b = np.ascontiguousarray(np.asarray(bins, dtype=np.int32))
    th = np.ascontiguousarray(np.asarray(thresholds, dtype=np.int64))
    if b.size != th.size:
        raise ValueError("one threshold per bin")
    out = ctypes.c_int32(0)
    rc = lib().memfine_mact_select(b.ctypes.data_as(I32P), th.ctypes.data_as(I64P), int(b.size),
                                   int(s_recv), ctypes.byref(out))
    _check(rc, "memfine_mact_select", allow=(OK, ERR_BUDGET))
    return rc, int(out.value)


def memfine_workspace_bytes(shape: Shape, chunks: int, pass_: int) -> int:
    v = lib().memfine_workspace_bytes(ctypes.byref(shape), int(chunks), int(pass_))
    if v < 0:
        raise MemfineError(int(v), "memfine_workspace_bytes")
    return int(v)


def memfine_workspace_held(stream=None) -> int:
    """Bytes of the library's cached workspace block for the stream."""
    out = ctypes.c_int64(0)
    _check(lib().memfine_workspace_held(_stream(stream), ctypes.byref(out)),
           "memfine_workspace_held")
    return int(out.value)


def memfine_workspace_trim(keep_bytes: int = 0, stream=None) -> None:
    _check(lib().memfine_workspace_trim(_stream(stream), int(keep_bytes)), "memfine_workspace_trim")


def memfine_pool_high_water(reset: bool = False) -> int:
    out = ctypes.c_int64(0)
    _check(lib().memfine_pool_high_water(ctypes.byref(out), 1 if reset else 0),
           "memfine_pool_high_water")
    return int(out.value)


def memfine_set_launch_options(tile: int = TILE_AUTO, raster: int = -1, split_tail: bool = True,
                               pair: bool = False, streams: bool = False,
                               chunk_order: int = CHUNK_TOKENS) -> None:
    o = LaunchOptions(int(tile), int(raster), int(bool(split_tail)), int(bool(pair)),
                      int(bool(streams)), int(chunk_order))
    _check(lib().memfine_set_launch_options(ctypes.byref(o)), "memfine_set_launch_options")


def memfine_get_launch_options() -> Dict[str, int]:
    o = LaunchOptions()
    _check(lib().memfine_get_launch_options(ctypes.byref(o)), "memfine_get_launch_options")
    return {f: getattr(o, f) for f, _ in LaunchOptions._fields_}


def memfine_moe_fwd(shape: Shape, chunks: int, X, idx, gates, W1, W2, Y, allocator=None,
                    stream=None) -> None:
    torch = _torch()
    dt = _dt(shape)
    T, h, F, E, k = shape.T, shape.h, shape.F, shape.E, shape.k
    rc = lib().memfine_moe_fwd(
        ctypes.byref(shape), int(chunks), _ptr(X, (T, h), dt, "X"),
        _ptr(idx, (T, k), torch.int32, "idx"), _ptr(gates, (T, k), torch.float32, "gates"),
        _ptr(W1, (E, 2 * F, h), dt, "W1"), _ptr(W2, (E, h, F), dt, "W2"),
        _ptr(Y, (T, h), dt, "Y"), _alloc_arg(allocator), _stream(stream))
    _check(rc, "memfine_moe_fwd")


def memfine_moe_fwd_noalloc(shape: Shape, chunks: int, X, idx, gates, W1, W2, Y,
                            stream=None) -> None:
    """memfine_moe_fwd with the chunk buffers in the library's static device
    scratch (no allocation); MemfineError(ERR_SCRATCH) when the largest chunk
    needs more than NOALLOC_SCRATCH_BYTES."""
    torch = _torch()
    dt = _dt(shape)
    T, h, F, E, k = shape.T, shape.h, shape.F, shape.E, shape.k
    rc = lib().memfine_moe_fwd_noalloc(
        ctypes.byref(shape), int(chunks), _ptr(X, (T, h), dt, "X"),
        _ptr(idx, (T, k), torch.int32, "idx"), _ptr(gates, (T, k), torch.float32, "gates"),
        _ptr(W1, (E, 2 * F, h), dt, "W1"), _ptr(W2, (E, h, F), dt, "W2"),
        _ptr(Y, (T, h), dt, "Y"), _stream(stream))
    _check(rc, "memfine_moe_fwd_noalloc")


def memfine_moe_bwd(shape: Shape, chunks: int, X, idx, gates, W1, W2, dY, dX, dW1, dW2, dgates,
                    accumulate_dW: bool = False, allocator=None, stream=None) -> None:
    torch = _torch()
    dt = _dt(shape)
    T, h, F, E, k = shape.T, shape.h, shape.F, shape.E, shape.k
    rc = lib().memfine_moe_bwd(
        ctypes.byref(shape), int(chunks), _ptr(X, (T, h), dt, "X"),
        _ptr(idx, (T, k), torch.int32, "idx"), _ptr(gates, (T, k), torch.float32, "gates"),
        _ptr(W1, (E, 2 * F, h), dt, "W1"), _ptr(W2, (E, h, F), dt, "W2"),
        _ptr(dY, (T, h), dt, "dY"), _ptr(dX, (T, h), dt, "dX"),
        _ptr(dW1, (E, 2 * F, h), torch.float32, "dW1"),
        _ptr(dW2, (E, h, F), torch.float32, "dW2"),
        _ptr(dgates, (T, k), torch.float32, "dgates"), 1 if accumulate_dW else 0,
        _alloc_arg(allocator), _stream(stream))
    _check(rc, "memfine_moe_bwd")


def memfine_status_str(code: int) -> str:
    return status_str(code)


def memfine_router_fwd(shape: Shape, X, Wr, idx, gates, logits=None, stream=None) -> None:
    """Router forward into caller-owned idx [T, k] int32, gates [T, k] fp32 and
    optionally logits [T, E] fp32."""
    torch = _torch()
    dt = _dt(shape)
    T, h, E, k = shape.T, shape.h, shape.E, shape.k
    rc = lib().memfine_router_fwd(
        ctypes.byref(shape), _ptr(X, (T, h), dt, "X"), _ptr(Wr, (E, h), dt, "Wr"),
        _ptr(idx, (T, k), torch.int32, "idx"), _ptr(gates, (T, k), torch.float32, "gates"),
        None if logits is None else _ptr(logits, (T, E), torch.float32, "logits"), _stream(stream))
    _check(rc, "memfine_router_fwd")


def memfine_router_bwd(shape: Shape, X, Wr, idx, gates, dgates, dX, dWr, accumulate_dX=False,
                       accumulate_dWr=False, allocator=None, stream=None) -> None:
    torch = _torch()
    dt = _dt(shape)
    T, h, E, k = shape.T, shape.h, shape.E, shape.k
    rc = lib().memfine_router_bwd(
        ctypes.byref(shape), _ptr(X, (T, h), dt, "X"), _ptr(Wr, (E, h), dt, "Wr"),
        _ptr(idx, (T, k), torch.int32, "idx"), _ptr(gates, (T, k), torch.float32, "gates"),
        _ptr(dgates, (T, k), torch.float32, "dgates"), _ptr(dX, (T, h), dt, "dX"),
        _ptr(dWr, (E, h), torch.float32, "dWr"), int(bool(accumulate_dX)),
        int(bool(accumulate_dWr)), _alloc_arg(allocator), _stream(stream))
    _check(rc, "memfine_router_bwd")


def memfine_profile_begin(kernels: Sequence[str] = tuple(KERNELS)) -> None:
    mask = 0
    for name in kernels:
        mask |= 1 << KERNELS.index(name)
    _check(lib().memfine_profile_begin(mask), "memfine_profile_begin")


def memfine_profile_end() -> Dict[str, Dict[str, float]]:
    arr = (KernelStat * len(KERNELS))()
    _check(lib().memfine_profile_end(arr), "memfine_profile_end")
    return {name: {"launches": arr[i].launches, "total_ms": arr[i].total_ms,
                   "flops": arr[i].flops, "bytes": arr[i].bytes}
            for i, name in enumerate(KERNELS) if arr[i].launches > 0}
