"""Python binding of libsra (include/sra.h): argument marshalling only.

Every step of Sparse Reference Attention runs in the HIP library; this module turns torch
tensors into pointers, sizes and the current HIP stream, allocates outputs/workspace with
torch, and maps status codes to exceptions. It fails loudly if the library is missing.
"""
from __future__ import annotations

import ctypes
import math
import os
import re
from typing import Dict, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsra.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "sra.h")

SRA_OK = 0
SRA_ERR_INVALID_ARGUMENT = 1
SRA_ERR_UNSUPPORTED = 2
SRA_ERR_WORKSPACE_TOO_SMALL = 3
SRA_ERR_HIP = 4
SRA_ERR_INTERNAL = 5

SCHED_FORWARD = 0
SCHED_BWD_DQ = 1
SCHED_BWD_DKDV = 2


class SRAError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{status_string(status)}: {message}")
        self.status = status


class _SampleGeom(ctypes.Structure):
    _fields_ = [
        ("gen_frames", ctypes.c_int32), ("gen_h", ctypes.c_int32), ("gen_w", ctypes.c_int32),
        ("ref_frames", ctypes.c_int32), ("ref_h", ctypes.c_int32), ("ref_w", ctypes.c_int32),
        ("group_frames", ctypes.c_int32), ("gen_window", ctypes.c_int32), ("ref_frame_valid", ctypes.c_void_p),
        ("ref_token_valid", ctypes.c_void_p),
    ]


class _Problem(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32), ("num_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float), ("samples", ctypes.POINTER(_SampleGeom)),
        ("gen_token_stride", ctypes.c_int64), ("ref_token_stride", ctypes.c_int64),
        ("flags", ctypes.c_uint32),
    ]


_lib_handle = None


def lib() -> ctypes.CDLL:
    """Loads libsra.so from this package directory (raises if it was not built).

    SRA_HOST_LIB names another build of the library to load instead: the host-only build of
    `build.py --sanitize` (scheduler and C ABI under AddressSanitizer and UBSan, no kernels),
    for the sanitizer run of the host tests. Its launches all fail with SRA_ERR_HIP."""
    global _lib_handle
    if _lib_handle is not None:
        return _lib_handle
    path = os.environ.get("SRA_HOST_LIB") or LIB_PATH
    if not os.path.exists(path):
        raise ImportError(f"libsra.so is not built ({path}); run `python -m paper_2606_13872_amd.build`")
    L = ctypes.CDLL(path)
    P = ctypes.POINTER(_Problem)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    sig = {
        "sra_workspace_size": [P, ctypes.c_int, ctypes.POINTER(sz)],
        "sra_forward": [P] + [vp] * 6 + [vp, vp, vp, vp] + [vp, sz, vp],
        "sra_forward_noalloc": [P] + [vp] * 6 + [vp, vp, vp, vp] + [vp],
        "sra_backward": [P] + [vp] * 6 + [vp, vp, vp, vp, vp, vp] + [vp] * 6 + [vp, sz, vp],
        "sra_pair_counts": [P, ctypes.POINTER(i64), ctypes.POINTER(i64)],
        "sra_schedule_info": [P, ctypes.c_int, ctypes.POINTER(i64), ctypes.POINTER(i64), ctypes.POINTER(i64)],
        "sra_schedule_mask": [P, ctypes.c_int, i32, vp],
        "sra_dense_mask": [P, i32, vp],
        "sra_schedule_export": [P, ctypes.c_int, vp, i64, vp, i64],
        "sra_release_caches": [],
        "sra_kernel_timing_enable": [ctypes.c_int],
        "sra_kernel_timing": [ctypes.c_int, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i64)],
    }
    for name, args in sig.items():
        if not hasattr(L, name):  # the host-only build has no sra_forward_noalloc (device code)
            continue
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    L.sra_status_string.argtypes = [ctypes.c_int]
    L.sra_status_string.restype = ctypes.c_char_p
    L.sra_last_error.argtypes = []
    L.sra_last_error.restype = ctypes.c_char_p
    L.sra_version.argtypes = []
    L.sra_version.restype = ctypes.c_int32
    _lib_handle = L
    return L


def status_string(status: int) -> str:
    try:
        return lib().sra_status_string(status).decode()
    except ImportError:
        return f"status {status}"


FLAG_GEN_QUERIES_ONLY = 1  # SRA_FLAG_GEN_QUERIES_ONLY: reference tokens are context only
FLAG_GEN_WINDOW = 2        # SRA_FLAG_GEN_WINDOW: temporal window on gen-gen attention


def _check(status: int) -> None:
    if status != SRA_OK:
        raise SRAError(status, lib().sra_last_error().decode())


def header_functions() -> list:
    """Names of the functions include/sra.h declares."""
    text = open(HEADER_PATH).read()
    return sorted(set(re.findall(r"^(?:sra_status|const char\*|int32_t)\s+(sra_\w+)\s*\(", text, re.M)))


class Problem:
    """A sra_problem built from per-sample geometry objects (attributes as in SampleGeom)."""

    def __init__(self, samples: Sequence, heads: int, head_dim: int, scale: Optional[float] = None,
                 gen_token_stride: int = 0, ref_token_stride: int = 0, flags: int = 0):
        self.samples = list(samples)
        self._geoms = (_SampleGeom * max(1, len(self.samples)))()
        self._valid = []
        # a window on any sample sets the flag; samples without one get a window over all frames
        if any(getattr(g, "gen_window", None) is not None for g in self.samples):
            flags |= FLAG_GEN_WINDOW
        for i, g in enumerate(self.samples):
            ptrs = []
            for name, n in (("frame_valid", g.ref_frames), ("ref_token_valid", g.ref_frames * g.ref_h * g.ref_w)):
                v = getattr(g, name, None)
                if v is None:
                    ptrs.append(None)
                    continue
                a = np.ascontiguousarray(np.asarray(v).astype(bool).astype(np.uint8))
                if a.shape != (n,):
                    raise ValueError(f"sample {i}: {name} needs {n} entries, got {a.shape}")
                self._valid.append(a)  # the library reads these host bytes during the call
                ptrs.append(a.ctypes.data_as(ctypes.c_void_p))
            w = getattr(g, "gen_window", None)
            self._geoms[i] = _SampleGeom(g.gen_frames, g.gen_h, g.gen_w, g.ref_frames, g.ref_h, g.ref_w,
                                         getattr(g, "group_frames", 1), g.gen_frames if w is None else int(w),
                                         ptrs[0], ptrs[1])
        self.c = _Problem(len(self.samples), heads, head_dim, 0.0 if scale is None else float(scale),
                          ctypes.cast(self._geoms, ctypes.POINTER(_SampleGeom)),
                          gen_token_stride, ref_token_stride, flags)
        self.heads, self.head_dim = heads, head_dim
        self.n_gen = sum(g.gen_frames * g.gen_h * g.gen_w for g in self.samples)
        self.n_ref = sum(g.ref_frames * g.ref_h * g.ref_w for g in self.samples)

    @property
    def ptr(self):
        return ctypes.byref(self.c)

    def workspace_size(self, backward: bool) -> int:
        """Bytes of workspace one call needs (fixed by the geometry, so asked once per direction)."""
        cache = self.__dict__.setdefault("_ws", {})
        b = bool(backward)
        if b not in cache:
            n = ctypes.c_size_t(0)
            _check(lib().sra_workspace_size(self.ptr, 1 if b else 0, ctypes.byref(n)))
            cache[b] = int(n.value)
        return cache[b]


_PROBLEMS: "OrderedDict" = None


_FROZEN_TYPES: Dict[type, bool] = {}


def _frozen_type(cls) -> bool:
    """Whether instances of cls are frozen dataclasses (immutable, so usable as a cache key)."""
    f = _FROZEN_TYPES.get(cls)
    if f is None:
        f = _FROZEN_TYPES[cls] = bool(getattr(getattr(cls, "__dataclass_params__", None), "frozen", False))
    return f


def _problem(samples, heads, head_dim, scale, gen_stride, ref_stride, flags) -> Problem:
    """Problem(...), reused across calls with the same geometry (samples are frozen, so a tuple of
    them is a key when their masks are tuples); built afresh when they cannot be hashed."""
    global _PROBLEMS
    from collections import OrderedDict

    if _PROBLEMS is None:
        _PROBLEMS = OrderedDict()
    frozen = all(_frozen_type(type(g)) for g in samples)
    try:
        if not frozen:  # geometry objects that may change between calls are never cached
            raise TypeError
        key = (tuple(samples), heads, head_dim, scale, gen_stride, ref_stride, flags)
        hit = _PROBLEMS.get(key)
    except TypeError:  # mutable geometry, or a mask given as a list or an array
        return Problem(samples, heads, head_dim, scale, gen_stride, ref_stride, flags)
    if hit is None:
        hit = Problem(samples, heads, head_dim, scale, gen_stride, ref_stride, flags)
        _PROBLEMS[key] = hit
        if len(_PROBLEMS) > 64:
            _PROBLEMS.popitem(last=False)
    else:
        _PROBLEMS.move_to_end(key)
    return hit


# ----------------------------------------------------------------------------- host hooks
def pair_counts(samples, heads=1, head_dim=128, flags=0) -> Tuple[int, int]:
    p = Problem(samples, heads, head_dim, flags=flags)
    g, r = ctypes.c_int64(0), ctypes.c_int64(0)
    _check(lib().sra_pair_counts(p.ptr, ctypes.byref(g), ctypes.byref(r)))
    return int(g.value), int(r.value)


def schedule_info(samples, which: int, heads=1, head_dim=128, flags=0) -> Tuple[int, int, int]:
    p = Problem(samples, heads, head_dim, flags=flags)
    a, b, c = ctypes.c_int64(0), ctypes.c_int64(0), ctypes.c_int64(0)
    _check(lib().sra_schedule_info(p.ptr, which, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)))
    return int(a.value), int(b.value), int(c.value)


def schedule_mask(samples, which: int, sample: int, heads=1, head_dim=128, flags=0):
    import numpy as np

    p = Problem(samples, heads, head_dim, flags=flags)
    g = p.samples[sample]
    n = g.gen_frames * g.gen_h * g.gen_w + g.ref_frames * g.ref_h * g.ref_w
    out = np.zeros((n, n), dtype=np.uint8)
    _check(lib().sra_schedule_mask(p.ptr, which, sample, out.ctypes.data_as(ctypes.c_void_p)))
    return out


def dense_mask(samples, sample: int, heads=1, head_dim=128, flags=0):
    """sra_dense_mask: the visibility rule of `sample` as a (G+R) x (G+R) uint8 matrix."""
    p = Problem(samples, heads, head_dim, flags=flags)
    if not 0 <= sample < len(p.samples):  # the library rejects it too; no buffer to size here
        _check(lib().sra_dense_mask(p.ptr, sample, None))
    g = p.samples[sample]
    n = g.gen_frames * g.gen_h * g.gen_w + g.ref_frames * g.ref_h * g.ref_w
    out = np.zeros((n, n), dtype=np.uint8)
    _check(lib().sra_dense_mask(p.ptr, sample, out.ctypes.data_as(ctypes.c_void_p)))
    return out


def schedule_export(samples, which: int, heads=1, head_dim=128, flags=0):
    import numpy as np

    n_items, n_spans, _ = schedule_info(samples, which, heads, head_dim, flags)
    p = Problem(samples, heads, head_dim, flags=flags)
    items = np.zeros((n_items, 8), dtype=np.int32)
    spans = np.zeros((n_spans, 4), dtype=np.int32)
    _check(lib().sra_schedule_export(p.ptr, which, items.ctypes.data_as(ctypes.c_void_p), items.size,
                                     spans.ctypes.data_as(ctypes.c_void_p), spans.size))
    return items, spans


def release_caches() -> None:
    _check(lib().sra_release_caches())


KERNELS = {"forward": 0, "delta": 1, "dkdv": 2, "dq": 3, "fill": 4, "gather": 5, "scatter": 6}


def kernel_timing_enable(on: bool = True) -> None:
    """Brackets every kernel launch with hipEvents on its stream (and resets the totals)."""
    _check(lib().sra_kernel_timing_enable(1 if on else 0))


def kernel_timing() -> Dict[str, Tuple[float, int]]:
    """{kernel: (total ms, launches)} since timing was enabled (waits for the events)."""
    out = {}
    for name, k in KERNELS.items():
        ms, n = ctypes.c_double(0), ctypes.c_int64(0)
        _check(lib().sra_kernel_timing(k, ctypes.byref(ms), ctypes.byref(n)))
        out[name] = (float(ms.value), int(n.value))
    return out


# ----------------------------------------------------------------------------- device calls
def _stream_ptr(device):
    """The current HIP stream of `device` (torch's, as a raw pointer)."""
    torch = _tm()
    raw = getattr(torch._C, "_cuda_getCurrentRawStream", None)
    if raw is not None:
        return ctypes.c_void_p(raw(device.index))
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None and t.numel() > 0 else ctypes.c_void_p(0)


def _token_stride(ts, name):
    s0 = None
    for t in ts:
        if t is None or t.numel() == 0:
            continue
        st = t.stride()
        if len(st) != 3 or st[2] != 1 or st[1] != t.shape[2]:
            raise ValueError(f"{name}: tensors must be [tokens, heads, head_dim] with contiguous heads")
        if s0 is None:
            s0 = st[0]
        elif st[0] != s0:
            raise ValueError(f"{name}: q, k and v must share one token stride")
    return 0 if s0 is None else int(s0)


def cu_seqlens(samples) -> Tuple[np.ndarray, np.ndarray]:
    """Packed-row offsets of the samples in each stream: [0, n_0, n_0 + n_1, ...] (int64), as
    the geometry fixes them (tokens of a sample are packed back to back in sample order)."""
    g = [0]
    r = [0]
    for s in samples:
        g.append(g[-1] + s.gen_frames * s.gen_h * s.gen_w)
        r.append(r[-1] + s.ref_frames * s.ref_h * s.ref_w)
    return np.array(g, dtype=np.int64), np.array(r, dtype=np.int64)


def _check_cu_seqlens(samples, cu_gen, cu_ref):
    """Optional caller-supplied offsets (any sequence or tensor) must equal the geometry's."""
    if cu_gen is None and cu_ref is None:
        return
    want = cu_seqlens(samples)
    for name, got, w in (("cu_seqlens_gen", cu_gen, want[0]), ("cu_seqlens_ref", cu_ref, want[1])):
        if got is None:
            continue
        a = np.asarray(got.detach().cpu() if hasattr(got, "detach") else got).astype(np.int64).ravel()
        if not np.array_equal(a, w):
            raise SRAError(SRA_ERR_INVALID_ARGUMENT, f"{name} {a.tolist()} does not match the geometry {w.tolist()}")


def _bad(msg):
    return SRAError(SRA_ERR_INVALID_ARGUMENT, msg)


_torch = None


def _tm():
    """torch, imported on first use (the host-only hooks of this module do not need it)."""
    global _torch
    if _torch is None:
        import torch
        _torch = torch
    return _torch


def _expect(t, name, shape, dtype, dense):
    """Checks one tensor argument: dtype, exact shape and (dense) row-major layout. The q/k/v
    inputs (dense=False) need contiguous heads only; their token stride is checked separately."""
    if not isinstance(t, _tm().Tensor):
        raise _bad(f"{name} must be a torch tensor, got {type(t).__name__}")
    if t.dtype != dtype:
        raise _bad(f"{name}: dtype {t.dtype}, expected {dtype}")
    if t.shape != shape:
        raise _bad(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
    if dense:
        if not t.is_contiguous():
            raise _bad(f"{name} must be dense (contiguous)")
    elif t.numel():
        st = t.stride()
        if st[2] != 1 or (shape[1] > 1 and st[1] != shape[2]):
            raise _bad(f"{name} must be [tokens, heads, head_dim] with contiguous heads")


def _same_device(tensors, device):
    """Every tensor of the (name, tensor) pairs must live on `device`, a GPU."""
    if device.type != "cuda":
        raise _bad(f"tensors must be on a GPU (HIP device), got {device}")
    idx = device.index
    for name, t in tensors:
        if t is not None and (not t.is_cuda or t.get_device() != idx):
            raise _bad(f"{name} is on {t.device}, q_gen on {device}")


def _inputs(q_gen, k_gen, v_gen, q_ref, k_ref, v_ref, samples, gen_only):
    """Validates q/k/v of both streams against the geometry; returns (H, d, n_gen, n_ref)."""
    torch = _tm()
    if not isinstance(q_gen, torch.Tensor) or q_gen.dim() != 3:
        raise _bad("q_gen must be a [tokens, heads, head_dim] tensor")
    H, d = int(q_gen.shape[1]), int(q_gen.shape[2])
    n_gen = sum(s.gen_frames * s.gen_h * s.gen_w for s in samples)
    n_ref = sum(s.ref_frames * s.ref_h * s.ref_w for s in samples)
    bf = torch.bfloat16
    sg, sr = (n_gen, H, d), (n_ref, H, d)
    _expect(q_gen, "q_gen", sg, bf, False)
    _expect(k_gen, "k_gen", sg, bf, False)
    _expect(v_gen, "v_gen", sg, bf, False)
    for name, t in (("q_ref", q_ref), ("k_ref", k_ref), ("v_ref", v_ref)):
        if t is None and (n_ref == 0 or (gen_only and name == "q_ref")):
            continue
        _expect(t, name, sr, bf, False)
    return H, d, n_gen, n_ref


def _out(out, name, shape, dtype, device):
    """The caller's output buffer `name`, or a new one (allocated only when none was given).
    dtype, shape and layout of a given buffer were checked by _precheck_outs; its device is
    checked here."""
    t = out.get(name)
    if t is None:
        return _tm().empty(shape, dtype=dtype, device=device)
    _same_device(((name, t),), device)
    return t


def _precheck_outs(out, specs):
    """dtype, shape and layout of the caller's output buffers, before any device check."""
    for name, shape, dtype in specs:
        t = (out or {}).get(name)
        if t is not None:
            _expect(t, name, shape, dtype, True)


def _workspace(out, nbytes, device):
    """The caller's workspace (a uint8 tensor on the device, used when large enough) or a new one."""
    import torch

    ws = out.get("workspace")
    if ws is not None:
        if not isinstance(ws, torch.Tensor) or ws.dtype != torch.uint8 or not ws.is_contiguous():
            raise _bad("workspace must be a contiguous uint8 tensor")
        _same_device((("workspace", ws),), device)
        if ws.numel() >= nbytes:
            return ws
    return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)


def _forward_args(q_gen, k_gen, v_gen, q_ref, k_ref, v_ref, samples, scale, out, gen_queries_only,
                  cu_seqlens_gen, cu_seqlens_ref):
    """Checks the forward's arguments and builds the problem and the output tensors."""
    import torch

    _check_cu_seqlens(samples, cu_seqlens_gen, cu_seqlens_ref)
    go = bool(gen_queries_only)
    if go:
        q_ref = None
    H, d, n_gen, n_ref = _inputs(q_gen, k_gen, v_gen, q_ref, k_ref, v_ref, samples, go)
    _precheck_outs(out, [("o_gen", (n_gen, H, d), torch.bfloat16), ("lse_gen", (H, n_gen), torch.float32)] +
                   ([] if go else [("o_ref", (n_ref, H, d), torch.bfloat16), ("lse_ref", (H, n_ref), torch.float32)]))
    dev = q_gen.device
    _same_device((("q_gen", q_gen), ("k_gen", k_gen), ("v_gen", v_gen), ("q_ref", q_ref), ("k_ref", k_ref),
                  ("v_ref", v_ref)), dev)
    p = _problem(samples, H, d, scale, _token_stride([q_gen, k_gen, v_gen], "gen"),
                 _token_stride([q_ref, k_ref, v_ref], "ref"), FLAG_GEN_QUERIES_ONLY if go else 0)
    out = out or {}
    o_gen = _out(out, "o_gen", (n_gen, H, d), torch.bfloat16, dev)
    lse_gen = _out(out, "lse_gen", (H, n_gen), torch.float32, dev)
    if go:
        o_ref = lse_ref = None
    else:
        o_ref = _out(out, "o_ref", (n_ref, H, d), torch.bfloat16, dev)
        lse_ref = _out(out, "lse_ref", (H, n_ref), torch.float32, dev)
    return p, q_ref, o_gen, o_ref, lse_gen, lse_ref, out, dev


def forward(q_gen, k_gen, v_gen, q_ref, k_ref, v_ref, samples, scale: Optional[float] = None,
            out: Optional[Dict] = None, gen_queries_only: bool = False, cu_seqlens_gen=None, cu_seqlens_ref=None):
    """SRA forward on the GPU. Returns (o_gen, o_ref, lse_gen, lse_ref).

    Inputs are bf16 [tokens, heads, head_dim] with contiguous heads (q, k and v of a stream
    share one token stride). `out` may hold caller buffers o_gen, o_ref (bf16, dense), lse_gen,
    lse_ref (fp32 [heads, tokens], dense) and workspace (uint8); every tensor must be on
    q_gen's GPU. A wrong dtype, shape, layout or device raises SRAError
    (SRA_ERR_INVALID_ARGUMENT) before anything reaches the library.
    gen_queries_only: the reference tokens are context only (cached reference K/V); only the
    generation rows are computed, q_ref may be None and o_ref / lse_ref are returned as None.
    cu_seqlens_gen / cu_seqlens_ref: optional packed-row offsets of the samples; they are
    checked against the geometry (SRAError with SRA_ERR_INVALID_ARGUMENT on a mismatch).
    """
    p, q_ref, o_gen, o_ref, lse_gen, lse_ref, out, dev = _forward_args(
        q_gen, k_gen, v_gen, q_ref, k_ref, v_ref, samples, scale, out, gen_queries_only, cu_seqlens_gen,
        cu_seqlens_ref)
    ws = _workspace(out, p.workspace_size(False), dev)
    _check(lib().sra_forward(p.ptr, _ptr(q_gen), _ptr(k_gen), _ptr(v_gen), _ptr(q_ref), _ptr(k_ref),
                             _ptr(v_ref), _ptr(o_gen), _ptr(o_ref), _ptr(lse_gen), _ptr(lse_ref),
                             _ptr(ws), ctypes.c_size_t(ws.numel()), _stream_ptr(dev)))
    return o_gen, o_ref, lse_gen, lse_ref


def forward_noalloc(q_gen, k_gen, v_gen, q_ref, k_ref, v_ref, samples, scale: Optional[float] = None,
                    out: Optional[Dict] = None, gen_queries_only: bool = False):
    """sra_forward_noalloc: the forward with the library's static device scratch as its
    workspace. With every output in `out` the call allocates nothing on the device (no torch
    allocation either). Same arguments and results as forward (a workspace in `out` is
    ignored); problems whose workspace exceeds noalloc_workspace_max() raise SRAError."""
    p, q_ref, o_gen, o_ref, lse_gen, lse_ref, out, dev = _forward_args(
        q_gen, k_gen, v_gen, q_ref, k_ref, v_ref, samples, scale, out, gen_queries_only, None, None)
    _check(lib().sra_forward_noalloc(p.ptr, _ptr(q_gen), _ptr(k_gen), _ptr(v_gen), _ptr(q_ref), _ptr(k_ref),
                                     _ptr(v_ref), _ptr(o_gen), _ptr(o_ref), _ptr(lse_gen), _ptr(lse_ref),
                                     _stream_ptr(dev)))
    return o_gen, o_ref, lse_gen, lse_ref


def noalloc_workspace_max() -> int:
    """SRA_NOALLOC_WORKSPACE_MAX of include/sra.h (bytes)."""
    m = re.search(r"#define\s+SRA_NOALLOC_WORKSPACE_MAX\s+\((\d+)u\s*<<\s*(\d+)\)", open(HEADER_PATH).read())
    return int(m.group(1)) << int(m.group(2))


def backward(q_gen, k_gen, v_gen, q_ref, k_ref, v_ref, o_gen, o_ref, lse_gen, lse_ref, do_gen, do_ref,
             samples, scale: Optional[float] = None, out: Optional[Dict] = None, gen_queries_only: bool = False,
             cu_seqlens_gen=None, cu_seqlens_ref=None):
    """SRA backward on the GPU. Returns dict dq_gen, dk_gen, dv_gen, dq_ref, dk_ref, dv_ref.

    q/k/v as for forward; o and do are bf16 [tokens, heads, head_dim] and lse fp32
    [heads, tokens], all dense. `out` may hold caller buffers for the six gradients (bf16,
    dense) and the workspace; every tensor must be on q_gen's GPU (SRAError otherwise).
    gen_queries_only: gradients of the generation rows alone (reference tokens are context
    only); q_ref, o_ref, lse_ref and do_ref may be None and dq_ref is returned as None.
    cu_seqlens_gen / cu_seqlens_ref: as for forward.
    """
    import torch

    _check_cu_seqlens(samples, cu_seqlens_gen, cu_seqlens_ref)
    go = bool(gen_queries_only)
    if go:
        q_ref = o_ref = lse_ref = do_ref = None
    H, d, n_gen, n_ref = _inputs(q_gen, k_gen, v_gen, q_ref, k_ref, v_ref, samples, go)
    _expect(o_gen, "o_gen", (n_gen, H, d), torch.bfloat16, True)
    _expect(do_gen, "do_gen", (n_gen, H, d), torch.bfloat16, True)
    _expect(lse_gen, "lse_gen", (H, n_gen), torch.float32, True)
    if not go:
        for name, t, shape, dt in (("o_ref", o_ref, (n_ref, H, d), torch.bfloat16),
                                   ("do_ref", do_ref, (n_ref, H, d), torch.bfloat16),
                                   ("lse_ref", lse_ref, (H, n_ref), torch.float32)):
            if t is None and n_ref == 0:
                continue
            _expect(t, name, shape, dt, True)
    _precheck_outs(out, [(n, (n_gen, H, d), torch.bfloat16) for n in ("dq_gen", "dk_gen", "dv_gen")] +
                   [(n, (n_ref, H, d), torch.bfloat16) for n in ("dq_ref", "dk_ref", "dv_ref")
                    if not (go and n == "dq_ref")])
    dev = q_gen.device
    _same_device((("q_gen", q_gen), ("k_gen", k_gen), ("v_gen", v_gen), ("q_ref", q_ref), ("k_ref", k_ref),
                  ("v_ref", v_ref), ("o_gen", o_gen), ("o_ref", o_ref), ("lse_gen", lse_gen), ("lse_ref", lse_ref),
                  ("do_gen", do_gen), ("do_ref", do_ref)), dev)
    p = _problem(samples, H, d, scale, _token_stride([q_gen, k_gen, v_gen], "gen"),
                 _token_stride([q_ref, k_ref, v_ref], "ref"), FLAG_GEN_QUERIES_ONLY if go else 0)
    out = out or {}
    g = {}
    for n in ("dq_gen", "dk_gen", "dv_gen"):
        g[n] = _out(out, n, (n_gen, H, d), torch.bfloat16, dev)
    for n in ("dq_ref", "dk_ref", "dv_ref"):
        g[n] = None if (go and n == "dq_ref") else _out(out, n, (n_ref, H, d), torch.bfloat16, dev)
    ws = _workspace(out, p.workspace_size(True), dev)
    _check(lib().sra_backward(p.ptr, _ptr(q_gen), _ptr(k_gen), _ptr(v_gen), _ptr(q_ref), _ptr(k_ref),
                              _ptr(v_ref), _ptr(o_gen), _ptr(o_ref), _ptr(lse_gen), _ptr(lse_ref),
                              _ptr(do_gen), _ptr(do_ref), _ptr(g["dq_gen"]), _ptr(g["dk_gen"]),
                              _ptr(g["dv_gen"]), _ptr(g["dq_ref"]), _ptr(g["dk_ref"]), _ptr(g["dv_ref"]),
                              _ptr(ws), ctypes.c_size_t(ws.numel()), _stream_ptr(dev)))
    return g


def useful_flops(samples, heads: int, head_dim: int) -> Tuple[int, int]:
    """Useful FLOP of one forward and one backward call: 4 d and 10 d per visible pair per head."""
    gp, rp = pair_counts(samples, heads, head_dim)
    pairs = (gp + rp) * heads
    return 4 * head_dim * pairs, 10 * head_dim * pairs


def default_scale(head_dim: int) -> float:
    return 1.0 / math.sqrt(head_dim)
