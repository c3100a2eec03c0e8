"""Python binding of libbevpool.so (the C ABI declared in include/bevpool.h).

The functions named ``bevpool_*`` mirror the C entry points one to one and
only marshal arguments: tensors become device pointers, the shape becomes a
``bevpool_shape`` struct and the current HIP stream is passed along.  The
lower-case helpers (``prepare``, ``forward``, ``backward``) additionally
allocate the output tensors with PyTorch.  Every step of the computation runs
in the library's HIP kernels; if the library cannot be loaded, every call
raises.
"""

from __future__ import annotations

import ctypes
import os
import re
from dataclasses import dataclass

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libbevpool.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "bevpool.h")

BEVPOOL_F32 = 0
BEVPOOL_F16 = 1
NOALLOC_SCRATCH_BYTES = 32 << 20  # BEVPOOL_NOALLOC_SCRATCH_BYTES
# status codes (enum bevpool_status)
BEVPOOL_OK, BEVPOOL_EINVAL, BEVPOOL_EOVERFLOW, BEVPOOL_EDTYPE, BEVPOOL_EWORKSPACE, BEVPOOL_ELAUNCH = \
    0, -1, -2, -3, -4, -5

_DTYPE_CODE = {torch.float32: BEVPOOL_F32, torch.float16: BEVPOOL_F16}
_CODE_DTYPE = {BEVPOOL_F32: torch.float32, BEVPOOL_F16: torch.float16}


class BevpoolError(RuntimeError):
    def __init__(self, status: int, func: str, message: str):
        super().__init__(f"{func} failed with status {status}: {message}")
        self.status = status


class bevpool_shape(ctypes.Structure):
    _fields_ = [(k, ctypes.c_int32) for k in ("B", "N", "D", "H", "W", "C", "X", "Y", "Z")]


class bevpool_frustum(ctypes.Structure):
    _fields_ = [("stride", ctypes.c_double), ("depth_start", ctypes.c_double), ("depth_step", ctypes.c_double),
                ("lo", ctypes.c_double * 3), ("res", ctypes.c_double * 3)]


CAMERA_WORDS = 16  # BEVPOOL_CAMERA_WORDS


def make_frustum(params: dict) -> bevpool_frustum:
    """bevpool_frustum from a dict with stride, depth_start, depth_step, lo (3), res (3)."""
    f = bevpool_frustum()
    f.stride, f.depth_start, f.depth_step = (float(params[k]) for k in ("stride", "depth_start", "depth_step"))
    for i in range(3):
        f.lo[i] = float(params["lo"][i])
        f.res[i] = float(params["res"][i])
    return f


_lib = None


def load_library(path: str | None = None) -> ctypes.CDLL:
    """Load libbevpool.so (raises if it has not been built)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    # (BEVPOOL_LIBRARY names another build of the same ABI, e.g. the
    # host-sanitizer build the ABI tests run against)
    p = path or os.environ.get("BEVPOOL_LIBRARY") or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} not found: build it with paper_2211_17111_amd.build.build()")
    lib = ctypes.CDLL(p)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    shp = ctypes.POINTER(bevpool_shape)
    lib.bevpool_version.restype = ctypes.c_int
    lib.bevpool_version.argtypes = []
    lib.bevpool_strerror.restype = ctypes.c_char_p
    lib.bevpool_strerror.argtypes = [ctypes.c_int]
    lib.bevpool_last_error.restype = ctypes.c_char_p
    lib.bevpool_last_error.argtypes = []
    lib.bevpool_prepare_workspace_size.restype = ctypes.c_int
    lib.bevpool_prepare_workspace_size.argtypes = [shp, ctypes.POINTER(sz)]
    lib.bevpool_prepare.restype = ctypes.c_int
    lib.bevpool_prepare.argtypes = [shp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.bevpool_forward.restype = ctypes.c_int
    lib.bevpool_forward_workspace_size.restype = ctypes.c_int
    lib.bevpool_forward_workspace_size.argtypes = [shp, ctypes.POINTER(sz)]
    lib.bevpool_forward.argtypes = [shp, ctypes.c_int, ctypes.c_int, vp, vp, vp, vp, vp, vp, vp,
                                    i32, i32, vp, vp, sz, vp]
    lib.bevpool_schedule_size.restype = ctypes.c_int
    lib.bevpool_schedule_size.argtypes = [shp, i32, i32, ctypes.POINTER(sz), ctypes.POINTER(sz)]
    lib.bevpool_schedule.restype = ctypes.c_int
    lib.bevpool_schedule.argtypes = [shp, vp, vp, i32, i32, vp, sz, vp, sz, vp]
    lib.bevpool_forward_scheduled.restype = ctypes.c_int
    lib.bevpool_forward_scheduled_workspace_size.restype = ctypes.c_int
    lib.bevpool_forward_scheduled_workspace_size.argtypes = [shp, i32, ctypes.POINTER(sz)]
    lib.bevpool_forward_scheduled.argtypes = [shp, ctypes.c_int, ctypes.c_int, vp, vp, vp, sz, i32, i32,
                                              i32, vp, vp, sz, vp]
    lib.bevpool_geometry.restype = ctypes.c_int
    lib.bevpool_geometry.argtypes = [shp, ctypes.POINTER(bevpool_frustum), vp, vp, vp]
    lib.bevpool_depth_lse.restype = ctypes.c_int
    lib.bevpool_depth_lse.argtypes = [shp, ctypes.c_int, vp, vp, vp]
    lib.bevpool_forward_scheduled_softmax.restype = ctypes.c_int
    lib.bevpool_forward_scheduled_softmax.argtypes = [shp, ctypes.c_int, ctypes.c_int, vp, vp, vp, vp, sz, i32,
                                                      i32, i32, vp, vp, sz, vp]
    lib.bevpool_forward_scheduled_noalloc.restype = ctypes.c_int
    lib.bevpool_forward_scheduled_noalloc.argtypes = [shp, ctypes.c_int, ctypes.c_int, vp, vp, vp, sz, i32,
                                                      i32, i32, vp, vp]
    lib.bevpool_backward_workspace_size.restype = ctypes.c_int
    lib.bevpool_backward_workspace_size.argtypes = [shp, ctypes.POINTER(sz)]
    lib.bevpool_backward.restype = ctypes.c_int
    lib.bevpool_backward.argtypes = [shp, ctypes.c_int, ctypes.c_int, vp, vp, vp, vp, vp, i32,
                                     vp, vp, vp, sz, vp]
    lib.bevpool_backward_scheduled.restype = ctypes.c_int
    lib.bevpool_backward_scheduled.argtypes = [shp, ctypes.c_int, ctypes.c_int, vp, vp, vp, vp, sz,
                                               i32, i32, vp, vp, vp]
    if path is None:
        _lib = lib
    return lib


def declared_symbols(header: str = HEADER_PATH) -> list[str]:
    """Names of the functions declared in include/bevpool.h."""
    with open(header) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bevpool_\w+)\s*\(", text)))


# ----------------------------------------------------------------- marshalling

def make_shape(shape) -> bevpool_shape:
    if isinstance(shape, bevpool_shape):
        return shape
    get = (lambda k: shape[k]) if isinstance(shape, dict) else (lambda k: getattr(shape, k))
    return bevpool_shape(*(int(get(k)) for k in ("B", "N", "D", "H", "W", "C", "X", "Y", "Z")))


def _ptr(x) -> int | None:
    if x is None:
        return None
    if isinstance(x, torch.Tensor):
        return x.data_ptr()
    return int(x)


def _stream(stream) -> int | None:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else None
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _check(lib, status: int, func: str):
    if status != 0:
        msg = lib.bevpool_last_error().decode() or lib.bevpool_strerror(status).decode()
        raise BevpoolError(status, func, msg)


def bevpool_version() -> int:
    return load_library().bevpool_version()


def bevpool_strerror(status: int) -> str:
    return load_library().bevpool_strerror(status).decode()


def bevpool_last_error() -> str:
    return load_library().bevpool_last_error().decode()


def bevpool_prepare_workspace_size(shape) -> int:
    lib = load_library()
    n = ctypes.c_size_t(0)
    _check(lib, lib.bevpool_prepare_workspace_size(ctypes.byref(make_shape(shape)), ctypes.byref(n)),
           "bevpool_prepare_workspace_size")
    return n.value


def bevpool_prepare(shape, coor, ranks_depth, ranks_feat, ranks_bev, interval_starts,
                    interval_lengths, counts, workspace, workspace_bytes, stream=None) -> None:
    lib = load_library()
    s = make_shape(shape)
    _check(lib, lib.bevpool_prepare(ctypes.byref(s), _ptr(coor), _ptr(ranks_depth), _ptr(ranks_feat),
                                    _ptr(ranks_bev), _ptr(interval_starts), _ptr(interval_lengths),
                                    _ptr(counts), _ptr(workspace), int(workspace_bytes),
                                    _stream(stream)),
           "bevpool_prepare")


def bevpool_forward_workspace_size(shape) -> int:
    lib = load_library()
    n = ctypes.c_size_t(0)
    _check(lib, lib.bevpool_forward_workspace_size(ctypes.byref(make_shape(shape)), ctypes.byref(n)),
           "bevpool_forward_workspace_size")
    return n.value


def bevpool_forward(shape, in_dtype, out_dtype, depth, feat, ranks_depth, ranks_feat, ranks_bev,
                    interval_starts, interval_lengths, n_valid, n_intervals, out, workspace,
                    workspace_bytes, stream=None) -> None:
    lib = load_library()
    s = make_shape(shape)
    _check(lib, lib.bevpool_forward(ctypes.byref(s), int(in_dtype), int(out_dtype), _ptr(depth),
                                    _ptr(feat), _ptr(ranks_depth), _ptr(ranks_feat), _ptr(ranks_bev),
                                    _ptr(interval_starts), _ptr(interval_lengths), int(n_valid),
                                    int(n_intervals), _ptr(out), _ptr(workspace), int(workspace_bytes),
                                    _stream(stream)),
           "bevpool_forward")


def bevpool_schedule_size(shape, n_valid, n_intervals) -> tuple[int, int]:
    lib = load_library()
    a, b = ctypes.c_size_t(0), ctypes.c_size_t(0)
    _check(lib, lib.bevpool_schedule_size(ctypes.byref(make_shape(shape)), int(n_valid), int(n_intervals),
                                          ctypes.byref(a), ctypes.byref(b)),
           "bevpool_schedule_size")
    return a.value, b.value


def bevpool_schedule(shape, ranks_depth, ranks_bev, n_valid, n_intervals, schedule, schedule_bytes,
                     workspace, workspace_bytes, stream=None) -> None:
    lib = load_library()
    s = make_shape(shape)
    _check(lib, lib.bevpool_schedule(ctypes.byref(s), _ptr(ranks_depth), _ptr(ranks_bev), int(n_valid),
                                     int(n_intervals), _ptr(schedule), int(schedule_bytes),
                                     _ptr(workspace), int(workspace_bytes), _stream(stream)),
           "bevpool_schedule")


def bevpool_forward_scheduled_workspace_size(shape, n_slots) -> int:
    lib = load_library()
    n = ctypes.c_size_t(0)
    _check(lib, lib.bevpool_forward_scheduled_workspace_size(ctypes.byref(make_shape(shape)),
                                                             int(n_slots), ctypes.byref(n)),
           "bevpool_forward_scheduled_workspace_size")
    return n.value


def bevpool_forward_scheduled(shape, in_dtype, out_dtype, depth, feat, schedule, schedule_bytes,
                              n_valid, n_intervals, n_slots, out, workspace, workspace_bytes,
                              stream=None) -> None:
    lib = load_library()
    s = make_shape(shape)
    _check(lib, lib.bevpool_forward_scheduled(ctypes.byref(s), int(in_dtype), int(out_dtype), _ptr(depth),
                                              _ptr(feat), _ptr(schedule), int(schedule_bytes),
                                              int(n_valid), int(n_intervals), int(n_slots), _ptr(out),
                                              _ptr(workspace), int(workspace_bytes), _stream(stream)),
           "bevpool_forward_scheduled")


def bevpool_geometry(shape, frustum, cams, coor, stream=None) -> None:
    lib = load_library()
    s = make_shape(shape)
    f = frustum if isinstance(frustum, bevpool_frustum) else make_frustum(frustum)
    _check(lib, lib.bevpool_geometry(ctypes.byref(s), ctypes.byref(f), _ptr(cams), _ptr(coor), _stream(stream)),
           "bevpool_geometry")


def geometry(cams: torch.Tensor, params: dict, shape, stream=None) -> torch.Tensor:
    """Voxel index (P, 3) int32 of every frustum point from cameras (B, N, 16)
    float64 on the device."""
    sd = _shape_dict(shape)
    _require(cams, "cams", torch.float64)
    if tuple(cams.shape) != (sd["B"], sd["N"], CAMERA_WORDS):
        raise ValueError(f"cams shape {tuple(cams.shape)} is not (B, N, {CAMERA_WORDS})")
    P = sd["B"] * sd["N"] * sd["D"] * sd["H"] * sd["W"]
    coor = torch.empty((P, 3), dtype=torch.int32, device=cams.device)
    bevpool_geometry(sd, params, cams, coor, stream)
    return coor


def bevpool_depth_lse(shape, in_dtype, logits, lse, stream=None) -> None:
    lib = load_library()
    s = make_shape(shape)
    _check(lib, lib.bevpool_depth_lse(ctypes.byref(s), int(in_dtype), _ptr(logits), _ptr(lse), _stream(stream)),
           "bevpool_depth_lse")


def bevpool_forward_scheduled_softmax(shape, in_dtype, out_dtype, logits, lse, feat, schedule, schedule_bytes,
                                      n_valid, n_intervals, n_slots, out, workspace, workspace_bytes,
                                      stream=None) -> None:
    lib = load_library()
    s = make_shape(shape)
    _check(lib, lib.bevpool_forward_scheduled_softmax(ctypes.byref(s), int(in_dtype), int(out_dtype),
                                                      _ptr(logits), _ptr(lse), _ptr(feat), _ptr(schedule),
                                                      int(schedule_bytes), int(n_valid), int(n_intervals),
                                                      int(n_slots), _ptr(out), _ptr(workspace),
                                                      int(workspace_bytes), _stream(stream)),
           "bevpool_forward_scheduled_softmax")


def bevpool_forward_scheduled_noalloc(shape, in_dtype, out_dtype, depth, feat, schedule, schedule_bytes,
                                      n_valid, n_intervals, n_slots, out, stream=None) -> None:
    lib = load_library()
    s = make_shape(shape)
    _check(lib, lib.bevpool_forward_scheduled_noalloc(ctypes.byref(s), int(in_dtype), int(out_dtype),
                                                      _ptr(depth), _ptr(feat), _ptr(schedule),
                                                      int(schedule_bytes), int(n_valid), int(n_intervals),
                                                      int(n_slots), _ptr(out), _stream(stream)),
           "bevpool_forward_scheduled_noalloc")


def bevpool_backward_workspace_size(shape) -> int:
    lib = load_library()
    n = ctypes.c_size_t(0)
    _check(lib, lib.bevpool_backward_workspace_size(ctypes.byref(make_shape(shape)), ctypes.byref(n)),
           "bevpool_backward_workspace_size")
    return n.value


def bevpool_backward(shape, in_dtype, out_dtype, grad_out, depth, feat, ranks_depth, ranks_bev,
                     n_valid, grad_depth, grad_feat, workspace, workspace_bytes, stream=None) -> None:
    lib = load_library()
    s = make_shape(shape)
    _check(lib, lib.bevpool_backward(ctypes.byref(s), int(in_dtype), int(out_dtype), _ptr(grad_out),
                                     _ptr(depth), _ptr(feat), _ptr(ranks_depth), _ptr(ranks_bev),
                                     int(n_valid), _ptr(grad_depth), _ptr(grad_feat),
                                     _ptr(workspace), int(workspace_bytes), _stream(stream)),
           "bevpool_backward")


def bevpool_backward_scheduled(shape, in_dtype, out_dtype, grad_out, depth, feat, schedule,
                               schedule_bytes, n_valid, n_intervals, grad_depth, grad_feat,
                               stream=None) -> None:
    lib = load_library()
    s = make_shape(shape)
    _check(lib, lib.bevpool_backward_scheduled(ctypes.byref(s), int(in_dtype), int(out_dtype),
                                               _ptr(grad_out), _ptr(depth), _ptr(feat),
                                               _ptr(schedule), int(schedule_bytes), int(n_valid),
                                               int(n_intervals), _ptr(grad_depth), _ptr(grad_feat),
                                               _stream(stream)),
           "bevpool_backward_scheduled")


# ------------------------------------------------------------ allocating helpers

@dataclass
class Plan:
    """Output of prepare: the sorted ranks and the interval table."""
    shape: dict
    ranks_depth: torch.Tensor
    ranks_feat: torch.Tensor
    ranks_bev: torch.Tensor
    interval_starts: torch.Tensor
    interval_lengths: torch.Tensor
    n_valid: int
    n_intervals: int


def _shape_dict(shape) -> dict:
    s = make_shape(shape)
    return {k: getattr(s, k) for k in ("B", "N", "D", "H", "W", "C", "X", "Y", "Z")}


def _require(t: torch.Tensor, name: str, dtype=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")


def prepare(coor: torch.Tensor, shape, stream=None) -> Plan:
    """Filter, sort and find intervals on the GPU; reads the two counts back."""
    sd = _shape_dict(shape)
    _require(coor, "coor", torch.int32)
    P = sd["B"] * sd["N"] * sd["D"] * sd["H"] * sd["W"]
    if coor.shape != (P, 3):
        raise ValueError(f"coor must be ({P}, 3), got {tuple(coor.shape)}")
    cells = sd["B"] * sd["Z"] * sd["Y"] * sd["X"]
    dev = coor.device
    i32 = dict(dtype=torch.int32, device=dev)
    rd = torch.empty(P, **i32)
    rf = torch.empty(P, **i32)
    rb = torch.empty(P, **i32)
    cap = min(P, cells)
    st = torch.empty(cap, **i32)
    ln = torch.empty(cap, **i32)
    counts = torch.zeros(2, **i32)
    ws_bytes = bevpool_prepare_workspace_size(sd)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    bevpool_prepare(sd, coor, rd, rf, rb, st, ln, counts, ws, ws_bytes, stream)
    nv, ni = (int(v) for v in counts.cpu().tolist())
    return Plan(sd, rd[:nv], rf[:nv], rb[:nv], st[:ni], ln[:ni], nv, ni)


def forward(depth: torch.Tensor, feat: torch.Tensor, plan: Plan, out_dtype=None,
            out: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
            stream=None) -> torch.Tensor:
    sd = plan.shape
    B, N, D, H, W, C, X, Y, Z = (sd[k] for k in ("B", "N", "D", "H", "W", "C", "X", "Y", "Z"))
    _require(depth, "depth")
    _require(feat, "feat", depth.dtype)
    if depth.dtype not in _DTYPE_CODE:
        raise ValueError(f"unsupported dtype {depth.dtype}")
    if tuple(depth.shape) != (B, N, D, H, W) or tuple(feat.shape) != (B, N, H, W, C):
        raise ValueError("depth/feat shapes do not match the plan")
    odt = out_dtype or depth.dtype
    if out is None:
        out = torch.empty((B, Z, Y, X, C), dtype=odt, device=depth.device)
    _require(out, "out", odt)
    if workspace is None:
        workspace = torch.empty(bevpool_forward_workspace_size(sd), dtype=torch.uint8, device=depth.device)
    bevpool_forward(sd, _DTYPE_CODE[depth.dtype], _DTYPE_CODE[odt], depth, feat, plan.ranks_depth,
                    plan.ranks_feat, plan.ranks_bev, plan.interval_starts, plan.interval_lengths,
                    plan.n_valid, plan.n_intervals, out, workspace,
                    workspace.numel() * workspace.element_size(), stream)
    return out


@dataclass
class Schedule:
    """Device buffer of a schedule built from a plan, with its header counts."""
    plan: Plan
    buffer: torch.Tensor
    counts: list[int]

    def header(self) -> list[int]:
        """The 16 header counts (pairs, items, segments, kept points, cells, cells found,
        empty cells, slots, ...), read back from the device."""
        return self.buffer[:64].view(torch.int32).cpu().tolist()

    @property
    def n_slots(self) -> int:
        return self.counts[7]


def schedule(plan: Plan, stream=None) -> Schedule:
    """Build the forward schedule of a plan on the GPU (checks its counts)."""
    sb, wb = bevpool_schedule_size(plan.shape, plan.n_valid, plan.n_intervals)
    dev = plan.ranks_depth.device
    buf = torch.empty(max(sb, 1), dtype=torch.uint8, device=dev)
    ws = torch.empty(max(wb, 1), dtype=torch.uint8, device=dev)
    bevpool_schedule(plan.shape, plan.ranks_depth, plan.ranks_bev, plan.n_valid, plan.n_intervals,
                     buf, sb, ws, wb, stream)
    sch = Schedule(plan, buf, [0] * 16)
    if plan.n_valid > 0:
        hdr = sch.header()  # synchronises with the build
        if hdr[3] != plan.n_valid or hdr[5] != plan.n_intervals:
            raise BevpoolError(-1, "bevpool_schedule", f"schedule counts {hdr} do not match the plan")
        sch.counts = hdr
    return sch


def forward_scheduled_workspace(sched: Schedule) -> torch.Tensor:
    """Workspace for forward_scheduled: one float32 row of C per slot of the schedule."""
    n = bevpool_forward_scheduled_workspace_size(sched.plan.shape, sched.n_slots)
    return torch.empty(max(n, 16), dtype=torch.uint8, device=sched.buffer.device)


def forward_scheduled(depth: torch.Tensor, feat: torch.Tensor, sched: Schedule, out_dtype=None,
                      out: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                      stream=None) -> torch.Tensor:
    plan = sched.plan
    sd = plan.shape
    B, N, D, H, W, C, X, Y, Z = (sd[k] for k in ("B", "N", "D", "H", "W", "C", "X", "Y", "Z"))
    _require(depth, "depth")
    _require(feat, "feat", depth.dtype)
    if tuple(depth.shape) != (B, N, D, H, W) or tuple(feat.shape) != (B, N, H, W, C):
        raise ValueError("depth/feat shapes do not match the plan")
    odt = out_dtype or depth.dtype
    if out is None:
        out = torch.empty((B, Z, Y, X, C), dtype=odt, device=depth.device)
    _require(out, "out", odt)
    if workspace is None:
        workspace = forward_scheduled_workspace(sched)
    bevpool_forward_scheduled(sd, _DTYPE_CODE[depth.dtype], _DTYPE_CODE[odt], depth, feat, sched.buffer,
                              sched.buffer.numel(), plan.n_valid, plan.n_intervals, sched.n_slots, out,
                              workspace, workspace.numel() * workspace.element_size(), stream)
    return out


def depth_lse(logits: torch.Tensor, shape, stream=None) -> torch.Tensor:
    """Per-pixel log-sum-exp over the depth bins of logits (B, N, D, H, W):
    float64 (B, N, H, W)."""
    sd = _shape_dict(shape)
    B, N, D, H, W = (sd[k] for k in ("B", "N", "D", "H", "W"))
    _require(logits, "logits")
    if tuple(logits.shape) != (B, N, D, H, W):
        raise ValueError(f"logits shape {tuple(logits.shape)} is not (B, N, D, H, W) = {(B, N, D, H, W)}")
    lse = torch.empty((B, N, H, W), dtype=torch.float64, device=logits.device)
    bevpool_depth_lse(sd, _DTYPE_CODE[logits.dtype], logits, lse, stream)
    return lse


def forward_scheduled_softmax(logits: torch.Tensor, feat: torch.Tensor, sched: Schedule,
                              lse: torch.Tensor | None = None, out_dtype=None,
                              out: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                              stream=None) -> torch.Tensor:
    """The scheduled forward with depth scores softmax(logits) over the depth
    bins, formed on the fly (lse from depth_lse when not given)."""
    plan = sched.plan
    sd = plan.shape
    B, N, D, H, W, C, X, Y, Z = (sd[k] for k in ("B", "N", "D", "H", "W", "C", "X", "Y", "Z"))
    _require(logits, "logits")
    _require(feat, "feat", logits.dtype)
    if tuple(logits.shape) != (B, N, D, H, W) or tuple(feat.shape) != (B, N, H, W, C):
        raise ValueError("logits/feat shapes do not match the plan")
    if lse is None:
        lse = depth_lse(logits, sd, stream)
    _require(lse, "lse", torch.float64)
    if tuple(lse.shape) != (B, N, H, W):
        raise ValueError(f"lse shape {tuple(lse.shape)} is not (B, N, H, W)")
    odt = out_dtype or logits.dtype
    if out is None:
        out = torch.empty((B, Z, Y, X, C), dtype=odt, device=logits.device)
    _require(out, "out", odt)
    if workspace is None:
        workspace = forward_scheduled_workspace(sched)
    bevpool_forward_scheduled_softmax(sd, _DTYPE_CODE[logits.dtype], _DTYPE_CODE[odt], logits, lse, feat,
                                      sched.buffer, sched.buffer.numel(), plan.n_valid, plan.n_intervals,
                                      sched.n_slots, out, workspace, workspace.numel() * workspace.element_size(),
                                      stream)
    return out


def _check_grad_inputs(grad_out: torch.Tensor, depth: torch.Tensor, feat: torch.Tensor, sd: dict):
    """grad_out must have out's shape (B, Z, Y, X, C) and a dtype the library
    accepts with depth's (float32 with float32; float16 or float32 with
    float16); depth and feat the plan's shapes."""
    B, N, D, H, W, C, X, Y, Z = (sd[k] for k in ("B", "N", "D", "H", "W", "C", "X", "Y", "Z"))
    _require(grad_out, "grad_out")
    _require(depth, "depth")
    _require(feat, "feat", depth.dtype)
    if depth.dtype not in _DTYPE_CODE or grad_out.dtype not in _DTYPE_CODE:
        raise ValueError(f"unsupported dtypes depth {depth.dtype}, grad_out {grad_out.dtype}")
    if depth.dtype == torch.float32 and grad_out.dtype != torch.float32:
        raise ValueError("float32 inputs need a float32 grad_out")
    if tuple(depth.shape) != (B, N, D, H, W) or tuple(feat.shape) != (B, N, H, W, C):
        raise ValueError("depth/feat shapes do not match the plan")
    if tuple(grad_out.shape) != (B, Z, Y, X, C):
        raise ValueError(f"grad_out must be {(B, Z, Y, X, C)}, got {tuple(grad_out.shape)}")


def backward(grad_out: torch.Tensor, depth: torch.Tensor, feat: torch.Tensor, plan: Plan,
             workspace: torch.Tensor | None = None, stream=None):
    sd = plan.shape
    _check_grad_inputs(grad_out, depth, feat, sd)
    gd = torch.empty_like(depth)
    gf = torch.empty_like(feat)
    ws_bytes = bevpool_backward_workspace_size(sd)
    if workspace is None:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=depth.device)
    bevpool_backward(sd, _DTYPE_CODE[depth.dtype], _DTYPE_CODE[grad_out.dtype], grad_out, depth, feat,
                     plan.ranks_depth, plan.ranks_bev, plan.n_valid, gd, gf, workspace,
                     workspace.numel() * workspace.element_size(), stream)
    return gd, gf


def backward_scheduled(grad_out: torch.Tensor, depth: torch.Tensor, feat: torch.Tensor,
                       sched: Schedule, stream=None):
    plan = sched.plan
    sd = plan.shape
    _check_grad_inputs(grad_out, depth, feat, sd)
    gd = torch.empty_like(depth)
    gf = torch.empty_like(feat)
    bevpool_backward_scheduled(sd, _DTYPE_CODE[depth.dtype], _DTYPE_CODE[grad_out.dtype], grad_out,
                               depth, feat, sched.buffer, sched.buffer.numel(), plan.n_valid,
                               plan.n_intervals, gd, gf, stream)
    return gd, gf


class BevPoolFunction(torch.autograd.Function):
    """Autograd wrapper: forward pools, backward returns grad_depth, grad_feat.
    Given a Schedule it runs the scheduled forward and backward, given a Plan
    the plan-only ones (same results within float32 rounding)."""

    @staticmethod
    def forward(ctx, depth, feat, plan, out_dtype=None):
        ctx.plan = plan
        ctx.save_for_backward(depth, feat)
        if isinstance(plan, Schedule):
            return forward_scheduled(depth, feat, plan, out_dtype)
        return forward(depth, feat, plan, out_dtype)

    @staticmethod
    def backward(ctx, grad_out):
        depth, feat = ctx.saved_tensors
        if isinstance(ctx.plan, Schedule):
            gd, gf = backward_scheduled(grad_out.contiguous(), depth, feat, ctx.plan)
        else:
            gd, gf = backward(grad_out.contiguous(), depth, feat, ctx.plan)
        return gd, gf, None, None


def bev_pool(depth, feat, plan, out_dtype=None):
    """Differentiable pooling of depth x feat into the BEV grid; `plan` is a
    Plan (from prepare) or a Schedule (from schedule, the faster paths)."""
    return BevPoolFunction.apply(depth, feat, plan, out_dtype)
