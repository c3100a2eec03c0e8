"""C-ABI contract of libbevpool.so, checked without a GPU.

Validation happens before any HIP call, so every documented error path can
be exercised here with dummy (never dereferenced) pointers.
"""

import ctypes

import pytest

from paper_2211_17111_amd import bevpool as bp

OK, EINVAL, EOVERFLOW, EDTYPE, EWORKSPACE, ELAUNCH = 0, -1, -2, -3, -4, -5


def test_status_constants_match_header():
    """The binding's status constants are the header's enum values."""
    import re
    src = open(bp.HEADER_PATH).read()
    enum = dict((m.group(1), int(m.group(2))) for m in re.finditer(r"(BEVPOOL_E?[A-Z]+) = (-?\d+)", src))
    for name in ("BEVPOOL_OK", "BEVPOOL_EINVAL", "BEVPOOL_EOVERFLOW", "BEVPOOL_EDTYPE", "BEVPOOL_EWORKSPACE",
                 "BEVPOOL_ELAUNCH"):
        assert getattr(bp, name) == enum[name], name
DUMMY = 0x1000  # non-NULL, never dereferenced: every call below fails validation first

SHAPE = dict(B=1, N=6, D=118, H=40, W=100, C=80, X=128, Y=128, Z=1)


@pytest.fixture(scope="module")
def lib():
    return bp.load_library()


def _shape(**kw):
    return bp.make_shape({**SHAPE, **kw})


def test_exports_every_declared_symbol(lib):
    names = bp.declared_symbols()
    assert set(names) == {
        "bevpool_version", "bevpool_strerror", "bevpool_last_error",
        "bevpool_prepare_workspace_size", "bevpool_prepare", "bevpool_forward",
        "bevpool_forward_workspace_size", "bevpool_schedule_size", "bevpool_schedule",
        "bevpool_forward_scheduled", "bevpool_forward_scheduled_workspace_size",
        "bevpool_forward_scheduled_noalloc", "bevpool_depth_lse", "bevpool_forward_scheduled_softmax",
        "bevpool_geometry",
        "bevpool_backward_workspace_size", "bevpool_backward", "bevpool_backward_scheduled",
    }
    for n in names:
        assert hasattr(lib, n), n


def test_version_and_strerror(lib):
    assert lib.bevpool_version() == 1
    for code in (OK, EINVAL, EOVERFLOW, EDTYPE, EWORKSPACE, ELAUNCH):
        assert lib.bevpool_strerror(code)
    assert lib.bevpool_strerror(12345) == b"unknown status"


def test_workspace_sizes(lib):
    s = _shape()
    n = ctypes.c_size_t()
    assert lib.bevpool_prepare_workspace_size(ctypes.byref(s), ctypes.byref(n)) == OK
    P = 6 * 118 * 40 * 100
    assert n.value >= 2 * 4 * P  # radix ping-pong buffers
    assert lib.bevpool_backward_workspace_size(ctypes.byref(s), ctypes.byref(n)) == OK
    assert n.value == 4 * P
    assert lib.bevpool_prepare_workspace_size(None, ctypes.byref(n)) == EINVAL
    assert lib.bevpool_prepare_workspace_size(ctypes.byref(s), None) == EINVAL


@pytest.mark.parametrize("dim", list("BNDHWCXYZ"))
def test_non_positive_dims_rejected(lib, dim):
    for v in (0, -3):
        s = _shape(**{dim: v})
        n = ctypes.c_size_t()
        assert lib.bevpool_prepare_workspace_size(ctypes.byref(s), ctypes.byref(n)) == EINVAL
        assert b"must be >= 1" in lib.bevpool_last_error()


def test_overflow_rejected(lib):
    n = ctypes.c_size_t()
    big = _shape(B=700)   # P = 1.98e9 < 2^31
    assert lib.bevpool_prepare_workspace_size(ctypes.byref(big), ctypes.byref(n)) == OK
    over = _shape(B=800)   # P = 2.27e9 >= 2^31
    assert lib.bevpool_prepare_workspace_size(ctypes.byref(over), ctypes.byref(n)) == EOVERFLOW
    wide = _shape(C=2048)
    assert lib.bevpool_prepare_workspace_size(ctypes.byref(wide), ctypes.byref(n)) == EOVERFLOW
    out_over = _shape(B=1, X=8192, Y=8192, Z=1, C=64)
    assert lib.bevpool_prepare_workspace_size(ctypes.byref(out_over), ctypes.byref(n)) == EOVERFLOW


def _fwd(lib, s, in_dt=0, out_dt=0, nv=100, ni=10, ptrs=None, out=DUMMY, ws=DUMMY, wsb=None):
    p = ptrs or [DUMMY] * 7
    if wsb is None:
        n = ctypes.c_size_t()
        lib.bevpool_forward_workspace_size(ctypes.byref(s), ctypes.byref(n))
        wsb = n.value
    return lib.bevpool_forward(ctypes.byref(s), in_dt, out_dt, *p, nv, ni, out, ws, wsb, None)


def test_forward_validation(lib):
    s = _shape()
    assert _fwd(lib, s, in_dt=2) == EDTYPE
    assert _fwd(lib, s, out_dt=7) == EDTYPE
    assert _fwd(lib, s, in_dt=0, out_dt=1) == EDTYPE   # f32 in, f16 out
    assert _fwd(lib, s, ni=-1) == EINVAL
    assert _fwd(lib, s, nv=10**6, ni=128 * 128 + 1) == EINVAL    # more intervals than cells
    assert _fwd(lib, s, nv=5, ni=6) == EINVAL          # more intervals than points
    assert _fwd(lib, s, nv=-1, ni=0) == EINVAL
    assert _fwd(lib, s, nv=6 * 118 * 40 * 100 + 1) == EINVAL
    assert _fwd(lib, s, out=None) == EINVAL
    for k in range(7):
        ptrs = [DUMMY] * 7
        ptrs[k] = None
        assert _fwd(lib, s, ptrs=ptrs) == EINVAL
        assert b"is NULL" in lib.bevpool_last_error()
    assert lib.bevpool_forward(None, 0, 0, *([DUMMY] * 7), 1, 1, DUMMY, DUMMY, 1 << 30, None) == EINVAL
    assert _fwd(lib, s, ws=None) == EWORKSPACE
    n = ctypes.c_size_t()
    assert lib.bevpool_forward_workspace_size(ctypes.byref(s), ctypes.byref(n)) == OK
    assert n.value > 0
    assert _fwd(lib, s, wsb=n.value - 1) == EWORKSPACE


def test_prepare_validation(lib):
    s = _shape()
    need = ctypes.c_size_t()
    lib.bevpool_prepare_workspace_size(ctypes.byref(s), ctypes.byref(need))
    args = [DUMMY] * 7
    assert lib.bevpool_prepare(ctypes.byref(s), *args, DUMMY, need.value - 1, None) == EWORKSPACE
    assert lib.bevpool_prepare(ctypes.byref(s), *args, None, need.value, None) == EWORKSPACE
    for k in range(7):
        a = [DUMMY] * 7
        a[k] = None
        assert lib.bevpool_prepare(ctypes.byref(s), *a, DUMMY, need.value, None) == EINVAL


def test_backward_validation(lib):
    s = _shape()
    need = ctypes.c_size_t()
    lib.bevpool_backward_workspace_size(ctypes.byref(s), ctypes.byref(need))
    def call(nv=5, ws=DUMMY, wsb=None, ptrs=None, in_dt=0, out_dt=0):
        p = ptrs or [DUMMY] * 7
        return lib.bevpool_backward(ctypes.byref(s), in_dt, out_dt, p[0], p[1], p[2], p[3], p[4],
                                    nv, p[5], p[6], ws, need.value if wsb is None else wsb, None)
    assert call(ws=None) == EWORKSPACE
    assert call(wsb=need.value - 4) == EWORKSPACE
    assert call(nv=-1) == EINVAL
    assert call(nv=6 * 118 * 40 * 100 + 1) == EINVAL
    assert call(in_dt=3) == EDTYPE
    for k in range(7):
        p = [DUMMY] * 7
        p[k] = None
        assert call(ptrs=p) == EINVAL


def test_binding_raises_with_message(lib):
    with pytest.raises(bp.BevpoolError) as ei:
        bp.bevpool_prepare_workspace_size(dict(SHAPE, C=0))
    assert ei.value.status == EINVAL and "C" in str(ei.value)


def test_schedule_validation(lib):
    s = _shape()
    sb, wb = ctypes.c_size_t(), ctypes.c_size_t()
    assert lib.bevpool_schedule_size(ctypes.byref(s), 1000, 100, ctypes.byref(sb), ctypes.byref(wb)) == OK
    assert sb.value > 4 * 1000 and wb.value > 4 * 4 * 1000
    assert lib.bevpool_schedule_size(ctypes.byref(s), -1, 0, ctypes.byref(sb), ctypes.byref(wb)) == EINVAL
    assert lib.bevpool_schedule_size(ctypes.byref(s), 10, 11, ctypes.byref(sb), ctypes.byref(wb)) == EINVAL
    assert lib.bevpool_schedule_size(ctypes.byref(s), 10, 0, ctypes.byref(sb), ctypes.byref(wb)) == EINVAL
    lib.bevpool_schedule_size(ctypes.byref(s), 1000, 100, ctypes.byref(sb), ctypes.byref(wb))
    call = lambda **k: lib.bevpool_schedule(ctypes.byref(s), k.get("rd", DUMMY), k.get("rb", DUMMY), 1000, 100,
                                            k.get("sc", DUMMY), k.get("sb", sb.value), k.get("ws", DUMMY),
                                            k.get("wb", wb.value), None)
    assert call(rd=None) == EINVAL
    assert call(sc=None) == EINVAL
    assert call(sb=sb.value - 1) == EINVAL
    assert call(ws=None) == EWORKSPACE
    assert call(wb=wb.value - 1) == EWORKSPACE
    need = 10 * s.C * 4  # ten slots
    f = lambda **k: lib.bevpool_forward_scheduled(ctypes.byref(s), k.get("i", 0), k.get("o", 0), DUMMY, DUMMY,
                                                  k.get("sc", DUMMY), k.get("sb", sb.value), 1000, 100,
                                                  k.get("ns", 10), k.get("out", DUMMY), k.get("ws", DUMMY),
                                                  k.get("wb", need), None)
    assert f(i=0, o=1) == EDTYPE
    assert f(sc=None) == EINVAL
    assert f(sb=16) == EINVAL
    assert f(out=None) == EINVAL
    # the slot count the caller read from the header sizes the workspace
    assert f(ns=-1) == EINVAL
    assert f(ns=1001) == EINVAL  # (more slots than kept points)
    assert f(ws=None) == EWORKSPACE
    assert f(wb=need - 1) == EWORKSPACE
    assert f(ns=11) == EWORKSPACE
    # the allocation-free forward: the same checks, and a bound on the slots
    g = lambda **k: lib.bevpool_forward_scheduled_noalloc(ctypes.byref(s), k.get("i", 0), k.get("o", 0), DUMMY,
                                                          DUMMY, k.get("sc", DUMMY), k.get("sb", sb.value),
                                                          1000, 100, k.get("ns", 10), k.get("out", DUMMY),
                                                          None)
    assert g(i=0, o=1) == EDTYPE
    assert g(sc=None) == EINVAL
    assert g(sb=16) == EINVAL
    assert g(out=None) == EINVAL
    assert g(ns=-1) == EINVAL
    assert g(ns=1001) == EINVAL
    n = ctypes.c_size_t(0)
    assert lib.bevpool_forward_scheduled_workspace_size(ctypes.byref(s), 10, ctypes.byref(n)) == OK
    assert n.value == 10 * s.C * 4
    assert lib.bevpool_forward_scheduled_workspace_size(ctypes.byref(s), -1, ctypes.byref(n)) == EINVAL
    b = lambda **k: lib.bevpool_backward_scheduled(ctypes.byref(s), k.get("i", 0), k.get("o", 0),
                                                   k.get("g", DUMMY), DUMMY, DUMMY, k.get("sc", DUMMY),
                                                   k.get("sb", sb.value), 1000, 100, DUMMY,
                                                   k.get("gf", DUMMY), None)
    assert b(i=0, o=1) == EDTYPE
    assert b(g=None) == EINVAL
    assert b(sc=None) == EINVAL
    assert b(sb=16) == EINVAL
    assert b(gf=None) == EINVAL


def test_noalloc_scratch_bound():
    """The allocation-free forward refuses, before any HIP call, a schedule
    whose slots exceed its static array, and the binding's constant is the
    header's."""
    import re
    src = open(bp.HEADER_PATH).read()
    m = re.search(r"#define BEVPOOL_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", src)
    assert m and bp.NOALLOC_SCRATCH_BYTES == int(m.group(1)) << int(m.group(2))
    lib = bp.load_library()
    s = bp.make_shape(dict(B=1, N=1, D=64, H=16, W=16, C=1024, X=64, Y=64, Z=1))
    n_slots = bp.NOALLOC_SCRATCH_BYTES // (1024 * 4) + 1  # one slot more than fits
    st = lib.bevpool_forward_scheduled_noalloc(ctypes.byref(s), 0, 0, DUMMY, DUMMY, DUMMY, 1 << 40, 16384, 4096,
                                               n_slots, DUMMY, None)
    assert st == EWORKSPACE
    assert "allocation-free" in bp.bevpool_last_error()


def test_softmax_validation():
    """The fused softmax entry points check their arguments before any HIP
    call."""
    lib = bp.load_library()
    s = bp.make_shape(dict(B=1, N=2, D=8, H=4, W=8, C=16, X=16, Y=16, Z=1))
    lse = lambda **k: lib.bevpool_depth_lse(ctypes.byref(s), k.get("i", 0), k.get("x", DUMMY), k.get("l", DUMMY),
                                            None)
    assert lse(x=None) == EINVAL
    assert lse(l=None) == EINVAL
    assert lse(i=7) == EDTYPE
    sb, wb = ctypes.c_size_t(0), ctypes.c_size_t(0)
    assert lib.bevpool_schedule_size(ctypes.byref(s), 400, 100, ctypes.byref(sb), ctypes.byref(wb)) == OK
    f = lambda **k: lib.bevpool_forward_scheduled_softmax(
        ctypes.byref(s), k.get("i", 0), k.get("o", 0), k.get("x", DUMMY), k.get("l", DUMMY), DUMMY, DUMMY,
        sb.value, 400, 100, k.get("ns", 4), k.get("out", DUMMY), k.get("ws", DUMMY), k.get("wb", 4 * 16 * 4),
        None)
    assert f(i=0, o=1) == EDTYPE
    assert f(x=None) == EINVAL
    assert f(l=None) == EINVAL
    assert f(out=None) == EINVAL
    assert f(ns=401) == EINVAL
    assert f(ws=None) == EWORKSPACE
    assert f(wb=4 * 16 * 4 - 1) == EWORKSPACE


def test_geometry_validation():
    lib = bp.load_library()
    s = bp.make_shape(dict(B=1, N=2, D=8, H=4, W=8, C=16, X=16, Y=16, Z=1))
    good = dict(stride=16.0, depth_start=1.0, depth_step=1.0, lo=(-8.0, -8.0, -5.0), res=(1.0, 1.0, 8.0))

    def g(**k):
        f = bp.make_frustum(dict(good, **k.get("f", {})))
        return lib.bevpool_geometry(ctypes.byref(s), None if k.get("nof") else ctypes.byref(f),
                                    k.get("cams", DUMMY), k.get("coor", DUMMY), None)

    assert g(nof=True) == EINVAL
    assert g(cams=None) == EINVAL
    assert g(coor=None) == EINVAL
    assert g(f=dict(stride=0.0)) == EINVAL
    assert g(f=dict(depth_step=-1.0)) == EINVAL
    assert g(f=dict(res=(1.0, 0.0, 8.0))) == EINVAL
    assert g(f=dict(lo=(float("nan"), -8.0, -5.0))) == EINVAL
    assert g(f=dict(depth_start=float("inf"))) == EINVAL

