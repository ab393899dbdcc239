"""Python binding of the MI355X layout-transform library (``libcosta_mi355x.so``).

Argument marshalling only: every function calls the C ABI of
``include/costa.h`` with the same name; all work runs in the library's HIP
kernels and host planner.  Device buffers are passed as ``torch`` tensors (or
raw integer addresses); torch is used for nothing else, except that it is
imported before the library so that the process holds a single HIP runtime.
Importing this module fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("COSTA_LIB") or os.path.join(_HERE, "libcosta_mi355x.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                      "(or python paper_2106_06601_amd/build.py)")

# One HIP runtime per process.  PyTorch ships its own libamdhip64 and its
# libraries ask for it by a name that does not match the ROCm copy this
# library links; loaded first, the ROCm copy would leave two runtimes in the
# process, of which one sees no device.  With torch loaded first, this library
# binds to torch's runtime.
try:
    import torch  # noqa: F401
except ImportError:  # no torch: the ROCm runtime alone
    pass

_lib = ctypes.CDLL(LIB_PATH)

SUCCESS, INVALID_VALUE, SHAPE_MISMATCH, OUT_OF_MEMORY, DEVICE, NOT_SUPPORTED = range(6)
OPS = {"N": 0, "T": 1, "C": 2}
ORDERS = {"col": 0, "row": 1}
DTYPES = {"f64": 0, "c128": 1, "f32": 2, "c64": 3}
KERNELS = ["pack", "unpack", "direct", "volume"]

_i32, _i64, _vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
_P = ctypes.POINTER


class CostaDesc(ctypes.Structure):
    _fields_ = [("op", ctypes.c_int), ("alpha", _vp), ("beta", _vp), ("A", _vp), ("A_local", _vp),
                ("B", _vp), ("B_local", _vp)]


class CostaStats(ctypes.Structure):
    _fields_ = [("total_elems", _i64), ("local_elems", _i64), ("remote_elems", _i64), ("model_bytes", _i64),
                ("message_bytes", _i64), ("workspace_bytes", _i64), ("overlay_blocks", _i64),
                ("pack_bytes", _i64), ("unpack_bytes", _i64), ("direct_bytes", _i64), ("waves", _i32),
                ("pieces_pack", _i32), ("pieces_unpack", _i32), ("pieces_direct", _i32),
                ("plan_ms", ctypes.c_double)]


class CostaPieceInfo(ctypes.Structure):
    _fields_ = [("kind", _i32), ("wave", _i32), ("group", _i64), ("src_off", _i64), ("dst_off", _i64),
                ("src_ld", _i64), ("dst_ld", _i64), ("src_buf", _i32), ("dst_buf", _i32), ("nx", _i32),
                ("ny", _i32), ("item", _i32), ("flags", _i32), ("ntasks", _i64),
                ("tile_x", _i32), ("tile_y", _i32), ("launch", _i32), ("reserved", _i32),
                ("wide_group", _i64), ("wide_ntasks", _i64)]


class CostaGrid(ctypes.Structure):
    _fields_ = [("nprow", _i32), ("npcol", _i32), ("rank_order", ctypes.c_int), ("nranks", _i32),
                ("rank_map", _vp)]


class CostaTiming(ctypes.Structure):
    _fields_ = [("ms", ctypes.c_double * 4), ("launches", _i64 * 4), ("bytes", _i64 * 4)]


_SIGS = {
    "costa_layout_create": [_i64, _i64, _i32, _vp, _i32, _vp, _vp, _i32, ctypes.c_int, _vp, _vp, _P(_vp)],
    "costa_layout_create_block_cyclic": [_i64, _i64, _i64, _i64, _i32, _i32, ctypes.c_int, ctypes.c_int, _P(_vp)],
    "costa_layout_create_scalapack": [_vp, _P(CostaGrid), _P(_vp)],
    "costa_layout_submatrix": [_vp, _i64, _i64, _i64, _i64, _P(_vp)],
    "costa_pxgemr2d": [ctypes.c_int, _i32, _i32, _vp, _i32, _i32, _vp, _P(CostaGrid), _vp, _i32, _i32, _vp,
                       _P(CostaGrid), _vp],
    "costa_pxtran": [ctypes.c_int, ctypes.c_int, _i32, _i32, _vp, _vp, _i32, _i32, _vp, _P(CostaGrid), _vp, _vp,
                     _i32, _i32, _vp, _P(CostaGrid), _vp],
    "costa_pdgemr2d": [_i32, _i32, _vp, _i32, _i32, _vp, _P(CostaGrid), _vp, _i32, _i32, _vp, _P(CostaGrid), _vp],
    "costa_pdtran": [_i32, _i32, _vp, _vp, _i32, _i32, _vp, _P(CostaGrid), _vp, _vp, _i32, _i32, _vp,
                     _P(CostaGrid), _vp],
    "costa_pztranu": [_i32, _i32, _vp, _vp, _i32, _i32, _vp, _P(CostaGrid), _vp, _vp, _i32, _i32, _vp,
                      _P(CostaGrid), _vp],
    "costa_pztranc": [_i32, _i32, _vp, _vp, _i32, _i32, _vp, _P(CostaGrid), _vp, _vp, _i32, _i32, _vp,
                      _P(CostaGrid), _vp],
    "costa_layout_local_elems": [_vp, _i32, _P(_i64)],
    "costa_layout_block": [_vp, _i32, _i32, _P(_i32), _P(_i64), _P(_i64)],
    "costa_layout_info": [_vp, _P(_i64), _P(_i64), _P(_i32), _P(_i32), _P(_i32), _P(ctypes.c_int)],
    "costa_layout_destroy": [_vp],
    "costa_volume_matrix": [_vp, _vp, ctypes.c_int, _vp, _vp],
    "costa_relabel": [_i32, _vp, _vp, _P(_i64), _P(_i64)],
    "costa_relabel_cost": [_i32, _vp, ctypes.c_double, _vp, _vp, ctypes.c_int, _vp, _P(ctypes.c_double),
                           _P(ctypes.c_double)],
    "costa_transform": [ctypes.c_int, ctypes.c_int, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp],
    "costa_transform_batched": [ctypes.c_int, _i32, _vp, _vp, _vp],
    "costa_transform_batched_noalloc": [ctypes.c_int, _i32, _vp, _vp, _vp],
    "costa_set_workspace_limit": [ctypes.c_size_t],
    "costa_plan_stats": [ctypes.c_int, _i32, _vp, _vp, _P(CostaStats)],
    "costa_plan_export": [ctypes.c_int, _i32, _vp, _vp, _vp, _i64, _P(_i64)],
    "costa_timing_enable": [ctypes.c_int],
    "costa_timing_read": [_P(CostaTiming)],
    "costa_finalize": [],
}
for _name, _args in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = ctypes.c_int
_lib.costa_status_string.argtypes = [ctypes.c_int]
_lib.costa_status_string.restype = ctypes.c_char_p
_lib.costa_last_error.argtypes = []
_lib.costa_last_error.restype = ctypes.c_char_p


class CostaError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        detail = _lib.costa_last_error().decode()
        super().__init__(f"{where}: {_lib.costa_status_string(status).decode()} ({detail})")


def _check(status: int, where: str) -> None:
    if status != SUCCESS:
        raise CostaError(status, where)


def _addr(x) -> int:
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


def _stream(stream) -> int:
    if stream is None:
        import torch
        return int(torch.cuda.current_stream().cuda_stream) if torch.cuda.is_available() else 0
    if isinstance(stream, int):
        return stream
    return int(stream.cuda_stream)


def _np64(a) -> Optional[np.ndarray]:
    return None if a is None else np.ascontiguousarray(a, dtype=np.int64)


def _scalar(dtype: str, v):
    if dtype == "f64":
        return ctypes.c_double(float(v))
    if dtype == "f32":
        return ctypes.c_float(float(v))
    v = complex(v)
    if dtype == "c128":
        return (ctypes.c_double * 2)(v.real, v.imag)
    return (ctypes.c_float * 2)(v.real, v.imag)


# ---------------------------------------------------------------------------
# layouts
# ---------------------------------------------------------------------------
def costa_layout_create(nrows: int, ncols: int, row_splits, col_splits, owners, nranks: int,
                        block_order: str = "col", block_offset=None, block_ld=None) -> int:
    rs, cs = _np64(row_splits), _np64(col_splits)
    ow = np.ascontiguousarray(owners, dtype=np.int32)
    bo, bl = _np64(block_offset), _np64(block_ld)
    h = _vp()
    _check(_lib.costa_layout_create(nrows, ncols, len(rs) - 1, rs.ctypes.data, len(cs) - 1, cs.ctypes.data,
                                    ow.ctypes.data if ow.size else None, nranks, ORDERS[block_order],
                                    None if bo is None else bo.ctypes.data, None if bl is None else bl.ctypes.data,
                                    ctypes.byref(h)), "costa_layout_create")
    return h.value


def costa_layout_create_block_cyclic(nrows: int, ncols: int, mb: int, nb: int, prow: int, pcol: int,
                                     rank_order: str = "row", block_order: str = "col") -> int:
    h = _vp()
    _check(_lib.costa_layout_create_block_cyclic(nrows, ncols, mb, nb, prow, pcol, ORDERS[rank_order],
                                                 ORDERS[block_order], ctypes.byref(h)),
           "costa_layout_create_block_cyclic")
    return h.value


def _grid(nprow: int, npcol: int, rank_order: str = "row", nranks: int = 0, rank_map=None) -> CostaGrid:
    """A grid; rank_map (nprow*npcol ranks, column-major over the grid) makes
    it a subset of `nranks` ranks.  The map array is kept on the returned
    structure for as long as it lives."""
    g = CostaGrid(nprow, npcol, ORDERS[rank_order], nranks, None)
    if rank_map is not None:
        rm = np.ascontiguousarray(rank_map, dtype=np.int32)
        g.rank_map = rm.ctypes.data
        g._keep = rm
    return g


def _desc9(desc) -> np.ndarray:
    d = np.ascontiguousarray(desc, dtype=np.int32)
    if d.size != 9:
        raise ValueError("a ScaLAPACK descriptor has 9 entries")
    return d


def costa_layout_create_scalapack(desc, nprow: int, npcol: int, rank_order: str = "row", nranks: int = 0,
                                  rank_map=None) -> int:
    d, g, h = _desc9(desc), _grid(nprow, npcol, rank_order, nranks, rank_map), _vp()
    _check(_lib.costa_layout_create_scalapack(d.ctypes.data, ctypes.byref(g), ctypes.byref(h)),
           "costa_layout_create_scalapack")
    return h.value


def costa_layout_submatrix(layout, i0: int, j0: int, m: int, n: int) -> int:
    h = _vp()
    _check(_lib.costa_layout_submatrix(_h(layout), i0, j0, m, n, ctypes.byref(h)), "costa_layout_submatrix")
    return h.value


def costa_layout_local_elems(layout: int, rank: int) -> int:
    n = _i64()
    _check(_lib.costa_layout_local_elems(layout, rank, ctypes.byref(n)), "costa_layout_local_elems")
    return n.value


def costa_layout_block(layout: int, bi: int, bj: int):
    o, off, ld = _i32(), _i64(), _i64()
    _check(_lib.costa_layout_block(layout, bi, bj, ctypes.byref(o), ctypes.byref(off), ctypes.byref(ld)),
           "costa_layout_block")
    return o.value, off.value, ld.value


def costa_layout_info(layout: int):
    nr, nc, br, bc, p, order = _i64(), _i64(), _i32(), _i32(), _i32(), ctypes.c_int()
    _check(_lib.costa_layout_info(layout, ctypes.byref(nr), ctypes.byref(nc), ctypes.byref(br), ctypes.byref(bc),
                                  ctypes.byref(p), ctypes.byref(order)), "costa_layout_info")
    return {"nrows": nr.value, "ncols": nc.value, "nbr": br.value, "nbc": bc.value, "nranks": p.value,
            "block_order": "col" if order.value == 0 else "row"}


def costa_layout_destroy(layout: int) -> None:
    _check(_lib.costa_layout_destroy(layout), "costa_layout_destroy")


class Layout:
    """Owning handle: destroys the C layout when collected."""

    def __init__(self, handle: int):
        self.handle = handle
        info = costa_layout_info(handle)
        self.__dict__.update(info)

    @classmethod
    def block_cyclic(cls, *args, **kw) -> "Layout":
        return cls(costa_layout_create_block_cyclic(*args, **kw))

    @classmethod
    def general(cls, *args, **kw) -> "Layout":
        return cls(costa_layout_create(*args, **kw))

    @classmethod
    def scalapack(cls, *args, **kw) -> "Layout":
        return cls(costa_layout_create_scalapack(*args, **kw))

    def submatrix(self, i0: int, j0: int, m: int, n: int) -> "Layout":
        return Layout(costa_layout_submatrix(self.handle, i0, j0, m, n))

    def local_elems(self, rank: int) -> int:
        return costa_layout_local_elems(self.handle, rank)

    def __del__(self):
        h, self.handle = getattr(self, "handle", None), None
        # at interpreter exit the module's globals may already be cleared;
        # the process is ending and the handle goes with it
        if h and _lib is not None:
            _lib.costa_layout_destroy(h)


def _h(x) -> int:
    return x.handle if isinstance(x, Layout) else int(x)


# ---------------------------------------------------------------------------
# volume, relabeling, transform
# ---------------------------------------------------------------------------
def costa_volume_matrix(A, B, op: str, stream=None) -> np.ndarray:
    P = costa_layout_info(_h(A))["nranks"]
    V = np.zeros((P, P), dtype=np.int64)
    _check(_lib.costa_volume_matrix(_h(A), _h(B), OPS[op], V.ctypes.data, _stream(stream)), "costa_volume_matrix")
    return V


def costa_relabel(V: np.ndarray):
    V = np.ascontiguousarray(V, dtype=np.int64)
    P = V.shape[0]
    sigma = np.zeros(P, dtype=np.int32)
    r0, r1 = _i64(), _i64()
    _check(_lib.costa_relabel(P, V.ctypes.data, sigma.ctypes.data, ctypes.byref(r0), ctypes.byref(r1)),
           "costa_relabel")
    return sigma.tolist(), r0.value, r1.value


RELABEL = {"exact": 0, "greedy": 1}


def costa_relabel_cost(V: np.ndarray, elem_bytes: float = 1.0, latency=None, inv_bandwidth=None,
                       method: str = "exact"):
    """(sigma, W(G), W(G_sigma)) under the locally-free cost (latency and
    inv_bandwidth None) or the latency-bandwidth cost."""
    V = np.ascontiguousarray(V, dtype=np.int64)
    P = V.shape[0]
    lat = None if latency is None else np.ascontiguousarray(latency, dtype=np.float64)
    ib = None if inv_bandwidth is None else np.ascontiguousarray(inv_bandwidth, dtype=np.float64)
    sigma = np.zeros(max(P, 1), dtype=np.int32)
    before, after = ctypes.c_double(), ctypes.c_double()
    _check(_lib.costa_relabel_cost(P, V.ctypes.data, elem_bytes, None if lat is None else lat.ctypes.data,
                                   None if ib is None else ib.ctypes.data, RELABEL[method], sigma.ctypes.data,
                                   ctypes.byref(before), ctypes.byref(after)), "costa_relabel_cost")
    return sigma[:P].tolist(), before.value, after.value


def _ptr_array(bufs: Sequence) -> ctypes.Array:
    return (_vp * len(bufs))(*[_addr(b) or None for b in bufs])


def _desc(dtype: str, op: str, alpha, beta, A, A_local, B, B_local, keep: List):
    al = None if alpha is None else _scalar(dtype, alpha)
    be = None if beta is None else _scalar(dtype, beta)
    ap = None if A_local is None else _ptr_array(A_local)
    bp = None if B_local is None else _ptr_array(B_local)
    keep.extend([al, be, ap, bp])
    d = CostaDesc()
    d.op = OPS[op]
    d.alpha = None if al is None else ctypes.cast(ctypes.pointer(al), _vp)
    d.beta = None if be is None else ctypes.cast(ctypes.pointer(be), _vp)
    d.A = _h(A)
    d.A_local = None if ap is None else ctypes.cast(ap, _vp)
    d.B = _h(B)
    d.B_local = None if bp is None else ctypes.cast(bp, _vp)
    return d


def _sigma(sigma):
    if sigma is None:
        return None, None
    s = np.ascontiguousarray(sigma, dtype=np.int32)
    return s, s.ctypes.data


def costa_transform(dtype: str, op: str, alpha, beta, A, A_local: Sequence, B, B_local: Sequence,
                    sigma=None, stream=None) -> None:
    keep: List = []
    d = _desc(dtype, op, alpha, beta, A, A_local, B, B_local, keep)
    s, sp = _sigma(sigma)
    _check(_lib.costa_transform(DTYPES[dtype], d.op, d.alpha, d.beta, d.A, d.A_local, d.B, d.B_local, sp,
                                _stream(stream)), "costa_transform")


def costa_transform_batched(dtype: str, descs: Sequence[dict], sigma=None, stream=None) -> None:
    """descs: dicts with keys op, alpha, beta, A, A_local, B, B_local."""
    keep: List = []
    arr = (CostaDesc * len(descs))(*[_desc(dtype, d["op"], d["alpha"], d["beta"], d["A"], d["A_local"], d["B"],
                                           d["B_local"], keep) for d in descs])
    s, sp = _sigma(sigma)
    _check(_lib.costa_transform_batched(DTYPES[dtype], len(descs), ctypes.cast(arr, _vp), sp, _stream(stream)),
           "costa_transform_batched")


# Size of the static device array of costa_transform_batched_noalloc (per
# device) and the part of it that holds the plan's tables.
NOALLOC_SCRATCH_BYTES = 64 << 20
NOALLOC_TABLE_BYTES = 16 << 20


def costa_transform_batched_noalloc(dtype: str, descs: Sequence[dict], sigma=None, stream=None) -> None:
    """costa_transform_batched without device allocation (tables and messages
    in the library's static scratch array); same descriptors."""
    keep: List = []
    arr = (CostaDesc * len(descs))(*[_desc(dtype, d["op"], d["alpha"], d["beta"], d["A"], d["A_local"], d["B"],
                                           d["B_local"], keep) for d in descs])
    s, sp = _sigma(sigma)
    _check(_lib.costa_transform_batched_noalloc(DTYPES[dtype], len(descs), ctypes.cast(arr, _vp), sp,
                                                _stream(stream)), "costa_transform_batched_noalloc")


def costa_plan_stats(dtype: str, descs: Sequence[dict], sigma=None) -> dict:
    keep: List = []
    arr = (CostaDesc * len(descs))(*[_desc(dtype, d["op"], d.get("alpha"), d.get("beta"), d["A"], None, d["B"],
                                           None, keep) for d in descs])
    s, sp = _sigma(sigma)
    st = CostaStats()
    _check(_lib.costa_plan_stats(DTYPES[dtype], len(descs), ctypes.cast(arr, _vp), sp, ctypes.byref(st)),
           "costa_plan_stats")
    return {name: getattr(st, name) for name, _ in CostaStats._fields_}


def costa_plan_export(dtype: str, descs: Sequence[dict], sigma=None) -> np.ndarray:
    """The plan's rectangles in launch order, as a numpy structured array."""
    keep: List = []
    arr = (CostaDesc * len(descs))(*[_desc(dtype, d["op"], d.get("alpha"), d.get("beta"), d["A"], None, d["B"],
                                           None, keep) for d in descs])
    s, sp = _sigma(sigma)
    cnt = _i64()
    _check(_lib.costa_plan_export(DTYPES[dtype], len(descs), ctypes.cast(arr, _vp), sp, None, 0,
                                  ctypes.byref(cnt)), "costa_plan_export")
    out = (CostaPieceInfo * max(1, cnt.value))()
    _check(_lib.costa_plan_export(DTYPES[dtype], len(descs), ctypes.cast(arr, _vp), sp, ctypes.cast(out, _vp),
                                  cnt.value, ctypes.byref(cnt)), "costa_plan_export")
    return np.ctypeslib.as_array(out)[:cnt.value].copy()


# ---------------------------------------------------------------------------
# ScaLAPACK-compatible routines (1-based indices, 9-entry descriptors; a grid
# is (nprow, npcol, rank_order[, nranks, rank_map]))
# ---------------------------------------------------------------------------
def _sl_args(a, ia, ja, desca, grida, c, ic, jc, descc, gridc, keep):
    da, dc = _desc9(desca), _desc9(descc)
    ga, gc = _grid(*grida), _grid(*gridc)
    ap, cp = _ptr_array(a), _ptr_array(c)
    keep.extend([da, dc, ga, gc, ap, cp])
    return (ctypes.cast(ap, _vp), ia, ja, da.ctypes.data, ctypes.byref(ga),
            ctypes.cast(cp, _vp), ic, jc, dc.ctypes.data, ctypes.byref(gc))


def costa_pxgemr2d(dtype: str, m: int, n: int, a, ia: int, ja: int, desca, grida, b, ib: int, jb: int, descb,
                   gridb, stream=None) -> None:
    keep: List = []
    _check(_lib.costa_pxgemr2d(DTYPES[dtype], m, n, *_sl_args(a, ia, ja, desca, grida, b, ib, jb, descb, gridb, keep),
                               _stream(stream)), "costa_pxgemr2d")


def costa_pxtran(dtype: str, op: str, m: int, n: int, alpha, a, ia: int, ja: int, desca, grida, beta, c,
                 ic: int, jc: int, descc, gridc, stream=None) -> None:
    keep: List = []
    al, be = _scalar(dtype, alpha), _scalar(dtype, beta)
    ap, ia_, ja_, da, ga, cp, ic_, jc_, dc, gc = _sl_args(a, ia, ja, desca, grida, c, ic, jc, descc, gridc, keep)
    _check(_lib.costa_pxtran(DTYPES[dtype], OPS[op], m, n, ctypes.cast(ctypes.pointer(al), _vp), ap, ia_, ja_, da,
                             ga, ctypes.cast(ctypes.pointer(be), _vp), cp, ic_, jc_, dc, gc, _stream(stream)),
           "costa_pxtran")


def costa_pdgemr2d(m: int, n: int, a, ia: int, ja: int, desca, grida, b, ib: int, jb: int, descb, gridb,
                   stream=None) -> None:
    keep: List = []
    _check(_lib.costa_pdgemr2d(m, n, *_sl_args(a, ia, ja, desca, grida, b, ib, jb, descb, gridb, keep),
                               _stream(stream)), "costa_pdgemr2d")


def _pxtran_named(name: str, dtype: str, m, n, alpha, a, ia, ja, desca, grida, beta, c, ic, jc, descc, gridc,
                  stream):
    keep: List = []
    al, be = _scalar(dtype, alpha), _scalar(dtype, beta)
    ap, ia_, ja_, da, ga, cp, ic_, jc_, dc, gc = _sl_args(a, ia, ja, desca, grida, c, ic, jc, descc, gridc, keep)
    _check(getattr(_lib, name)(m, n, ctypes.cast(ctypes.pointer(al), _vp), ap, ia_, ja_, da, ga,
                               ctypes.cast(ctypes.pointer(be), _vp), cp, ic_, jc_, dc, gc, _stream(stream)), name)


def costa_pdtran(m, n, alpha, a, ia, ja, desca, grida, beta, c, ic, jc, descc, gridc, stream=None) -> None:
    _pxtran_named("costa_pdtran", "f64", m, n, alpha, a, ia, ja, desca, grida, beta, c, ic, jc, descc, gridc, stream)


def costa_pztranu(m, n, alpha, a, ia, ja, desca, grida, beta, c, ic, jc, descc, gridc, stream=None) -> None:
    _pxtran_named("costa_pztranu", "c128", m, n, alpha, a, ia, ja, desca, grida, beta, c, ic, jc, descc, gridc,
                  stream)


def costa_pztranc(m, n, alpha, a, ia, ja, desca, grida, beta, c, ic, jc, descc, gridc, stream=None) -> None:
    _pxtran_named("costa_pztranc", "c128", m, n, alpha, a, ia, ja, desca, grida, beta, c, ic, jc, descc, gridc,
                  stream)


def costa_set_workspace_limit(nbytes: int) -> None:
    _check(_lib.costa_set_workspace_limit(nbytes), "costa_set_workspace_limit")


def costa_timing_enable(on: bool = True) -> None:
    _check(_lib.costa_timing_enable(1 if on else 0), "costa_timing_enable")


def costa_timing_read() -> dict:
    t = CostaTiming()
    _check(_lib.costa_timing_read(ctypes.byref(t)), "costa_timing_read")
    return {k: {"ms": t.ms[i], "launches": t.launches[i], "bytes": t.bytes[i]} for i, k in enumerate(KERNELS)}


def costa_finalize() -> None:
    _check(_lib.costa_finalize(), "costa_finalize")


def costa_status_string(status: int) -> str:
    return _lib.costa_status_string(status).decode()


def costa_last_error() -> str:
    return _lib.costa_last_error().decode()


def layout_from_spec(spec) -> Layout:
    """Layout from a recipe object with the attributes of a block-cyclic
    (nrows, ncols, mb, nb, prow, pcol, rank_order, block_order) or general
    (nrows, ncols, row_splits, col_splits, owners, nranks, block_order) grid,
    or of a ScaLAPACK descriptor (desc(), nprow, npcol, rank_order)."""
    if spec.kind == "block_cyclic":
        return Layout.block_cyclic(spec.nrows, spec.ncols, spec.mb, spec.nb, spec.prow, spec.pcol,
                                   spec.rank_order, spec.block_order)
    if spec.kind == "scalapack":
        return Layout.scalapack(spec.desc(), spec.nprow, spec.npcol, spec.rank_order, getattr(spec, "world", 0),
                                getattr(spec, "rank_map", None))
    return Layout.general(spec.nrows, spec.ncols, spec.row_splits, spec.col_splits, spec.owners, spec.nranks,
                          spec.block_order)
