"""Seeded synthetic inputs for the layout-transform workloads.

This module is shared by the tests, the benchmark and the CPU oracle.  It holds
no part of the transform itself: only

* the counter-based value generator of ``gen.h`` (a numpy copy of it, and a
  device/host fill through ``libcosta_synth.so``),
* the workload recipes: matrix shapes, grids, block sizes, random splits and
  owners, op, alpha and beta, with the shapes of the paper's experiments
  (Section 7: block-size change of the ScaLAPACK benchmark, relabeling between
  row- and column-major process grids, the tall-and-skinny transposed RPA
  operands reshuffled into a COSMA-like layout).

Values are uniform on [-1, 1) on a 2^-52 grid (2^-23 for 32-bit types).
Element ``idx`` of the local buffer of rank ``r`` of matrix role ``role``
(B = 1, A_0 = 2) in batch item ``k`` gets ``value(seed, stream(role, k, r), idx)``.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcosta_synth.so")

ROLE_B = 1
ROLE_A = 2
DEFAULT_SEED = 0x5EED2106066010  # fixed seed of every workload

DTYPES = {"f64": 0, "c128": 1, "f32": 2, "c64": 3}
ITEMSIZE = {"f64": 8, "c128": 16, "f32": 4, "c64": 8}
NUMPY = {"f64": np.float64, "c128": np.complex128, "f32": np.float32, "c64": np.complex64}

_M64 = (1 << 64) - 1
_GOLDEN = 0x9E3779B97F4A7C15


# --------------------------------------------------------------------------
# scalar and numpy copies of gen.h
# --------------------------------------------------------------------------
def mix64(z: int) -> int:
    z &= _M64
    z ^= z >> 30
    z = (z * 0xBF58476D1CE4E5B9) & _M64
    z ^= z >> 27
    z = (z * 0x94D049BB133111EB) & _M64
    z ^= z >> 31
    return z


def bits(seed: int, stream: int, idx: int) -> int:
    return mix64((seed ^ mix64(stream) ^ (((idx + 1) * _GOLDEN) & _M64)) & _M64)


def stream(role: int, item: int, rank: int) -> int:
    return (role << 32) | ((item & 0xFFFF) << 16) | (rank & 0xFFFF)


def _mix64_np(z: np.ndarray) -> np.ndarray:
    z = z ^ (z >> np.uint64(30))
    z = z * np.uint64(0xBF58476D1CE4E5B9)
    z = z ^ (z >> np.uint64(27))
    z = z * np.uint64(0x94D049BB133111EB)
    z = z ^ (z >> np.uint64(31))
    return z


def bits_np(seed: int, strm: int, idx: np.ndarray) -> np.ndarray:
    idx = np.asarray(idx, dtype=np.uint64)
    with np.errstate(over="ignore"):
        key = np.uint64((seed ^ mix64(strm)) & _M64)
        return _mix64_np(key ^ ((idx + np.uint64(1)) * np.uint64(_GOLDEN)))


def _real64(b: np.ndarray) -> np.ndarray:
    return 2.0 * ((b >> np.uint64(11)).astype(np.float64) * 2.0**-53) - 1.0


def _real32(b: np.ndarray) -> np.ndarray:
    k = (b >> np.uint64(40)).astype(np.float32)
    return np.float32(2.0) * (k * np.float32(2.0**-24)) - np.float32(1.0)


def values(dtype: str, seed: int, strm: int, n: int, start: int = 0) -> np.ndarray:
    """Elements [start, start+n) of the buffer with stream `strm` (numpy)."""
    idx = np.arange(start, start + n, dtype=np.uint64)
    if dtype == "f64":
        return _real64(bits_np(seed, strm, idx))
    if dtype == "f32":
        return _real32(bits_np(seed, strm, idx))
    if dtype in ("c128", "c64"):
        re_b = bits_np(seed, strm, np.uint64(2) * idx)
        im_b = bits_np(seed, strm, np.uint64(2) * idx + np.uint64(1))
        if dtype == "c128":
            return _real64(re_b) + 1j * _real64(im_b)
        out = np.empty(n, dtype=np.complex64)
        out.real = _real32(re_b)
        out.imag = _real32(im_b)
        return out
    raise ValueError(dtype)


def below(seed: int, strm: int, ctr: int, n: int):
    """Uniform integer in [0, n) by rejection; returns (value, next counter)."""
    lim = _M64 - ((_M64 % n + 1) % n)
    while True:
        b = bits(seed, strm, ctr)
        ctr += 1
        if b <= lim:
            return b % n, ctr


def random_cuts(seed: int, strm: int, n: int, count: int) -> List[int]:
    """`count` distinct cut points drawn uniformly from [1, n-1], sorted."""
    if count > n - 1:
        raise ValueError("too many cuts")
    got: List[int] = []
    seen = set()
    ctr = 0
    while len(got) < count:
        c, ctr = below(seed, strm, ctr, n - 1)
        c += 1
        if c not in seen:
            seen.add(c)
            got.append(c)
    return sorted(got)


def random_owners(seed: int, strm: int, count: int, nranks: int) -> List[int]:
    out = []
    ctr = 0
    for _ in range(count):
        o, ctr = below(seed, strm, ctr, nranks)
        out.append(o)
    return out


# --------------------------------------------------------------------------
# compiled fills (device and host)
# --------------------------------------------------------------------------
_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built (run __graft_entry__.build())")
        try:  # one HIP runtime per process: torch's, when torch is installed
            import torch  # noqa: F401
        except ImportError:
            pass
        L = ctypes.CDLL(LIB_PATH)
        L.synth_fill.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64,
                                 ctypes.c_uint64, ctypes.c_void_p]
        L.synth_fill.restype = ctypes.c_int
        L.synth_fill_host.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64,
                                      ctypes.c_uint64]
        L.synth_fill_host.restype = ctypes.c_int
        L.synth_fill_host_range.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64,
                                            ctypes.c_uint64, ctypes.c_uint64]
        L.synth_fill_host_range.restype = ctypes.c_int
        _lib = L
    return _lib


def fill_device(dtype: str, ptr: int, n: int, seed: int, strm: int, hip_stream: int = 0) -> None:
    """Fill n elements at device address `ptr` on `hip_stream` (asynchronous)."""
    rc = lib().synth_fill(DTYPES[dtype], ctypes.c_void_p(ptr), n, seed, strm, ctypes.c_void_p(hip_stream))
    if rc != 0:
        raise RuntimeError(f"synth_fill failed ({rc})")


def fill_host(dtype: str, arr: np.ndarray, seed: int, strm: int) -> None:
    """Fill a contiguous numpy array in place (same values as the device fill)."""
    assert arr.flags["C_CONTIGUOUS"] and arr.dtype == NUMPY[dtype]
    rc = lib().synth_fill_host(DTYPES[dtype], ctypes.c_void_p(arr.ctypes.data), arr.size, seed, strm)
    if rc != 0:
        raise RuntimeError(f"synth_fill_host failed ({rc})")


def fill_host_parallel(dtype: str, arr: np.ndarray, seed: int, strm: int, threads: int = 16,
                       chunk: int = 1 << 22) -> None:
    """fill_host in chunks on `threads` threads (the C loop runs outside the GIL)."""
    from concurrent.futures import ThreadPoolExecutor
    assert arr.flags["C_CONTIGUOUS"] and arr.dtype == NUMPY[dtype]
    n = arr.size
    if n == 0:
        return
    L = lib()
    es = arr.itemsize
    base = arr.ctypes.data

    def part(first: int) -> int:
        m = min(chunk, n - first)
        return L.synth_fill_host_range(DTYPES[dtype], ctypes.c_void_p(base + first * es), first, m, seed, strm)

    with ThreadPoolExecutor(max_workers=max(1, threads)) as ex:
        rcs = list(ex.map(part, range(0, n, chunk)))
    if any(rcs):
        raise RuntimeError("synth_fill_host_range failed")


# --------------------------------------------------------------------------
# workload recipes
# --------------------------------------------------------------------------
@dataclass
class BlockCyclic:
    """ScaLAPACK-style layout: mb x nb blocks dealt cyclically over a prow x pcol grid.

    rank_order 'row': rank = pr * pcol + pc; 'col': rank = pr + pc * prow.
    block_order: storage order of each rank's local matrix ('col' or 'row').
    """
    nrows: int
    ncols: int
    mb: int
    nb: int
    prow: int
    pcol: int
    rank_order: str = "row"
    block_order: str = "col"
    kind: str = "block_cyclic"

    @property
    def nranks(self) -> int:
        return self.prow * self.pcol


@dataclass
class ScaLapack:
    """A ScaLAPACK array descriptor (DTYPE_ = 1) on a BLACS-style process grid.

    m x n global matrix in mb x nb blocks; the first block row and column live
    on process row rsrc and process column csrc; every rank stores its local
    matrix column-major with leading dimension lld.  rank_order 'row': rank =
    pr * npcol + pc; 'col': rank = pr + pc * nprow.  With rank_map (nprow *
    npcol entries, column-major over the grid, like a BLACS user map) the
    process at (pr, pc) is rank rank_map[pr + pc * nprow] of `world` ranks.
    """
    m: int
    n: int
    mb: int
    nb: int
    rsrc: int
    csrc: int
    lld: int
    nprow: int
    npcol: int
    rank_order: str = "row"
    kind: str = "scalapack"
    world: int = 0                      # ranks in all (0: nprow * npcol)
    rank_map: Optional[List[int]] = None

    @property
    def nranks(self) -> int:
        return self.world or self.nprow * self.npcol

    @property
    def nrows(self) -> int:
        return self.m

    @property
    def ncols(self) -> int:
        return self.n

    def desc(self) -> List[int]:
        """The nine descriptor entries (DTYPE_, CTXT_, M_, N_, MB_, NB_, RSRC_, CSRC_, LLD_)."""
        return [1, 0, self.m, self.n, self.mb, self.nb, self.rsrc, self.csrc, self.lld]


@dataclass
class ScaLapackCall:
    """One ScaLAPACK-style call: routine 'gemr2d' (sub(C) = sub(A)), 'tran' /
    'tranu' (sub(C) = beta sub(C) + alpha sub(A)^T) or 'tranc' (conjugate
    transpose).  sub(C) is the m x n window of C at 1-based (ic, jc); sub(A)
    the m x n (gemr2d) or n x m (tran*) window of A at (ia, ja)."""
    routine: str
    dtype: str
    m: int
    n: int
    alpha: complex
    beta: complex
    A: ScaLapack
    ia: int
    ja: int
    C: ScaLapack
    ic: int
    jc: int


@dataclass
class General:
    """Arbitrary grid: splits, owners (row-major over blocks), block storage order.

    Local storage is the default packing: each rank stores its blocks one after
    another, in row-major order of (block row, block col), each block packed
    with its own leading extent as stride.
    """
    nrows: int
    ncols: int
    row_splits: List[int]
    col_splits: List[int]
    owners: List[int]
    nranks: int
    block_order: str = "col"
    kind: str = "general"


@dataclass
class Item:
    A: object          # target layout (A is M x N)
    B: object          # source layout (M x N for op 'N', N x M otherwise)
    op: str            # 'N', 'T' or 'C'
    alpha: complex
    beta: complex


@dataclass
class Workload:
    name: str
    dtype: str
    items: List[Item]
    relabel: bool
    description: str = ""
    seed: int = DEFAULT_SEED


def _c3_source(n: int, cuts: int, nranks: int, seed: int) -> General:
    rs = [0] + random_cuts(seed, stream(3, 0, 0), n, cuts) + [n]
    cs = [0] + random_cuts(seed, stream(3, 0, 1), n, cuts) + [n]
    owners = random_owners(seed, stream(3, 0, 2), (len(rs) - 1) * (len(cs) - 1), nranks)
    return General(n, n, rs, cs, owners, nranks, "col")


def _cosma_like(n: int, g: int) -> General:
    splits = [k * n // g for k in range(g + 1)]
    owners = [bi * g + bj for bi in range(g) for bj in range(g)]
    return General(n, n, splits, splits, owners, g * g, "col")


def random_layout_pair(P: int, seed: int, n: int = 4096, cuts: int = None) -> tuple:
    """Two independent random general grids of an n x n matrix over P ranks
    (the relabeling comparison's "random layouts"): `cuts` distinct random
    interior cut points per dimension (default about 2 sqrt(P)), every block's
    owner drawn uniformly from the P ranks.  Returns (target A, source B)."""
    if cuts is None:
        cuts = max(1, int(round(2 * P ** 0.5)))
    out = []
    for role in (0, 1):
        rs = [0] + random_cuts(seed, stream(4, role, 0), n, cuts) + [n]
        cs = [0] + random_cuts(seed, stream(4, role, 1), n, cuts) + [n]
        owners = random_owners(seed, stream(4, role, 2), (len(rs) - 1) * (len(cs) - 1), P)
        out.append(General(n, n, rs, cs, owners, P, "col"))
    return out[0], out[1]


def workload(name: str, scale: str = "full", seed: int = DEFAULT_SEED) -> Workload:
    """The five workloads at full size ('full') or at a reduced size with the same
    grids, block sizes and ragged structure ('small', for element-wise parity)."""
    small = scale == "small"
    if name == "reshuffle_transpose_1k":
        n = 1024
        B = BlockCyclic(n, n, 32, 32, 2, 2, "row", "col")
        A = BlockCyclic(n, n, 64, 64, 2, 2, "col", "col")
        return Workload(name, "f64", [Item(A, B, "T", 1.0, 0.0)], True,
                        "fp64 1024^2, 2x2 grid 32^2 row-major ranks -> 2x2 grid 64^2 col-major ranks, "
                        "transpose, alpha=1 beta=0, relabeling on", seed)
    if name == "blocksize_change_16k":
        n = 2048 if small else 16384
        B = BlockCyclic(n, n, 128, 128, 4, 4)
        A = BlockCyclic(n, n, 256, 256, 4, 4)
        return Workload(name, "f64", [Item(A, B, "N", 1.0, 0.0)], True,
                        f"fp64 {n}^2, 4x4 grid 128^2 -> 4x4 grid 256^2, identity, alpha=1 beta=0, "
                        "relabeling on", seed)
    if name == "scaled_transpose_20k":
        n = 2000 if small else 20000
        B = BlockCyclic(n, n, 64, 64, 8, 4, "row", "col")
        A = BlockCyclic(n, n, 100, 100, 4, 8, "row", "row")
        return Workload(name, "f64", [Item(A, B, "T", 2.0, 0.5)], False,
                        f"fp64 {n}^2, 8x4 grid 64^2 col-major blocks -> 4x8 grid 100^2 row-major blocks, "
                        "transpose, alpha=2 beta=0.5", seed)
    if name == "cosma_complex_16k":
        n = 2048 if small else 16384
        B = _c3_source(n, 40, 64, seed)
        A = _cosma_like(n, 8)
        return Workload(name, "c128", [Item(A, B, "C", 1.0 + 0j, 0.0 + 0j)], False,
                        f"complex128 {n}^2, 41x41 random splits with random owners over 64 ranks -> "
                        "8x8 COSMA-like grid, conjugate transpose, alpha=1 beta=0", seed)
    if name == "rpa_batched_tall_skinny":
        m, ncol = (4096, 4096) if small else (4096, 524288)
        items = []
        for k in range(8):
            A = BlockCyclic(m, ncol, 512, 512, 8, 8)
            if k < 4:
                B = BlockCyclic(m, ncol, 64, 64, 1, 64)
                items.append(Item(A, B, "N", 1.0, 1.0))
            else:
                B = BlockCyclic(ncol, m, 64, 64, 1, 64)
                items.append(Item(A, B, "T", 1.0, 1.0))
        return Workload(name, "f64", items, False,
                        f"8 x fp64 {m}x{ncol}, 1x64 grid 64^2 -> 8x8 grid 512^2, 4 identity + 4 transpose, "
                        "alpha=1 beta=1", seed)
    raise KeyError(name)


WORKLOADS = ["reshuffle_transpose_1k", "blocksize_change_16k", "scaled_transpose_20k",
             "cosma_complex_16k", "rpa_batched_tall_skinny"]


def _lld(m: int, mb: int, nprow: int, pad: int) -> int:
    """A valid local leading dimension: a whole share of blocks per process
    row (ceil(ceil(m/mb)/nprow) blocks) plus `pad` rows of slack."""
    return -(-(-(-m // mb)) // nprow) * mb + pad


def scalapack_call(name: str, scale: str = "full") -> ScaLapackCall:
    """ScaLAPACK-style calls of the paper's ScaLAPACK comparison: a 16 x 16
    process grid, fp64, 32 x 32 source blocks -> 128 x 128 target blocks, the
    source a submatrix starting mid-block of a larger matrix, the target's
    first block on process (3, 5), padded leading dimensions; at full size
    ('full', 16384^2) or with the same grids and blocks at 2048^2 ('small').
    pztranc_8k is the complex conjugate transpose on 8 x 8 grids, and
    pdgemr2d_scatter_16k deals a matrix held by one process out to a 4 x 4
    grid of the same 16 ranks."""
    small = scale == "small"
    n = 2048 if small else 16384
    big = n + 512
    src = ScaLapack(big, big, 32, 32, 0, 0, _lld(big, 32, 16, 8), 16, 16)
    dst = ScaLapack(n, n, 128, 128, 3, 5, _lld(n, 128, 16, 8), 16, 16)
    if name == "pdgemr2d_16k":
        return ScaLapackCall("gemr2d", "f64", n, n, 1.0, 0.0, src, 17, 273, dst, 1, 1)
    if name == "pdtran_16k":
        return ScaLapackCall("tran", "f64", n, n, 1.0, 0.0, src, 17, 273, dst, 1, 1)
    if name == "pdgemr2d_scatter_16k":
        # a matrix held by one process (rank 0 of 16) dealt out to a 4 x 4 grid
        root = ScaLapack(n, n, 128, 128, 0, 0, n, 1, 1, world=16, rank_map=[0])
        grid = ScaLapack(n, n, 128, 128, 0, 0, _lld(n, 128, 4, 0), 4, 4)
        return ScaLapackCall("gemr2d", "f64", n, n, 1.0, 0.0, root, 1, 1, grid, 1, 1)
    if name == "pztranc_8k":
        m = 1024 if small else 8192
        a = ScaLapack(m + 100, m + 100, 64, 64, 1, 2, _lld(m + 100, 64, 8, 4), 8, 8, "col")
        c = ScaLapack(m, m, 96, 96, 0, 0, _lld(m, 96, 8, 0), 8, 8)
        return ScaLapackCall("tranc", "c128", m, m, 1.0 - 1.0j, 0.5, a, 50, 51, c, 1, 1)
    raise KeyError(name)


SCALAPACK_CALLS = ["pdgemr2d_16k", "pdtran_16k", "pztranc_8k", "pdgemr2d_scatter_16k"]
