"""CPU oracle for the COSTA layout transform -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never calls it and
shares no code with it (the only common piece is the seeded input generator of
``synth/``).

Contents
--------
* ``liboracle.so`` (``costa_oracle.c``): storage maps (general grids,
  block-cyclic layouts and ScaLAPACK descriptors), element-by-element
  transform of whole matrices or of windows (submatrices), brute-force volume
  matrix, expected values at sampled points.
* Relabeling (Section 4): the communication cost W(G_sigma) of the relabeled
  graph computed from its definition, the relabeling gain delta (eq:delta)
  computed from its definition, and the communication-optimal relabeling
  argmin_sigma W(G_sigma) (Definition of COPR) by

  - brute force over all P! permutations (P <= 8),
  - dynamic programming over subsets of used senders (P <= 16),
  - scipy's linear-assignment solver as a library step plus a fix-and-check
    pass for the tie-break (any P);

  all three return the same canonical relabeling: among all optimal ones, the
  lexicographically smallest array sigma[0..P-1].

Convention (Section 4.1, relabeled graph): V[s][t] is the volume that sender s
(owner in L(B)) must deliver to receiver label t (owner in L(A)); relabeling
moves label t to physical rank sigma[t], so V[s][t] stays local iff s == sigma[t].
"""
from __future__ import annotations

import ctypes
import itertools
import os
import subprocess
from typing import Dict, List, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "costa_oracle.c")
# COSTA_ORACLE_LIB: load another build of the same source (the tests'
# sanitizer run builds one)
LIB_PATH = os.environ.get("COSTA_ORACLE_LIB") or os.path.join(HERE, "liboracle.so")

OPS = {"N": 0, "T": 1, "C": 2}
DTYPES = {"f64": 0, "c128": 1, "f32": 2, "c64": 3}
NUMPY = {"f64": np.float64, "c128": np.complex128, "f32": np.float32, "c64": np.complex64}


def build(out=None, cc="gcc", extra=()) -> str:
    """Compile the oracle (no contraction of a*b+c into FMA); by default with
    gcc into oracle/liboracle.so."""
    out = out or LIB_PATH
    cmd = [cc, "-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared", *extra,
           "-o", out, SRC]
    subprocess.run(cmd, check=True)
    return out


class _OLayout(ctypes.Structure):
    _fields_ = [
        ("kind", ctypes.c_int32), ("row_major", ctypes.c_int32),
        ("nrows", ctypes.c_int64), ("ncols", ctypes.c_int64), ("nranks", ctypes.c_int32),
        ("mb", ctypes.c_int64), ("nb", ctypes.c_int64), ("prow", ctypes.c_int32), ("pcol", ctypes.c_int32),
        ("rank_row_major", ctypes.c_int32),
        ("nbr", ctypes.c_int32), ("nbc", ctypes.c_int32),
        ("rsplit", ctypes.c_void_p), ("csplit", ctypes.c_void_p), ("owners", ctypes.c_void_p),
        ("boff", ctypes.c_void_p), ("bld", ctypes.c_void_p),
        ("rsrc", ctypes.c_int32), ("csrc", ctypes.c_int32), ("lld", ctypes.c_int64),
        ("rank_map", ctypes.c_void_p),
    ]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH) or os.path.getmtime(LIB_PATH) < os.path.getmtime(SRC):
            build()
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        L.oracle_default_packing.argtypes = [ctypes.c_int32, ctypes.c_int32, P, P, P, ctypes.c_int32,
                                             ctypes.c_int32, P, P, P]
        L.oracle_local_elems.argtypes = [P, ctypes.c_int32]
        L.oracle_local_elems.restype = ctypes.c_int64
        L.oracle_locate_many.argtypes = [P, ctypes.c_int64, P, P, P, P]
        L.oracle_volume.argtypes = [P, P, ctypes.c_int, P]
        L.oracle_transform.argtypes = [ctypes.c_int, ctypes.c_int, P, P, P, P, P, P, P, ctypes.c_int64,
                                       ctypes.c_int64]
        L.oracle_expect_at.argtypes = [ctypes.c_int, ctypes.c_int, P, P, P, P, P, ctypes.c_uint64,
                                       ctypes.c_uint32, ctypes.c_int64, P, P, P, P, P]
        L.oracle_fill.argtypes = [ctypes.c_int, P, ctypes.c_int64, ctypes.c_uint64, ctypes.c_uint64]
        i64 = ctypes.c_int64
        L.oracle_volume_window.argtypes = [P, i64, i64, P, i64, i64, i64, i64, ctypes.c_int, P]
        L.oracle_numroc.argtypes = [i64, i64, i64, i64, i64]
        L.oracle_numroc.restype = i64
        L.oracle_transform_window.argtypes = [ctypes.c_int, ctypes.c_int, P, P, P, P, i64, i64, P, P, i64, i64, i64,
                                              P, i64, i64]
        L.oracle_expect_at_window.argtypes = [ctypes.c_int, ctypes.c_int, P, P, P, i64, i64, P, i64, i64, P,
                                              ctypes.c_uint64, ctypes.c_uint32, i64, P, P, P, P, P]
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


class OLayout:
    """The oracle's own view of a layout, built from a synth recipe."""

    def __init__(self, spec):
        self.spec = spec
        s = _OLayout()
        s.nrows, s.ncols = spec.nrows, spec.ncols
        s.row_major = 1 if getattr(spec, "block_order", "col") == "row" else 0
        s.nranks = spec.nranks
        self._keep = []
        if spec.kind == "block_cyclic":
            s.kind = 0
            s.mb, s.nb, s.prow, s.pcol = spec.mb, spec.nb, spec.prow, spec.pcol
            s.rank_row_major = 1 if spec.rank_order == "row" else 0
        elif spec.kind == "scalapack":
            # a ScaLAPACK descriptor: block-cyclic, column-major local matrices
            s.kind = 0
            s.row_major = 0
            s.mb, s.nb, s.prow, s.pcol = spec.mb, spec.nb, spec.nprow, spec.npcol
            s.rank_row_major = 1 if spec.rank_order == "row" else 0
            s.rsrc, s.csrc, s.lld = spec.rsrc, spec.csrc, spec.lld
            if getattr(spec, "rank_map", None) is not None:
                rm = np.ascontiguousarray(spec.rank_map, dtype=np.int32)
                assert rm.size == spec.nprow * spec.npcol
                s.rank_map = _ptr(rm)
                self._keep = [rm]
        else:
            s.kind = 1
            rs = np.asarray(spec.row_splits, dtype=np.int64)
            cs = np.asarray(spec.col_splits, dtype=np.int64)
            ow = np.asarray(spec.owners, dtype=np.int32)
            nbr, nbc = len(rs) - 1, len(cs) - 1
            boff = np.zeros(nbr * nbc, dtype=np.int64)
            bld = np.zeros(nbr * nbc, dtype=np.int64)
            loc = np.zeros(spec.nranks, dtype=np.int64)
            rc = lib().oracle_default_packing(nbr, nbc, _ptr(rs), _ptr(cs), _ptr(ow), spec.nranks, s.row_major,
                                              _ptr(boff), _ptr(bld), _ptr(loc))
            if rc != 0:
                raise ValueError("owner out of range")
            s.nbr, s.nbc = nbr, nbc
            s.rsplit, s.csplit, s.owners, s.boff, s.bld = _ptr(rs), _ptr(cs), _ptr(ow), _ptr(boff), _ptr(bld)
            self._keep = [rs, cs, ow, boff, bld]
        self.c = s
        self.nranks = spec.nranks

    @property
    def ref(self):
        return ctypes.byref(self.c)

    def local_elems(self, rank: int) -> int:
        return int(lib().oracle_local_elems(self.ref, rank))

    def locate(self, rows: np.ndarray, cols: np.ndarray):
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        cols = np.ascontiguousarray(cols, dtype=np.int64)
        rank = np.zeros(rows.size, dtype=np.int32)
        off = np.zeros(rows.size, dtype=np.int64)
        lib().oracle_locate_many(self.ref, rows.size, _ptr(rows), _ptr(cols), _ptr(rank), _ptr(off))
        return rank, off


# --------------------------------------------------------------------------
# volume matrix and transform
# --------------------------------------------------------------------------
def volume(A: OLayout, B: OLayout, op: str) -> np.ndarray:
    """V[s, t] by brute-force counting over every element of A."""
    P = A.nranks
    V = np.zeros((P, P), dtype=np.int64)
    if lib().oracle_volume(A.ref, B.ref, OPS[op], _ptr(V)) != 0:
        raise ValueError("layouts live on different process counts")
    return V


def volume_window(A: OLayout, ia: int, ja: int, B: OLayout, ib: int, jb: int, m: int, n: int,
                  op: str) -> np.ndarray:
    """V[s, t] of the m x n window of A at 0-based (ia, ja) receiving op of the
    window of B at (ib, jb), by brute-force counting."""
    P = A.nranks
    V = np.zeros((P, P), dtype=np.int64)
    if lib().oracle_volume_window(A.ref, ia, ja, B.ref, ib, jb, m, n, OPS[op], _ptr(V)) != 0:
        raise ValueError("layouts live on different process counts")
    return V


def volume_separable(A, B, op: str) -> np.ndarray:
    """V[s, t] for two block-cyclic recipes by counting rows and columns per
    pair of process coordinates: element (i, j) of A is owned by process
    (pr(i), pc(j)) and its source by process (pr_B(i'), pc_B(j')), so the
    element count factorises into a row count times a column count.  For
    sizes where the element-by-element count is too slow (10^10 elements)."""
    def coords(n, b, p):
        return (np.arange(n) // b) % p

    def rank(spec, pr, pc):
        return pr * spec.pcol + pc if spec.rank_order == "row" else pr + pc * spec.prow

    prA, pcA = coords(A.nrows, A.mb, A.prow), coords(A.ncols, A.nb, A.pcol)
    P = A.prow * A.pcol
    V = np.zeros((P, P), np.int64)
    if op == "N":
        rb, cb = coords(B.nrows, B.mb, B.prow), coords(B.ncols, B.nb, B.pcol)
        nr, nc = B.prow, B.pcol
    else:  # A row i reads B column i, A column j reads B row j
        rb, cb = coords(A.nrows, B.nb, B.pcol), coords(A.ncols, B.mb, B.prow)
        nr, nc = B.pcol, B.prow
    rows = np.zeros((nr, A.prow), np.int64)
    np.add.at(rows, (rb, prA), 1)
    cols = np.zeros((nc, A.pcol), np.int64)
    np.add.at(cols, (cb, pcA), 1)
    for x, a, y, c in itertools.product(range(nr), range(A.prow), range(nc), range(A.pcol)):
        prB, pcB = (x, y) if op == "N" else (y, x)
        V[rank(B, prB, pcB), rank(A, a, c)] += rows[x, a] * cols[y, c]
    return V


def _scalar2(x) -> np.ndarray:
    x = complex(x)
    return np.array([x.real, x.imag], dtype=np.float64)


def transform(dtype: str, op: str, alpha, beta, A: OLayout, A_bufs: Sequence[np.ndarray], B: OLayout,
              B_bufs: Sequence[np.ndarray], sigma: Optional[Sequence[int]] = None,
              row_begin: int = 0, row_end: Optional[int] = None) -> None:
    """In place on the host buffers A_bufs[r] (physical ranks)."""
    P = A.nranks
    assert len(A_bufs) == P and len(B_bufs) == P
    for a in list(A_bufs) + list(B_bufs):
        assert a.dtype == NUMPY[dtype] and a.flags["C_CONTIGUOUS"]
    Ap = (ctypes.c_void_p * P)(*[_ptr(a) for a in A_bufs])
    Bp = (ctypes.c_void_p * P)(*[_ptr(b) for b in B_bufs])
    sg = None
    if sigma is not None:
        sg = np.ascontiguousarray(sigma, dtype=np.int32)
    al, be = _scalar2(alpha), _scalar2(beta)
    rc = lib().oracle_transform(DTYPES[dtype], OPS[op], _ptr(al), _ptr(be), A.ref, Ap, B.ref, Bp,
                                None if sg is None else _ptr(sg), row_begin,
                                A.spec.nrows if row_end is None else row_end)
    if rc != 0:
        raise ValueError("layouts live on different process counts")


def expect_at(dtype: str, op: str, alpha, beta, A: OLayout, B: OLayout, sigma, seed: int, item: int,
              rows: np.ndarray, cols: np.ndarray):
    """(physical rank, offset, expected value) of sampled points of the final A,
    for inputs made by the seeded generator."""
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    n = rows.size
    rank = np.zeros(n, dtype=np.int32)
    off = np.zeros(n, dtype=np.int64)
    val = np.zeros(2 * n, dtype=np.float64)
    sg = None if sigma is None else np.ascontiguousarray(sigma, dtype=np.int32)
    al, be = _scalar2(alpha), _scalar2(beta)
    lib().oracle_expect_at(DTYPES[dtype], OPS[op], _ptr(al), _ptr(be), A.ref, B.ref,
                           None if sg is None else _ptr(sg), seed, item, n, _ptr(rows), _ptr(cols),
                           _ptr(rank), _ptr(off), _ptr(val))
    val = val.reshape(n, 2)
    if dtype in ("c128", "c64"):
        v = val[:, 0] + 1j * val[:, 1]
    else:
        v = val[:, 0]
    return rank, off, v.astype(NUMPY[dtype])


def transform_window(dtype: str, op: str, alpha, beta, A: OLayout, A_bufs: Sequence[np.ndarray], ia: int, ja: int,
                     B: OLayout, B_bufs: Sequence[np.ndarray], ib: int, jb: int, m: int, n: int,
                     sigma: Optional[Sequence[int]] = None) -> None:
    """The m x n window of A at 0-based (ia, ja) receives alpha*op(window of B
    at (ib, jb)) + beta*(itself), in place on the host buffers; the rest of A is
    left alone (Section 5, a submatrix by truncated splits)."""
    P = A.nranks
    assert len(A_bufs) == P and len(B_bufs) == P
    for a in list(A_bufs) + list(B_bufs):
        assert a.dtype == NUMPY[dtype] and a.flags["C_CONTIGUOUS"]
    Ap = (ctypes.c_void_p * P)(*[_ptr(a) for a in A_bufs])
    Bp = (ctypes.c_void_p * P)(*[_ptr(b) for b in B_bufs])
    sg = None if sigma is None else np.ascontiguousarray(sigma, dtype=np.int32)
    al, be = _scalar2(alpha), _scalar2(beta)
    rc = lib().oracle_transform_window(DTYPES[dtype], OPS[op], _ptr(al), _ptr(be), A.ref, Ap, ia, ja, B.ref, Bp,
                                       ib, jb, n, None if sg is None else _ptr(sg), 0, m)
    if rc != 0:
        raise ValueError("layouts live on different process counts")


def expect_at_window(dtype: str, op: str, alpha, beta, A: OLayout, ia: int, ja: int, B: OLayout, ib: int, jb: int,
                     seed: int, item: int, rows: np.ndarray, cols: np.ndarray):
    """expect_at for the window form of transform_window; rows and cols are
    window coordinates."""
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    n = rows.size
    rank = np.zeros(n, dtype=np.int32)
    off = np.zeros(n, dtype=np.int64)
    val = np.zeros(2 * n, dtype=np.float64)
    al, be = _scalar2(alpha), _scalar2(beta)
    lib().oracle_expect_at_window(DTYPES[dtype], OPS[op], _ptr(al), _ptr(be), A.ref, ia, ja, B.ref, ib, jb, None,
                                  seed, item, n, _ptr(rows), _ptr(cols), _ptr(rank), _ptr(off), _ptr(val))
    val = val.reshape(n, 2)
    v = val[:, 0] + 1j * val[:, 1] if dtype in ("c128", "c64") else val[:, 0]
    return rank, off, v.astype(NUMPY[dtype])


# --------------------------------------------------------------------------
# ScaLAPACK-style calls (pxgemr2d, pxtran, pxtranu, pxtranc)
# --------------------------------------------------------------------------
def numroc(n: int, nb: int, iproc: int, isrc: int, nprocs: int) -> int:
    """Rows (or columns) of an n-long dimension in blocks of nb that process
    iproc holds when dealing starts at process isrc (ScaLAPACK NUMROC)."""
    return int(lib().oracle_numroc(n, nb, iproc, isrc, nprocs))


def scalapack_call(call, A_bufs: Sequence[np.ndarray], C_bufs: Sequence[np.ndarray]) -> None:
    """Runs a ScaLAPACK-style call (a ``synth.ScaLapackCall``) on host buffers:
    gemr2d copies the m x n window of A at 1-based (ia, ja) into the window of
    C at (ic, jc); tran / tranu put beta*sub(C) + alpha*sub(A)^T there, tranc
    the conjugate transpose (sub(A) is then n x m)."""
    if call.routine == "gemr2d":
        op, alpha, beta = "N", 1.0, 0.0
    elif call.routine in ("tran", "tranu"):
        op, alpha, beta = "T", call.alpha, call.beta
    elif call.routine == "tranc":
        op, alpha, beta = "C", call.alpha, call.beta
    else:
        raise ValueError(call.routine)
    transform_window(call.dtype, op, alpha, beta, OLayout(call.C), C_bufs, call.ic - 1, call.jc - 1,
                     OLayout(call.A), A_bufs, call.ia - 1, call.ja - 1, call.m, call.n)


def fill(dtype: str, arr: np.ndarray, seed: int, strm: int) -> None:
    assert arr.dtype == NUMPY[dtype] and arr.flags["C_CONTIGUOUS"]
    lib().oracle_fill(DTYPES[dtype], _ptr(arr), arr.size, seed, strm)


# --------------------------------------------------------------------------
# relabeling (Section 4)
# --------------------------------------------------------------------------
def w_locally_free(i: int, j: int, vol: int) -> int:
    """Locally-free-volume-based cost, equation (eq:locally_free_w)."""
    return vol if i != j else 0


def w_topology(latency: np.ndarray, inv_bandwidth: np.ndarray, elem_bytes: float = 1.0):
    """Network-topology cost of Section 3: w(p_i, p_j, s) = L(p_i, p_j) +
    B(p_i, p_j) * V(s) for a non-empty package of V(s) bytes."""
    def w(i: int, j: int, vol: int):
        return latency[i, j] + inv_bandwidth[i, j] * (vol * elem_bytes)
    return w


def total_cost(V: np.ndarray, sigma: Sequence[int], w=w_locally_free):
    """W(G_sigma): sum over the edges of the relabeled graph (Definitions of
    W(G) and of the relabeled graph: package S_ij now goes to p_sigma(j))."""
    P = V.shape[0]
    W = 0
    for i in range(P):
        for j in range(P):
            if V[i, j] != 0:  # (p_i, p_j) in E iff S_ij is non-empty
                W += w(i, sigma[j], int(V[i, j]))
    return W


def gain(V: np.ndarray, x: int, y: int, w=w_locally_free):
    """delta(p_x, p_y) from its definition, equation (eq:delta): the sum over
    the left neighbours p_i of p_x of w(p_i, p_x, S_ix) - w(p_i, p_y, S_ix)."""
    P = V.shape[0]
    d = 0
    for i in range(P):
        if V[i, x] != 0:
            d += w(i, x, int(V[i, x])) - w(i, y, int(V[i, x]))
    return d


def total_gain(V: np.ndarray, sigma: Sequence[int], w=w_locally_free):
    """Delta_sigma = sum_j delta(p_j, p_sigma(j))."""
    return sum(gain(V, j, sigma[j], w) for j in range(V.shape[0]))


def relabel_bruteforce_cost(V: np.ndarray, w) -> List[int]:
    """argmin_sigma W(G_sigma) under a general cost w, over all P! relabelings
    (first minimiser in lexicographic order).  P <= 8."""
    P = V.shape[0]
    if P > 8:
        raise ValueError("brute force is for P <= 8")
    best, best_sigma = None, None
    for perm in itertools.permutations(range(P)):
        W = total_cost(V, perm, w)
        if best is None or W < best:
            best, best_sigma = W, list(perm)
    return best_sigma


def relabel_greedy(V: np.ndarray, w=w_locally_free) -> List[int]:
    """Algorithm 1 with the matching the paper's implementation uses (Section 6:
    a simple greedy 2-approximation): weights[i][j] = delta(p_i, p_j), edges
    taken by decreasing weight (ties: smaller i, then smaller j) while both ends
    are free; sigma[i] = j for every matched (p_i, p_j).

    The gains can be negative, and completing the greedy matching to a perfect
    one can then give a total gain below zero, below the identity's (always a
    perfect matching, with gain 0, as the proof of Theorem 2 in Section 4.2
    notes), which no 2-approximation of a maximum >= 0 can return.  The
    identity is kept in that case."""
    P = V.shape[0]
    weights = [[gain(V, i, j, w) for j in range(P)] for i in range(P)]
    edges = sorted(((i, j) for i in range(P) for j in range(P)), key=lambda e: (-weights[e[0]][e[1]], e[0], e[1]))
    sigma = [-1] * P
    used = [False] * P
    for i, j in edges:
        if sigma[i] < 0 and not used[j]:
            sigma[i] = j
            used[j] = True
    if sum(weights[i][sigma[i]] for i in range(P)) < 0:
        return list(range(P))
    return sigma


def retained(V: np.ndarray, sigma: Sequence[int]) -> int:
    """Volume that stays local under sigma (sum of V[s][t] with s == sigma[t])."""
    return int(sum(int(V[sigma[t], t]) for t in range(V.shape[0])))


def relabel_bruteforce(V: np.ndarray) -> List[int]:
    """argmin_sigma W(G_sigma) over all P! permutations in lexicographic order;
    the first minimiser found is the lexicographically smallest."""
    P = V.shape[0]
    if P > 8:
        raise ValueError("brute force is for P <= 8")
    best, best_sigma = None, None
    for perm in itertools.permutations(range(P)):
        W = total_cost(V, perm)
        if best is None or W < best:
            best, best_sigma = W, list(perm)
    return best_sigma


def relabel_dp(V: np.ndarray) -> List[int]:
    """Exact COPR by dynamic programming over the set of physical ranks already
    used by labels 0..t-1 (t = popcount); ties broken towards the smallest
    sigma[t], label by label, which gives the lexicographically smallest optimum."""
    P = V.shape[0]
    if P > 16:
        raise ValueError("dynamic programming is for P <= 16")
    Vi = [[int(V[s, t]) for t in range(P)] for s in range(P)]
    full = (1 << P) - 1
    NEG = -1
    best = [NEG] * (1 << P)  # best retained volume for labels popcount(mask)..P-1
    best[full] = 0
    for mask in range(full - 1, -1, -1):
        t = bin(mask).count("1")
        b = NEG
        for s in range(P):
            if not (mask >> s) & 1:
                v = Vi[s][t] + best[mask | (1 << s)]
                if v > b:
                    b = v
        best[mask] = b
    sigma, mask = [], 0
    for t in range(P):
        for s in range(P):
            if not (mask >> s) & 1 and Vi[s][t] + best[mask | (1 << s)] == best[mask]:
                sigma.append(s)
                mask |= 1 << s
                break
    return sigma


def _lap_max(V: np.ndarray) -> int:
    from scipy.optimize import linear_sum_assignment
    if V.shape[0] == 0:
        return 0
    r, c = linear_sum_assignment(V.astype(np.float64), maximize=True)
    return int(sum(int(V[i, j]) for i, j in zip(r, c)))


def relabel_exact(V: np.ndarray) -> List[int]:
    """Any P: the optimum value from scipy's assignment solver (a library
    step), then label by label the smallest sender that still allows it."""
    P = V.shape[0]
    Vi = np.asarray(V, dtype=np.int64)
    opt = _lap_max(Vi)
    sigma: List[int] = []
    used = set()
    fixed = 0
    for t in range(P):
        rest_t = list(range(t + 1, P))
        for s in range(P):
            if s in used:
                continue
            rest_s = [x for x in range(P) if x not in used and x != s]
            sub = Vi[np.ix_(rest_s, rest_t)] if rest_t else np.zeros((0, 0), dtype=np.int64)
            if fixed + int(Vi[s, t]) + _lap_max(sub) == opt:
                sigma.append(s)
                used.add(s)
                fixed += int(Vi[s, t])
                break
    return sigma


def relabel(V: np.ndarray) -> List[int]:
    P = V.shape[0]
    if P <= 8:
        return relabel_bruteforce(V)
    if P <= 16:
        return relabel_dp(V)
    return relabel_exact(V)
