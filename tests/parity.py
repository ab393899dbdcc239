"""Device-vs-oracle parity helpers (used by the GPU tests and the smoke check).

Inputs come from the seeded generator (synth): element idx of the buffer of
rank r gets value(seed, stream(role, pair, r), idx), on the device through
libcosta_synth.so and on the host through the same definition in the oracle.
Expected values come only from the oracle.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle
import synth

C = None  # the library binding, imported lazily so CPU-only collection works

TORCH = {"f64": torch.float64, "c128": torch.complex128, "f32": torch.float32, "c64": torch.complex64}
UINT = {"f64": np.uint64, "c128": np.uint64, "f32": np.uint32, "c64": np.uint32}


def lib():
    global C
    if C is None:
        import paper_2106_06601_amd as mod
        C = mod
    return C


def bits(x: np.ndarray, dtype: str) -> np.ndarray:
    """Raw bit patterns (complex: both parts)."""
    return np.ascontiguousarray(x).view(UINT[dtype])


class Case:
    """One (batched) transform of a workload on the device."""

    def __init__(self, w: synth.Workload, sigma="auto", a_init="gen", device="cuda:0"):
        L = lib()
        self.w = w
        self.dtype = w.dtype
        self.dev = torch.device(device)
        self.P = w.items[0].A.nranks
        self.LA = [L.layout_from_spec(it.A) for it in w.items]
        self.LB = [L.layout_from_spec(it.B) for it in w.items]
        self.OA = [oracle.OLayout(it.A) for it in w.items]
        self.OB = [oracle.OLayout(it.B) for it in w.items]
        self.stream = torch.cuda.current_stream(self.dev)
        self.V = None
        if sigma == "auto":
            if w.relabel:
                self.V = sum(L.costa_volume_matrix(a, b, it.op) for a, b, it in zip(self.LA, self.LB, w.items))
                self.sigma = L.costa_relabel(self.V)[0]
            else:
                self.sigma = None
        else:
            self.sigma = sigma
        sg = self.sigma if self.sigma is not None else list(range(self.P))
        inv = [0] * self.P
        for t, r in enumerate(sg):
            inv[r] = t
        self.inv = inv
        td = TORCH[self.dtype]
        self.A, self.B = [], []
        for k, it in enumerate(w.items):
            # physical rank r holds label inv[r]
            a = [torch.empty(self.LA[k].local_elems(inv[r]), dtype=td, device=self.dev) for r in range(self.P)]
            b = [torch.empty(self.LB[k].local_elems(s), dtype=td, device=self.dev) for s in range(self.P)]
            self.A.append(a)
            self.B.append(b)
        self.a_init = a_init
        self.fill()

    def fill(self):
        h = self.stream.cuda_stream
        for k in range(len(self.w.items)):
            for s, t in enumerate(self.B[k]):
                if t.numel():
                    synth.fill_device(self.dtype, t.data_ptr(), t.numel(), self.w.seed,
                                      synth.stream(synth.ROLE_B, k, s), h)
            for r, t in enumerate(self.A[k]):
                if not t.numel():
                    continue
                if self.a_init == "gen":
                    synth.fill_device(self.dtype, t.data_ptr(), t.numel(), self.w.seed,
                                      synth.stream(synth.ROLE_A, k, r), h)
                else:
                    t.fill_(float("nan"))

    def run(self):
        L = lib()
        w = self.w
        if len(w.items) == 1:
            it = w.items[0]
            L.costa_transform(self.dtype, it.op, it.alpha, it.beta, self.LA[0], self.A[0], self.LB[0], self.B[0],
                              self.sigma, self.stream)
        else:
            descs = [dict(op=it.op, alpha=it.alpha, beta=it.beta, A=self.LA[k], A_local=self.A[k], B=self.LB[k],
                          B_local=self.B[k]) for k, it in enumerate(w.items)]
            L.costa_transform_batched(self.dtype, descs, self.sigma, self.stream)

    # -- checks --------------------------------------------------------------
    def check_full(self):
        """Every element of every A buffer equal, bit for bit, to the oracle's."""
        torch.cuda.synchronize()
        npt = oracle.NUMPY[self.dtype]
        for k, it in enumerate(self.w.items):
            hb = []
            for s in range(self.P):
                a = np.zeros(self.OB[k].local_elems(s), dtype=npt)
                oracle.fill(self.dtype, a, self.w.seed, synth.stream(synth.ROLE_B, k, s))
                hb.append(a)
            ha = []
            for r in range(self.P):
                a = np.zeros(self.OA[k].local_elems(self.inv[r]), dtype=npt)
                if self.a_init == "gen":
                    oracle.fill(self.dtype, a, self.w.seed, synth.stream(synth.ROLE_A, k, r))
                else:
                    a[:] = np.nan
                ha.append(a)
            oracle.transform(self.dtype, it.op, it.alpha, it.beta, self.OA[k], ha, self.OB[k], hb, self.sigma)
            for r in range(self.P):
                got = self.A[k][r].cpu().numpy()
                exp = ha[r]
                if not np.array_equal(bits(got, self.dtype), bits(exp, self.dtype)):
                    bad = np.nonzero(bits(got, self.dtype) != bits(exp, self.dtype))[0]
                    raise AssertionError(f"pair {k} rank {r}: {bad.size} of {exp.size} elements differ; first at "
                                         f"{bad[:5]}: got {got.ravel()[bad[:3] % max(1, got.size)]} "
                                         f"expected {exp.ravel()[bad[:3] % max(1, exp.size)]}")

    def check_rows(self, k: int, row_begin: int = 0, row_end=None, ranks=None, threads: int = 16):
        """Every element of the given physical ranks of pair k (default: all of
        them) equal, bit for bit, to the oracle's result, which is computed on
        bands of the target rows [row_begin, row_end) by `threads` host
        threads at once (disjoint rows write disjoint elements).  The ranks
        compared must hold no element outside those rows.  Host inputs come
        from the generator, filled on the same threads."""
        from concurrent.futures import ThreadPoolExecutor
        torch.cuda.synchronize()
        it = self.w.items[k]
        npt = oracle.NUMPY[self.dtype]
        row_end = it.A.nrows if row_end is None else row_end
        ranks = list(range(self.P)) if ranks is None else list(ranks)
        hb = []
        for s in range(self.P):
            b = np.empty(self.OB[k].local_elems(s), dtype=npt)
            synth.fill_host_parallel(self.dtype, b, self.w.seed, synth.stream(synth.ROLE_B, k, s), threads)
            hb.append(b)
        ha = []
        for r in range(self.P):
            a = np.empty(self.OA[k].local_elems(self.inv[r]), dtype=npt)
            if self.a_init == "gen":
                synth.fill_host_parallel(self.dtype, a, self.w.seed, synth.stream(synth.ROLE_A, k, r), threads)
            else:
                a[:] = np.nan
            ha.append(a)
        N = it.A.ncols
        band = max(1, min(1024, (1 << 21) // max(1, N)))
        bands = [(r0, min(row_end, r0 + band)) for r0 in range(row_begin, row_end, band)]
        with ThreadPoolExecutor(max_workers=threads) as ex:
            list(ex.map(lambda b: oracle.transform(self.dtype, it.op, it.alpha, it.beta, self.OA[k], ha,
                                                   self.OB[k], hb, self.sigma, b[0], b[1]), bands))
        del hb
        checked = 0
        for r in ranks:
            got = bits(self.A[k][r].cpu().numpy(), self.dtype)
            exp = bits(ha[r], self.dtype)
            if not np.array_equal(got, exp):
                bad = np.nonzero(got != exp)[0]
                raise AssertionError(f"pair {k} rank {r}: {bad.size} of {exp.size} elements differ; first at "
                                     f"{bad[:5]}")
            checked += ha[r].size
        return checked

    def sample_points(self, k: int, n_random: int, n_corners: int, seed: int = 0):
        """Random points plus first/last rows and columns of overlay intervals."""
        it = self.w.items[k]
        rng = np.random.default_rng(seed)
        M, N = it.A.nrows, it.A.ncols
        rows = [rng.integers(0, M, n_random)]
        cols = [rng.integers(0, N, n_random)]

        def cuts(spec, dim):
            if spec.kind == "block_cyclic":
                b = spec.mb if dim == 0 else spec.nb
                n = spec.nrows if dim == 0 else spec.ncols
                return np.arange(0, n, b, dtype=np.int64)
            return np.asarray(spec.row_splits[:-1] if dim == 0 else spec.col_splits[:-1], dtype=np.int64)

        tr = it.op != "N"
        rc = np.union1d(cuts(it.A, 0), cuts(it.B, 1 if tr else 0))
        cc = np.union1d(cuts(it.A, 1), cuts(it.B, 0 if tr else 1))
        rb = np.unique(np.concatenate([rc, rc - 1, [M - 1]]))
        cb = np.unique(np.concatenate([cc, cc - 1, [N - 1]]))
        rb, cb = rb[(rb >= 0) & (rb < M)], cb[(cb >= 0) & (cb < N)]
        if rb.size * cb.size <= n_corners:
            ii, jj = np.meshgrid(rb, cb, indexing="ij")
            rows.append(ii.ravel())
            cols.append(jj.ravel())
        else:
            rows.append(rng.choice(rb, n_corners))
            cols.append(rng.choice(cb, n_corners))
        return np.concatenate(rows).astype(np.int64), np.concatenate(cols).astype(np.int64)

    def check_sampled(self, n_random=200000, n_corners=400000, seed=0):
        torch.cuda.synchronize()
        checked = 0
        for k, it in enumerate(self.w.items):
            i, j = self.sample_points(k, n_random, n_corners, seed + k)
            rank, off, exp = oracle.expect_at(self.dtype, it.op, it.alpha, it.beta, self.OA[k], self.OB[k],
                                              self.sigma, self.w.seed, k, i, j)
            got = np.empty_like(exp)
            for r in np.unique(rank):
                sel = np.nonzero(rank == r)[0]
                idx = torch.from_numpy(off[sel]).to(self.dev)
                got[sel] = self.A[k][int(r)].index_select(0, idx).cpu().numpy()
            bad = np.nonzero(bits(got, self.dtype) != bits(exp, self.dtype))[0]
            if bad.size:
                raise AssertionError(f"pair {k}: {bad.size} of {exp.size} sampled elements differ, e.g. "
                                     f"A({i[bad[0]]},{j[bad[0]]}) = {got[bad[0]]} expected {exp[bad[0]]}")
            checked += exp.size
        return checked

    def check_all_written(self):
        """With A prefilled with NaN and beta = 0: no NaN left anywhere."""
        torch.cuda.synchronize()
        for k in range(len(self.w.items)):
            for r, t in enumerate(self.A[k]):
                if t.numel() and bool(torch.isnan(t).any()):
                    raise AssertionError(f"pair {k} rank {r}: elements left unwritten")

    def free(self):
        self.A = self.B = None
        torch.cuda.synchronize()
        torch.cuda.empty_cache()  # hand the memory back, so later tests see it as free
