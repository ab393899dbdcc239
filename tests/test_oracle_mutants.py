"""The oracle's pins catch plausible mistakes in the oracle (CPU only).

Each mutant below plants one mistake -- a wrong sign, a transposed index, a
dropped term, a swapped operand -- in a copy of the oracle (its C core or its
Python relabeling), builds that copy with the usual oracle build, and runs the
oracle's pin modules against it in a child process.  Every mutant must make
at least one pin fail; the unmutated copy must pass.  The mistakes are planted
only in the copies, never in the oracle the other tests use.
"""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PIN_MODULES = ["test_oracle_pins.py", "test_oracle_scalapack.py"]
C_SRC = "oracle/costa_oracle.c"
PY_SRC = "oracle/__init__.py"

pytestmark = pytest.mark.spawns

# (name, file, text of the correct code, the mistake planted in its place)
MUTANTS = [
    ("complex product, real part sign", C_SRC, "r.re = p1 - p2;", "r.re = p1 + p2;"),
    ("complex product, imaginary part sign", C_SRC, "r.im = p3 + p4;", "r.im = p3 - p4;"),
    ("real beta term scales B instead of A", C_SRC, "t2.re = beta.re * a_old.re;", "t2.re = beta.re * b.re;"),
    ("complex beta term uses alpha", C_SRC, "t2 = cmul(beta, a_old);", "t2 = cmul(alpha, a_old);"),
    ("complex64 product, real part sign", C_SRC, "float t1r = p1 - p2, t1i = p3 + p4;",
     "float t1r = p1 + p2, t1i = p3 + p4;"),
    ("complex64 beta term, real part sign", C_SRC, "float t2r = q1 - q2, t2i = q3 + q4;",
     "float t2r = q1 + q2, t2i = q3 + q4;"),
    ("complex64 beta term, imaginary part sign", C_SRC, "float t2r = q1 - q2, t2i = q3 + q4;",
     "float t2r = q1 - q2, t2i = q3 - q4;"),
    ("complex64 beta imaginary part dropped", C_SRC,
     "float q1 = beta[0] * a_old[0], q2 = beta[1] * a_old[1], q3 = beta[0] * a_old[1], q4 = beta[1] * a_old[0];",
     "float q1 = beta[0] * a_old[0], q2 = 0.0f, q3 = beta[0] * a_old[1], q4 = 0.0f;"),
    ("real beta term dropped", C_SRC, "\n  return cadd(t1, t2);\n}", "\n  return t1;\n}"),
    ("alpha = 1 shortcut for any real alpha", C_SRC, "int alpha_one = alpha.re == 1.0 && alpha.im == 0.0;",
     "int alpha_one = alpha.im == 0.0;"),
    ("transpose reads B(i, j)", C_SRC, "else { *bi = j; *bj = i; }", "else { *bi = i; *bj = j; }"),
    ("conjugate not applied", C_SRC,
     "cplx b = {src[0], cpx ? src[1] : 0.0};\n        if (op == O_OP_C && cpx) b.im = -b.im;",
     "cplx b = {src[0], cpx ? src[1] : 0.0};"),
    ("conjugate negates the real part", C_SRC,
     "cplx b = {src[0], cpx ? src[1] : 0.0};\n        if (op == O_OP_C && cpx) b.im = -b.im;",
     "cplx b = {src[0], cpx ? src[1] : 0.0};\n        if (op == O_OP_C && cpx) b.re = -b.re;"),
    ("first process row ignored", C_SRC, "int64_t pr = (i / L->mb + L->rsrc) % L->prow;",
     "int64_t pr = (i / L->mb) % L->prow;"),
    ("rank order swapped", C_SRC, "L->rank_row_major ? pr * L->pcol + pc : pr + pc * L->prow",
     "L->rank_row_major ? pr + pc * L->prow : pr * L->pcol + pc"),
    ("global row used as local row", C_SRC, "int64_t li = (i / (L->mb * L->prow)) * L->mb + i % L->mb;",
     "int64_t li = (i / L->mb) * L->mb + i % L->mb;"),
    ("local column block index off by the grid", C_SRC, "int64_t lj = (j / (L->nb * L->pcol)) * L->nb + j % L->nb;",
     "int64_t lj = (j / (L->nb * L->pcol)) * L->nb + j % (L->nb * L->pcol);"),
    ("numroc drops the partial last block", C_SRC, "else if (dist == extra) num += n % nb;", ";"),
    ("numroc ignores the source process", C_SRC, "int64_t dist = (iproc - isrc + nprocs) % nprocs;",
     "int64_t dist = iproc % nprocs;"),
    ("general grid storage order swapped", C_SRC,
     "(L->row_major ? ri * L->bld[b] + cj : ri + cj * L->bld[b])",
     "(L->row_major ? ri + cj * L->bld[b] : ri * L->bld[b] + cj)"),
    ("split lookup off by one at block starts", C_SRC, "if (s[mid] <= x) lo = mid;", "if (s[mid] < x) lo = mid;"),
    ("default packing ld uses the other extent", C_SRC, "bld[b] = row_major ? w : h;", "bld[b] = row_major ? h : w;"),
    ("volume matrix transposed", C_SRC, "V[(int64_t)s * P + t] += 1;", "V[(int64_t)t * P + s] += 1;"),
    ("relabeling ignored when placing A", C_SRC,
     "locate(A, ia + i, ja + j, &t, &oa);\n      int32_t r = sigma ? sigma[t] : t;",
     "locate(A, ia + i, ja + j, &t, &oa);\n      int32_t r = t;"),
    ("window offset of B dropped", C_SRC, "locate(B, ib + bi, jb + bj, &s, &ob);\n      if (dtype",
     "locate(B, bi, bj, &s, &ob);\n      if (dtype"),
    ("locally-free cost charges local packages", PY_SRC, "return vol if i != j else 0", "return vol"),
    ("relabeled package sent to sigma of the sender", PY_SRC, "W += w(i, sigma[j], int(V[i, j]))",
     "W += w(sigma[i], j, int(V[i, j]))"),
    ("gain sign flipped", PY_SRC, "d += w(i, x, int(V[i, x])) - w(i, y, int(V[i, x]))",
     "d += w(i, y, int(V[i, x])) - w(i, x, int(V[i, x]))"),
    ("retained volume read transposed", PY_SRC, "int(V[sigma[t], t])", "int(V[t, sigma[t]])"),
    ("brute force keeps the last optimum", PY_SRC, "W = total_cost(V, perm)\n        if best is None or W < best:",
     "W = total_cost(V, perm)\n        if best is None or W <= best:"),
    ("DP tie-break towards larger ranks", PY_SRC,
     "for t in range(P):\n        for s in range(P):\n            if not (mask >> s) & 1 and Vi[s][t]",
     "for t in range(P):\n        for s in reversed(range(P)):\n            if not (mask >> s) & 1 and Vi[s][t]"),
    ("greedy takes the lightest edges first", PY_SRC, "key=lambda e: (-weights[e[0]][e[1]], e[0], e[1])",
     "key=lambda e: (weights[e[0]][e[1]], e[0], e[1])"),
    ("greedy keeps a losing matching", PY_SRC, "if sum(weights[i][sigma[i]] for i in range(P)) < 0:",
     "if False:"),
    ("exact relabeling forgets the fixed volume", PY_SRC, "fixed += int(Vi[s, t])", "fixed += 0"),
    ("topology cost uses the reverse link", PY_SRC, "latency[i, j] + inv_bandwidth[i, j] * (vol * elem_bytes)",
     "latency[i, j] + inv_bandwidth[j, i] * (vol * elem_bytes)"),
    ("separable volume: transposed source grid", PY_SRC, "prB, pcB = (x, y) if op == \"N\" else (y, x)",
     "prB, pcB = (x, y)"),
    ("separable volume: B's block sizes swapped for op", PY_SRC,
     "rb, cb = coords(A.nrows, B.nb, B.pcol), coords(A.ncols, B.mb, B.prow)",
     "rb, cb = coords(A.nrows, B.mb, B.pcol), coords(A.ncols, B.nb, B.prow)"),
]


def _make_tree(dst: str, mutant=None) -> None:
    ign = shutil.ignore_patterns("__pycache__", "*.so", "*.o", "*.hip")
    shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(dst, "oracle"), ignore=ign)
    shutil.copytree(os.path.join(ROOT, "synth"), os.path.join(dst, "synth"), ignore=ign)
    os.makedirs(os.path.join(dst, "tests"))
    for f in ["conftest.py"] + PIN_MODULES:
        shutil.copy(os.path.join(ROOT, "tests", f), os.path.join(dst, "tests", f))
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), os.path.join(dst, "tests", "golden"))
    if mutant is not None:
        _, rel, old, new = mutant
        path = os.path.join(dst, rel)
        text = open(path).read()
        assert text.count(old) == 1, f"mutant site not unique in {rel}: {old!r}"
        with open(path, "w") as fh:
            fh.write(text.replace(old, new))


def _run_pins(tree: str) -> subprocess.CompletedProcess:
    env = {k: v for k, v in os.environ.items() if k not in ("COSTA_ORACLE_LIB", "LD_PRELOAD", "PYTHONPATH")}
    env["PYTHONDONTWRITEBYTECODE"] = "1"
    build = subprocess.run([sys.executable, "-c", "import oracle; oracle.build()"], cwd=tree, env=env,
                           stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=300)
    if build.returncode != 0:
        return build
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                           *[os.path.join("tests", m) for m in PIN_MODULES]],
                          cwd=tree, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                          timeout=600)


def test_every_planted_mistake_fails_a_pin(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("no gcc")
    clean = str(tmp_path / "clean")
    _make_tree(clean)
    r = _run_pins(clean)
    assert r.returncode == 0, "unmutated oracle copy fails its pins:\n" + r.stdout[-3000:]

    def one(k):
        tree = str(tmp_path / f"m{k}")
        _make_tree(tree, MUTANTS[k])
        return k, _run_pins(tree)

    with ThreadPoolExecutor(max_workers=min(6, os.cpu_count() or 1)) as ex:
        results = list(ex.map(one, range(len(MUTANTS))))
    survivors = [MUTANTS[k][0] for k, r in results if r.returncode == 0]
    assert not survivors, f"mistakes no pin detects: {survivors}"
