"""Helpers of the CPU plan replays: the addressing of a work rectangle and
the element arithmetic, written out with numpy (every product and sum
rounded on its own)."""
import numpy as np

import oracle
import synth


def _index(p):
    x = np.arange(p["nx"], dtype=np.int64)[None, :]
    y = np.arange(p["ny"], dtype=np.int64)[:, None]
    dst = p["dst_off"] + y * p["dst_ld"] + x
    if p["flags"] & 1:
        src = p["src_off"] + x * p["src_ld"] + y
    else:
        src = p["src_off"] + y * p["src_ld"] + x
    return src.ravel(), dst.ravel()


def _combine(dtype, b, a, alpha, beta, conj):
    """alpha*b + beta*a with every product and sum rounded on its own."""
    cplx = dtype in ("c128", "c64")
    f = np.float64 if dtype in ("f64", "c128") else np.float32
    if cplx and conj:
        b = np.conj(b)  # sign flip of the imaginary part
    if alpha == 1 and beta == 0:
        return b
    if not cplx:
        t1 = f(alpha.real) * b
        return t1 if beta == 0 else t1 + f(beta.real) * a
    ar, ai = f(alpha.real), f(alpha.imag)
    br_, bi_ = b.real, b.imag
    t1r = ar * br_ - ai * bi_
    t1i = ar * bi_ + ai * br_
    if beta != 0:
        er, ei = f(beta.real), f(beta.imag)
        t1r = t1r + (er * a.real - ei * a.imag)
        t1i = t1i + (er * a.imag + ei * a.real)
    out = np.empty(b.shape, dtype=oracle.NUMPY[dtype])
    out.real = t1r
    out.imag = t1i
    return out


def many_rank_cases():
    """(dtype, op, alpha, beta, A, B, sigma) at many virtual ranks; sigma
    "auto" means relabeling on."""
    BC = synth.BlockCyclic
    return [
        # P = 1024: the source's 16 block columns leave half of its process
        # columns empty (zero-size buffers); relabeling on
        ("f64", "T", 2.0, 0.5,
         BC(2048, 2048, 64, 64, 32, 32, "row", "col"), BC(2048, 2048, 16, 128, 32, 32, "col", "row"), "auto"),
        # P = 4096: one 64 x 64 block per target rank, a random relabeling
        ("c128", "C", 1.0, 0.0,
         BC(4096, 4096, 64, 64, 64, 64, "col", "col"), BC(4096, 4096, 96, 32, 64, 64, "row", "col"),
         np.random.default_rng(41).permutation(4096).tolist()),
    ]


def short_walk_cases():
    """Layouts whose transform is all row walks of 4-64 elements that start
    and end inside 128-byte lines (blocks cut by the other grid's splits):
    16-byte units and single elements (odd leading dimension), all four
    element types, every arithmetic mode."""
    BC = synth.BlockCyclic
    return [
        # the scaled transpose's grids at 4000^2
        synth.Workload("walk0", "f64", [synth.Item(BC(4000, 4000, 100, 100, 4, 8, "row", "row"),
                                                   BC(4000, 4000, 64, 64, 8, 4, "row", "col"), "T", 2.0, 0.5)],
                       False, seed=51),
        # local rows of A 749 elements long (odd): single-element units
        synth.Workload("walk1", "f64", [synth.Item(BC(3000, 2996, 100, 107, 4, 4, "row", "row"),
                                                   BC(3000, 2996, 64, 64, 4, 4, "col", "row"), "N", -1.5, 0.0)],
                       False, seed=52),
        synth.Workload("walk2", "f32", [synth.Item(BC(3000, 3600, 100, 100, 4, 4, "row", "row"),
                                                   BC(3600, 3000, 64, 64, 4, 4, "row", "col"), "T", 0.3, 1.0)],
                       False, seed=53),
        synth.Workload("walk3", "c128", [synth.Item(BC(2400, 2400, 100, 100, 4, 4, "col", "col"),
                                                    BC(2400, 2400, 64, 64, 4, 4, "row", "row"), "C",
                                                    0.5 - 0.25j, 0.25 + 1j)], False, seed=54),
        synth.Workload("walk4", "c64", [synth.Item(BC(2400, 2400, 100, 100, 4, 4, "row", "row"),
                                                   BC(2400, 2400, 64, 64, 4, 4, "col", "col"), "T", 1.0, 0.0)],
                       False, seed=55),
    ]


def stack_cases():
    """Layouts whose row walks stack (rectangles with rows of 128-512 bytes
    that follow one another along a local column, at least 256 units wide):
    ScaLAPACK descriptors on 2 x 2 grids, 32-row source blocks into 128-row
    target blocks with a different first process, padded leading dimensions
    (columns alternately off the 128-byte lines) -- stacks on the source side
    (pack) and on the destination side (unpack and the direct rectangles with
    it, for pairs that do not read A); 16-byte units and single elements (odd
    padding), all four element types, copy and scale (and axpby, whose
    rectangles stack in the pack only), stacks whose last wave is partly idle
    (1000 local rows) and row counts that are not a multiple of the rows per
    wave task (blocks of 26 columns)."""
    SL = synth.ScaLapack

    def pair(m, n, pad_a, pad_b, mb=32):
        B = SL(m, n, mb, mb, 0, 0, -(-(-(-m // mb)) // 2) * mb + pad_b, 2, 2)
        A = SL(m, n, 128, 128, 1, 0, -(-(-(-m // 128)) // 2) * 128 + pad_a, 2, 2)
        return A, B

    out = []
    A, B = pair(2048, 90, 8, 8)
    out.append(synth.Workload("stack0", "f64", [synth.Item(A, B, "N", 1.0, 0.0)], False, seed=61))
    A, B = pair(2000, 96, 8, 8)
    out.append(synth.Workload("stack1", "f64", [synth.Item(A, B, "N", 2.0, 0.5)], False, seed=62))
    A, B = pair(2048, 64, 1, 3)
    out.append(synth.Workload("stack2", "f32", [synth.Item(A, B, "N", -1.5, 0.0)], False, seed=63))
    A, B = pair(2048, 58, 4, 4, mb=16)
    out.append(synth.Workload("stack3", "c128", [synth.Item(A, B, "N", 0.5 - 0.25j, 0.0)], False, seed=64))
    A, B = pair(2048, 70, 4, 4)
    out.append(synth.Workload("stack4", "c64", [synth.Item(A, B, "N", 1.0, 0.0)], False, seed=65))
    return out


def random_stack_case(seed):
    """A random ScaLAPACK-descriptor pair whose row walks stack: 2 x 2 grids,
    source blocks of 128-512 bytes of rows inside 128-row target blocks whose
    first process row is the other one, random sizes and padded leading
    dimensions (odd pads: single-element units), element type by seed, beta
    0 for even seeds (stacks on both sides) and 0.5 for odd ones."""
    rng = np.random.default_rng(1000 + seed)
    SL = synth.ScaLapack
    dtype = ["f64", "f32", "c128", "c64"][seed % 4]
    es = synth.ITEMSIZE[dtype]
    mb = int(rng.choice([128, 256, 512])) // es
    m = int(rng.integers(1600, 2600))
    n = int(rng.integers(8, 90))

    def lld(mm, b):
        return -(-(-(-mm // b)) // 2) * b + int(rng.integers(1, 9))
    B = SL(m, n, mb, mb, 0, 0, lld(m, mb), 2, 2)
    A = SL(m, n, 128, 128, 1, 0, lld(m, 128), 2, 2)
    beta = 0.0 if seed % 2 == 0 else 0.5
    return synth.Workload(f"rs{seed}", dtype, [synth.Item(A, B, "N", 1.0 if seed % 3 else 2.0, beta)], False,
                          seed=300 + seed)


def long_stack_case():
    """Local columns of 70,000 rows cut into 16-row source blocks (128 bytes
    of fp64), 3 columns: stacks longer than the 4096 rectangles a stack may
    hold, so the planner cuts them."""
    SL = synth.ScaLapack
    m = 2 * 70000

    def lld(mm, b):
        return -(-(-(-mm // b)) // 2) * b + 3
    B = SL(m, 3, 16, 16, 0, 0, lld(m, 16), 2, 1)
    A = SL(m, 3, 128, 128, 1, 0, lld(m, 128), 2, 1)
    return synth.Workload("long_stack", "f64", [synth.Item(A, B, "N", 1.0, 0.0)], False, seed=77)
