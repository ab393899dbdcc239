"""costa_transform_batched_noalloc against costa_transform_batched (GPU).

The allocation-free entry point keeps its plan tables and message buffers in
the library's static scratch array.  Each case runs both entry points on the
same seeded inputs (two copies of A with the same initial contents) and
compares every element bit for bit; consecutive calls change the plan the
scratch array holds (a large plan in many waves, then smaller ones, then the
first again with other buffers).
"""
import pytest
import torch

import synth
from parity import Case, lib
from replay import stack_cases

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _bytes(t):
    return t.contiguous().view(torch.uint8)


class Twin:
    """A workload on the device with a second copy of A for the no-allocation call."""

    def __init__(self, name, size=None):
        if isinstance(name, synth.Workload):
            self.w = name
        else:
            self.w = synth.workload(name, size) if size else synth.workload(name)
        self.case = Case(self.w)
        self.A2 = [[a.clone() for a in ak] for ak in self.case.A]

    def descs(self, A):
        c = self.case
        return [dict(op=it.op, alpha=it.alpha, beta=it.beta, A=c.LA[k], A_local=A[k], B=c.LB[k], B_local=c.B[k])
                for k, it in enumerate(self.w.items)]

    def run_and_compare(self):
        C = lib()
        c = self.case
        s = c.stream
        C.costa_transform_batched(self.w.dtype, self.descs(c.A), c.sigma, s)
        C.costa_transform_batched_noalloc(self.w.dtype, self.descs(self.A2), c.sigma, s)
        torch.cuda.synchronize()
        for k in range(len(self.w.items)):
            for r in range(c.P):
                a, b = c.A[k][r], self.A2[k][r]
                assert torch.equal(_bytes(a), _bytes(b)), f"{self.w.name} pair {k} rank {r} differs"

    def reset_a(self):
        """Both copies of A back to the seeded initial values."""
        self.case.fill()
        for ak, bk in zip(self.case.A, self.A2):
            for a, b in zip(ak, bk):
                b.copy_(a)
        torch.cuda.synchronize()

    def free(self):
        self.A2 = None
        self.case.free()


def test_noalloc_matches_the_allocating_entry_point():
    C = lib()
    # 1) the block-size change at full size: 1.6 GB of messages, many waves of
    #    the scratch array's message area; relabeling on
    _say("noalloc: blocksize_change_16k full size")
    big = Twin("blocksize_change_16k")
    stats = C.costa_plan_stats(big.w.dtype, big.descs(big.case.A), big.case.sigma)
    assert stats["message_bytes"] > C.NOALLOC_SCRATCH_BYTES  # needs several waves there
    big.run_and_compare()
    # 2) a smaller input right after it: the scaled transpose (alpha = 2,
    #    beta = 0.5: A is read) at reduced size, then the 1024^2 transpose
    #    with relabeling and the tall-skinny batch (mixed ops) at reduced size
    #    and two layouts whose row walks stack (fp64 and single-element
    #    float units)
    for name, size in (("scaled_transpose_20k", "small"), ("reshuffle_transpose_1k", None),
                       ("rpa_batched_tall_skinny", "small"), (stack_cases()[0], None), (stack_cases()[2], None)):
        _say(f"noalloc: {getattr(name, 'name', name)} {size or 'full size'}")
        t = Twin(name, size)
        t.run_and_compare()
        t.run_and_compare()  # the same plan again: tables already resident
        t.free()
    # 3) the first plan again, on new buffers (its tables and call table are
    #    uploaded again)
    _say("noalloc: blocksize_change_16k again, new buffers")
    big.free()
    big = Twin("blocksize_change_16k")
    big.run_and_compare()
    big.free()
