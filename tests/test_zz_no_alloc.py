"""ps_mf_loss_noalloc -- the loss for callers that cannot allocate device memory, with its
partial sums in a fixed static array -- against the allocating ps_mf_loss and the oracle,
through the C ABI (MI355X).

Two calls in a row on two handles, the second with a smaller input, so the second call
finds the first one's partial sums in the shared array and must not use them.
"""
import sys

import numpy as np
import pytest

import oracle
from paper_1410_8043_amd import synth

pytestmark = pytest.mark.gpu

LOSS_RTOL = 1e-5


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def test_noalloc_loss_matches_the_allocating_loss_twice():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_1410_8043_amd import ps_mf

    cases = [(synth.scaled(synth.CONFIGS["full"], 0.05), 128, 3), (synth.scaled(synth.CONFIGS["medium"], 0.02), 33, 1)]
    parts = []
    for spec, K, s in cases:
        w = synth.generate(spec, K=K)
        say(f"no-alloc loss: {spec.name} N={spec.N} M={spec.M} nnz={w.nnz} K={K} P={spec.P} s={s} B={spec.B}")
        with ps_mf.PsMf(spec.N, spec.M, K, spec.P, s, spec.eta, spec.lam, B=spec.B, mb_seed=spec.seed,
                        stream=torch.cuda.current_stream()) as g:
            g.load_ratings(w.user, w.item, w.val)
            g.set_factors(w.L0, w.R0)
            g.clock(3)
            got = ps_mf.ps_mf_loss_noalloc(g.h)
            want = g.loss()
            again = ps_mf.ps_mf_loss_noalloc(g.h)
        parts.append(w.nnz)
        _, _, ref, o = oracle.run(w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=K, P=spec.P, s=s,
                                  eta=spec.eta, lam=spec.lam, clocks=3, B=spec.B, seed=spec.seed)
        o.close()
        say(f"no-alloc loss: {got!r} allocating: {want!r} oracle: {ref!r}")
        # the same kernels sum the same partials in the same fixed order
        assert got == want and again == got
        assert abs(got - ref) <= LOSS_RTOL * ref
    assert parts[1] < parts[0]
