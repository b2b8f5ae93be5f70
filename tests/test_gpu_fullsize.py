"""Parity at the full 100M-rating, K=128 size in the launch configuration bench.py times.

The oracle cannot run whole clocks of this workload in test time, so it computes sampled
rows one by one: the rows of version 1 (every worker reads version 0 at clock 0, so any
policy and any s) and, under SSP_WORST at s = 7, the rows of version 8 (clocks 0..7 all
read version 0).  The loss at version 0 is compared in full.
"""
import sys

import numpy as np
import pytest

import oracle
from paper_1410_8043_amd import synth

pytestmark = pytest.mark.gpu

FACTOR_TOL = 1e-4
LOSS_RTOL = 1e-5


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def full():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    spec = synth.CONFIGS["full"]
    say("full-size: generating the 100M-rating workload")
    w = synth.generate(spec)
    ud = np.bincount(w.user, minlength=spec.N)
    idg = np.bincount(w.item, minlength=spec.M)
    rng = np.random.default_rng(2024)
    order_u = np.argsort(-ud, kind="stable")
    order_i = np.argsort(-idg, kind="stable")
    users = np.unique(np.concatenate([order_u[:16], order_u[-16:], rng.choice(spec.N, 96, replace=False)]))
    items = np.unique(np.concatenate([order_i[:16], order_i[-16:], rng.choice(spec.M, 48, replace=False)]))
    say("full-size: oracle load (canonical sort of 100M ratings)")
    o = oracle.Oracle(spec.N, spec.M, spec.K, spec.P, 7, spec.eta, spec.lam, oracle.SSP_WORST, oracle.ROWMEAN,
                      spec.B, spec.seed)
    o.load(w.user, w.item, w.val)
    o.set_factors(w.L0, w.R0)
    yield spec, w, o, users, items
    o.close()


def gpu_handle(spec, w, s, policy):
    import torch

    from paper_1410_8043_amd import ps_mf

    g = ps_mf.PsMf(spec.N, spec.M, spec.K, spec.P, s, spec.eta, spec.lam, policy=policy, B=spec.B,
                   mb_seed=spec.seed, stream=torch.cuda.current_stream())
    g.load_ratings(w.user, w.item, w.val)
    g.set_factors(w.L0, w.R0)
    return g


@pytest.mark.timeout(1800)
@pytest.mark.parametrize("s", [0, 1, 3, 7])
def test_full_config_first_clock_sampled_rows(full, s):
    spec, w, o, users, items = full
    Lo, Ro = o.rows_from_v0(1, users, items)
    say(f"full-size: s={s} SSP_LAZY, one clock")
    g = gpu_handle(spec, w, s, 0)
    try:
        if s == 0:
            lg, lo = g.loss(), o.loss()
            assert abs(lg - lo) <= LOSS_RTOL * lo, (lg, lo)
        g.clock(1)
        L, R = g.get_version(1)
    finally:
        g.close()
    err = max(np.abs(L[users] - Lo).max(), np.abs(R[items] - Ro).max())
    say(f"full-size: s={s} max |GPU - oracle| over {users.size} users and {items.size} items = {err:.3e}")
    assert err <= FACTOR_TOL


@pytest.mark.timeout(1800)
def test_full_config_worst_s7_eight_clocks_sampled_rows(full):
    spec, w, o, users, items = full
    Lo, Ro = o.rows_from_v0(8, users, items)
    say("full-size: s=7 SSP_WORST, eight clocks")
    g = gpu_handle(spec, w, 7, 1)
    try:
        g.clock(8)
        L, R = g.get_version(8)
        from paper_1410_8043_amd import ps_mf
        log = g.export_index(ps_mf.IDX_VERSION_LOG).reshape(8, spec.P)
    finally:
        g.close()
    assert np.all(log == 0)
    err = max(np.abs(L[users] - Lo).max(), np.abs(R[items] - Ro).max())
    say(f"full-size: WORST s=7 after 8 clocks max |GPU - oracle| = {err:.3e}")
    assert err <= FACTOR_TOL
