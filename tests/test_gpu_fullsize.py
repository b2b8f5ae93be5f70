"""Parity at the full 100M-rating, K=128 size in the launch configuration bench.py times.

The oracle cannot run whole clocks of this workload in test time, so it computes sampled
rows one by one: the rows of version 1 (every worker reads version 0 at clock 0, so any
policy and any s) and, under SSP_WORST at s = 7, the rows of version 8 (clocks 0..7 all
read version 0).  The loss at version 0 is compared in full.  The sequential step's user
rows of version 1 come from single-worker oracles (a worker's chain depends only on its
own ratings and the view), and the value-bounded views are checked by properties that
hold at any size.
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


def gpu_handle(spec, w, s, policy, **opts):
    import torch

    from paper_1410_8043_amd import ps_mf

    g = ps_mf.PsMf(spec.N, spec.M, spec.K, spec.P, s, spec.eta, spec.lam, policy=policy, B=spec.B,
                   mb_seed=spec.seed, stream=torch.cuda.current_stream(), **opts)
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


@pytest.mark.timeout(1800)
def test_full_config_seq_first_clock_user_rows_of_two_workers(full):
    """STEP_SEQ as bench.py --step seq runs it (256 sub-epochs).  At clock 0 every worker
    starts from version 0, and its users' rows of version 1 are its own chain's result.  The
    chain of worker p is rebuilt by a P = 1 oracle holding only p's ratings, with user
    i = p + P k renumbered k: user groups (i div P) mod G and item groups are unchanged, so
    the order is the same."""
    from paper_1410_8043_amd import ps_mf

    spec, w, _, _, _ = full
    per_worker = np.bincount(w.user % spec.P, minlength=spec.P)
    workers = [int(np.argmax(per_worker)), 5]
    say(f"full-size: SEQ, one clock; workers {workers} ({per_worker[workers].tolist()} ratings)")
    g = gpu_handle(spec, w, 3, 0, step=ps_mf.STEP_SEQ)
    try:
        g.clock(1)
        L, _ = g.get_version(1)
    finally:
        g.close()
    for p in workers:
        sel = (w.user % spec.P) == p
        Np = (spec.N - p + spec.P - 1) // spec.P
        o = oracle.Oracle(Np, spec.M, spec.K, 1, 3, spec.eta, spec.lam, oracle.SSP_LAZY, oracle.SEQ, strata=256)
        o.load(w.user[sel] // spec.P, w.item[sel], w.val[sel])
        o.set_factors(w.L0[p::spec.P], w.R0)
        o.clock(1)
        Lo, _ = o.get_factors()
        o.close()
        err = np.abs(L[p::spec.P] - Lo).max()
        say(f"full-size: SEQ worker {p}: max |GPU - oracle| over its {Np} user rows = {err:.3e}")
        assert err <= FACTOR_TOL


@pytest.mark.timeout(1800)
def test_full_config_vap_limits_and_norms(full):
    """PS_MF_VAP with no bound reads exactly what SSP_WORST reads, bit for bit; the exported
    in-transit norms are the max-norms of the GPU's own versions; with a bound, every
    chosen view is the stalest whose norm fits it."""
    from paper_1410_8043_amd import ps_mf

    spec, w, _, _, _ = full
    say("full-size: VAP unbounded vs SSP_WORST, s=3, four clocks")
    g = gpu_handle(spec, w, 3, ps_mf.VAP, value_bound=float("inf"))
    h = gpu_handle(spec, w, 3, ps_mf.SSP_WORST)
    try:
        g.clock(4)
        h.clock(4)
        Lg, Rg = g.get_factors()
        Lh, Rh = h.get_factors()
        assert np.array_equal(Lg, Lh) and np.array_equal(Rg, Rh)
        assert np.array_equal(g.export_index(ps_mf.IDX_VERSION_LOG), h.export_index(ps_mf.IDX_VERSION_LOG))
        norms = g.export_index(ps_mf.IDX_VAP_NORMS).reshape(4, 4)
        x3, x2, x1 = (g.get_version(v) for v in (3, 2, 1))
        for d, xo in ((1, x2), (2, x1)):
            want = max(np.abs(x3[0] - xo[0]).max(), np.abs(x3[1] - xo[1]).max())
            assert norms[3, d] == want, (d, norms[3, d], want)
    finally:
        g.close()
        h.close()
    v0 = 0.003
    say(f"full-size: VAP v0={v0}, s=3, fifteen clocks")
    g = gpu_handle(spec, w, 3, ps_mf.VAP, value_bound=v0)
    try:
        g.clock(15)
        vlog = g.export_index(ps_mf.IDX_VERSION_LOG).reshape(15, spec.P)
        norms = g.export_index(ps_mf.IDX_VAP_NORMS).reshape(15, 4)
        loss = g.loss()
    finally:
        g.close()
    assert np.all(vlog == vlog[:, :1])
    d = np.arange(15) - vlog[:, 0]
    say(f"full-size: VAP delays {d.tolist()}")
    for c in range(15):
        bound = v0 / np.sqrt(c + 1.0)
        fits = [k for k in range(min(c, 3) + 1) if k == 0 or norms[c, k] <= bound]
        assert d[c] == max(fits)
    assert len(set(d[4:].tolist())) > 1 and np.isfinite(loss)
