"""Pins of the CPU oracle against what the paper and the mathematics fix (no GPU).

Each test checks the oracle against something other than itself: hand-worked values,
finite differences of the objective, a dense brute force of a different code shape,
closed-form invariants, and the published SplitMix64 output sequence.
"""
import numpy as np
import pytest

import oracle
from dense_ref import block_of, loss_dense, run_dense, splitmix64
from golden_cases import load_cases
from paper_1410_8043_amd import synth


def rand_problem(rng, N, M, nnz, K, dup=0, scale=0.3):
    cells = rng.choice(N * M, size=nnz, replace=False)
    user = (cells // M).astype(np.int32)
    item = (cells % M).astype(np.int32)
    if dup:
        extra = rng.integers(0, nnz, size=dup)
        user = np.concatenate([user, user[extra]])
        item = np.concatenate([item, item[extra]])
    perm = rng.permutation(user.shape[0])
    user, item = user[perm], item[perm]
    val = rng.integers(1, 6, size=user.shape[0]).astype(np.float32)
    L0 = (scale * rng.standard_normal((N, K))).astype(np.float32)
    R0 = (scale * rng.standard_normal((M, K))).astype(np.float32)
    return user, item, val, L0, R0


# ---------------------------------------------------------------- hand-worked values
@pytest.mark.parametrize("case", load_cases(), ids=lambda c: c["name"])
def test_hand_examples(case):
    u = np.array([r[0] for r in case["ratings"]], np.int32)
    i = np.array([r[1] for r in case["ratings"]], np.int32)
    v = np.array([r[2] for r in case["ratings"]], np.float32)
    o = oracle.Oracle(case["N"], case["M"], case["K"], case["P"], case["s"], case["eta"], case["lam"],
                      case["policy"], case["step"], 1, 0, case["owner"])
    o.load(u, i, v)
    o.set_factors(case["L0"], case["R0"])
    for ex in sorted(case["expect"], key=lambda e: e["clock"]):
        o.clock(ex["clock"] - o.clock_value)
        L, R = o.get_factors()
        np.testing.assert_allclose(L.ravel(), ex["L"], atol=1e-6, rtol=0)
        np.testing.assert_allclose(R.ravel(), ex["R"], atol=1e-6, rtol=0)
        if ex["loss"] is not None:
            assert abs(o.loss() - ex["loss"]) <= 1e-5 * abs(ex["loss"])


# ---------------------------------------------------------------- SplitMix64
def test_splitmix64_published_sequence():
    # the first outputs of SplitMix64 seeded with 0, as published with its reference code
    expected = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    st = 0
    got = []
    for _ in range(3):
        got.append(oracle.splitmix64(st))
        st = (st + 0x9E3779B97F4A7C15) & ((1 << 64) - 1)
    assert got == expected
    assert synth.splitmix64_sequence(0, 3) == expected
    assert [splitmix64(x) for x in (0, 0x9E3779B97F4A7C15)] == expected[:2]


# ---------------------------------------------------------------- finite differences
def objective(user, item, val, L, R, lam):
    """F_w = 1/2 sum over ratings of (r - L_i.R_j)^2 + lambda(|L_i|^2 + |R_j|^2), fp64."""
    L = L.astype(np.float64)
    R = R.astype(np.float64)
    tot = 0.0
    for t in range(len(user)):
        li, rj = L[user[t]], R[item[t]]
        e = float(val[t]) - li @ rj
        tot += 0.5 * (e * e + lam * (li @ li + rj @ rj))
    return tot


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_update_is_minus_eta_times_finite_difference_gradient(seed):
    rng = np.random.default_rng(seed)
    N, M, K, lam, eta = 5, 6, 3, 0.3, 0.25
    user, item, val, L0, R0 = rand_problem(rng, N, M, 14, K, dup=2)
    # exactly representable inputs keep the fp32 rounding of the new version tiny
    L0 = (np.round(L0 * 64) / 64).astype(np.float32)
    R0 = (np.round(R0 * 64) / 64).astype(np.float32)
    o = oracle.Oracle(N, M, K, 1, 0, eta, lam, oracle.SSP_LAZY, oracle.SUM)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    o.clock(1)
    L1, R1 = o.get_factors()
    h = 1e-6
    gL = np.zeros((N, K))
    gR = np.zeros((M, K))
    for a in range(N):
        for k in range(K):
            Lp = L0.astype(np.float64).copy(); Lp[a, k] += h
            Lm = L0.astype(np.float64).copy(); Lm[a, k] -= h
            gL[a, k] = (objective(user, item, val, Lp, R0, lam) - objective(user, item, val, Lm, R0, lam)) / (2 * h)
    for a in range(M):
        for k in range(K):
            Rp = R0.astype(np.float64).copy(); Rp[a, k] += h
            Rm = R0.astype(np.float64).copy(); Rm[a, k] -= h
            gR[a, k] = (objective(user, item, val, L0, Rp, lam) - objective(user, item, val, L0, Rm, lam)) / (2 * h)
    stepL = (L1.astype(np.float64) - L0) / (-eta)
    stepR = (R1.astype(np.float64) - R0) / (-eta)
    scale = max(np.abs(gL).max(), np.abs(gR).max())
    assert np.abs(stepL - gL).max() <= 2e-6 * scale * 10
    assert np.abs(stepR - gR).max() <= 2e-6 * scale * 10


# ---------------------------------------------------------------- dense brute force
@pytest.mark.parametrize("step", [oracle.ROWMEAN, oracle.SUM])
@pytest.mark.parametrize("B", [1, 3])
def test_full_batch_gd_matches_dense(step, B):
    rng = np.random.default_rng(10 + B + 7 * step)
    N, M, K = 9, 7, 4
    user, item, val, L0, R0 = rand_problem(rng, N, M, 30, K, dup=3)
    kw = dict(N=N, M=M, K=K, P=1, s=0, eta=0.05, lam=0.1, clocks=5, step=step, B=B, seed=1234)
    hist = run_dense(user, item, val, L0, R0, **kw)
    o = oracle.Oracle(N, M, K, 1, 0, 0.05, 0.1, oracle.SSP_LAZY, step, B, 1234)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    for c in range(1, 6):
        o.clock(1)
        L, R = o.get_factors()
        np.testing.assert_allclose(L, hist[c][0], atol=1e-6, rtol=0)
        np.testing.assert_allclose(R, hist[c][1], atol=1e-6, rtol=0)


@pytest.mark.parametrize("policy", [oracle.SSP_LAZY, oracle.SSP_WORST, oracle.ESSP])
@pytest.mark.parametrize("s", [1, 2, 3])
@pytest.mark.parametrize("P", [1, 3])
def test_delayed_gd_matches_dense(policy, s, P):
    rng = np.random.default_rng(100 * s + 10 * P + policy)
    N, M, K = 8, 6, 3
    user, item, val, L0, R0 = rand_problem(rng, N, M, 25, K)
    owner = rng.integers(0, P, size=N).astype(np.int32)
    kw = dict(N=N, M=M, K=K, P=P, s=s, eta=0.05, lam=0.05, clocks=7, policy=policy, step=oracle.ROWMEAN,
              owner=owner)
    hist = run_dense(user, item, val, L0, R0, **kw)
    o = oracle.Oracle(N, M, K, P, s, 0.05, 0.05, policy, oracle.ROWMEAN, 1, 0, owner)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    o.clock(7)
    L, R = o.get_factors()
    np.testing.assert_allclose(L, hist[7][0], atol=1e-6, rtol=0)
    np.testing.assert_allclose(R, hist[7][1], atol=1e-6, rtol=0)
    # the ring still holds versions clock-s .. clock
    for v in range(7 - s, 8):
        Lv, Rv = o.get_version(v)
        np.testing.assert_allclose(Lv, hist[v][0], atol=1e-6, rtol=0)


def test_p1_lazy_is_delay_c_mod_s_plus_1():
    """At P=1, SSP_LAZY reads version c - (c mod (s+1)): check the recurrence directly."""
    rng = np.random.default_rng(5)
    N, M, K, s = 6, 5, 2, 2
    user, item, val, L0, R0 = rand_problem(rng, N, M, 15, K)
    hist = run_dense(user, item, val, L0, R0, N=N, M=M, K=K, P=1, s=s, eta=0.1, lam=0.05, clocks=6,
                     policy=oracle.SSP_WORST, step=oracle.SUM)
    o = oracle.Oracle(N, M, K, 1, s, 0.1, 0.05, oracle.SSP_LAZY, oracle.SUM)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    for c in range(6):
        assert o.view_version(0, c) == c - (c % (s + 1))
    # clocks 0..2 read v0 under both policies; at clock 3 LAZY reads v3, WORST reads v1
    o.clock(3)
    L3, _ = o.get_factors()
    assert np.array_equal(L3, hist[3][0])
    o.clock(1)
    L4, _ = o.get_factors()
    assert not np.allclose(L4, hist[4][0], atol=1e-7)
    lazy = run_dense(user, item, val, L0, R0, N=N, M=M, K=K, P=1, s=s, eta=0.1, lam=0.05, clocks=6,
                     policy=oracle.SSP_LAZY, step=oracle.SUM)
    o.clock(2)
    np.testing.assert_allclose(o.get_factors()[0], lazy[6][0], atol=1e-6, rtol=0)


# ---------------------------------------------------------------- invariants
def test_sharding_invariance_at_s0_is_bit_exact():
    rng = np.random.default_rng(7)
    N, M, K = 40, 30, 8
    user, item, val, L0, R0 = rand_problem(rng, N, M, 300, K)
    ref = None
    for P, owner in [(1, None), (4, None), (7, rng.integers(0, 7, size=N)), (40, rng.permutation(N))]:
        for policy in (oracle.SSP_LAZY, oracle.SSP_WORST, oracle.ESSP):
            L, R, loss, _ = oracle.run(user, item, val, L0, R0, N=N, M=M, K=K, P=P, s=0, eta=0.05, lam=0.05,
                                       clocks=4, policy=policy, owner=owner)
            if ref is None:
                ref = (L, R, loss)
            assert np.array_equal(L, ref[0]) and np.array_equal(R, ref[1]) and loss == ref[2]


def test_essp_is_identical_for_every_s_at_least_1():
    rng = np.random.default_rng(8)
    N, M, K = 30, 20, 4
    user, item, val, L0, R0 = rand_problem(rng, N, M, 200, K)
    outs = [oracle.run(user, item, val, L0, R0, N=N, M=M, K=K, P=5, s=s, eta=0.05, lam=0.05, clocks=6,
                       policy=oracle.ESSP)[:3] for s in (1, 3, 7)]
    for L, R, loss in outs[1:]:
        assert np.array_equal(L, outs[0][0]) and np.array_equal(R, outs[0][1]) and loss == outs[0][2]
    worst = oracle.run(user, item, val, L0, R0, N=N, M=M, K=K, P=5, s=1, eta=0.05, lam=0.05, clocks=6,
                       policy=oracle.SSP_WORST)
    assert np.array_equal(worst[0], outs[0][0]) and np.array_equal(worst[1], outs[0][1])


@pytest.mark.parametrize("step", [oracle.ROWMEAN, oracle.SUM])
def test_descent_on_noiseless_planted_data(step):
    rng = np.random.default_rng(9)
    N, M, k, K = 30, 25, 2, 4
    U = rng.standard_normal((N, k))
    V = rng.standard_normal((M, k))
    cells = rng.choice(N * M, size=400, replace=False)
    user = (cells // M).astype(np.int32)
    item = (cells % M).astype(np.int32)
    val = np.einsum("tk,tk->t", U[user], V[item]).astype(np.float32)
    L0 = (0.3 * rng.standard_normal((N, K))).astype(np.float32)
    R0 = (0.3 * rng.standard_normal((M, K))).astype(np.float32)
    eta = 0.01 if step == oracle.SUM else 0.2
    o = oracle.Oracle(N, M, K, 3, 0, eta, 0.0, oracle.SSP_LAZY, step)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    losses = [o.loss()]
    for _ in range(40):
        o.clock(1)
        losses.append(o.loss())
    assert all(b < a for a, b in zip(losses, losses[1:]))
    assert losses[-1] < 0.5 * losses[0]


@pytest.mark.parametrize("policy", [oracle.SSP_LAZY, oracle.SSP_WORST, oracle.ESSP])
@pytest.mark.parametrize("s", [0, 1, 3, 7])
def test_version_bound_invariant(policy, s):
    rng = np.random.default_rng(11)
    N, M, K, P, T = 20, 10, 2, 6, 20
    user, item, val, L0, R0 = rand_problem(rng, N, M, 60, K)
    o = oracle.Oracle(N, M, K, P, s, 0.01, 0.05, policy)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    o.clock(T)
    log = o.export(oracle.X_VERSION_LOG).reshape(T, P)
    for c in range(T):
        assert np.all(log[c] >= max(0, c - s)) and np.all(log[c] <= c)
    if policy == oracle.SSP_WORST:
        assert np.all(log == np.maximum(0, np.arange(T) - s)[:, None])
    if policy == oracle.ESSP:
        assert np.all(log == np.maximum(0, np.arange(T) - min(s, 1))[:, None])
    if policy == oracle.SSP_LAZY and s > 0:
        # staleness is spread over 0..s once the ring is full
        d = np.arange(T)[:, None] - log
        assert set(np.unique(d[s:])) == set(range(s + 1))


def test_loss_matches_dense_sum():
    rng = np.random.default_rng(12)
    N, M, K = 50, 40, 6
    user, item, val, L0, R0 = rand_problem(rng, N, M, 500, K, dup=5)
    L, R, loss, _ = oracle.run(user, item, val, L0, R0, N=N, M=M, K=K, P=3, s=2, eta=0.05, lam=0.05, clocks=3)
    ref = loss_dense(user, item, val, L, R)
    assert abs(loss - ref) <= 1e-12 * ref


# ---------------------------------------------------------------- integer layout
@pytest.mark.parametrize("B", [1, 4])
def test_layout_against_brute_force(B):
    rng = np.random.default_rng(13)
    N, M, K, P = 60, 45, 2, 5
    user, item, val, L0, R0 = rand_problem(rng, N, M, 800, K, dup=10)
    seed = 0x14108043
    o = oracle.Oracle(N, M, K, P, 0, 0.01, 0.05, oracle.SSP_LAZY, oracle.ROWMEAN, B, seed)
    o.load(user, item, val)
    assert np.array_equal(o.export(oracle.X_OWNER), np.arange(N) % P)
    blocks = np.array([block_of(i, j, seed, B) for i, j in zip(user, item)])
    total = 0
    for b in range(B):
        sel = np.nonzero(blocks == b)[0]
        ucnt = np.bincount(user[sel], minlength=N)
        icnt = np.bincount(item[sel], minlength=M)
        assert np.array_equal(o.export(oracle.X_USER_COUNT, b), ucnt)
        assert np.array_equal(o.export(oracle.X_ITEM_COUNT, b), icnt)
        rp = o.export(oracle.X_ROW_PTR, b)
        assert rp[0] == 0 and np.array_equal(np.diff(rp), ucnt)
        perm = o.export(oracle.X_PERM, b)
        col = o.export(oracle.X_COL, b)
        # canonical order: sorted by (user, item, load index), a permutation of the block
        expect = sel[np.lexsort((sel, item[sel], user[sel]))]
        assert np.array_equal(perm, expect)
        assert np.array_equal(col, item[perm])
        total += sel.size
    assert total == user.shape[0]


def test_rows_from_v0_matches_full_clocks():
    rng = np.random.default_rng(14)
    N, M, K, s = 40, 30, 4, 3
    user, item, val, L0, R0 = rand_problem(rng, N, M, 300, K)
    o = oracle.Oracle(N, M, K, 4, s, 0.05, 0.05, oracle.SSP_WORST)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    us = np.array([0, 5, 17, 39])
    its = np.array([1, 2, 29])
    Ls, Rs = o.rows_from_v0(s + 1, us, its)
    o.clock(s + 1)
    L, R = o.get_factors()
    assert np.array_equal(Ls, L[us]) and np.array_equal(Rs, R[its])
    with pytest.raises(oracle.OracleError):
        o2 = oracle.Oracle(N, M, K, 4, s, 0.05, 0.05, oracle.SSP_LAZY)
        o2.load(user, item, val)
        o2.set_factors(L0, R0)
        o2.rows_from_v0(2, us, its)


def test_argument_errors():
    with pytest.raises(oracle.OracleError):
        oracle.Oracle(0, 1, 1, 1, 0, 0.1, 0.1)
    with pytest.raises(oracle.OracleError):
        oracle.Oracle(1, 1, 1, 1, -1, 0.1, 0.1)
    o = oracle.Oracle(2, 2, 1, 1, 0, 0.1, 0.1)
    with pytest.raises(oracle.OracleError):
        o.load(np.array([2]), np.array([0]), np.array([1.0]))
    with pytest.raises(oracle.OracleError):
        o.clock(1)
