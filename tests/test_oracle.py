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
                      case["policy"], case["step"], 1, 0, case["owner"], strata=case["strata"],
                      value_bound=case["v0"])
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


# ---------------------------------------------------------------- staleness profile (Fig. 1 left)
def staleness_run(policy, s, P, clocks, B=1, seed=0, owner=None, N=40, M=30, nnz=600):
    rng = np.random.default_rng(seed)
    user, item, val, L0, R0 = rand_problem(rng, N, M, nnz, 4)
    o = oracle.Oracle(N, M, 4, P, s, 0.01, 0.05, policy, oracle.ROWMEAN, B, 7, owner)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    o.clock(clocks)
    hist = o.export(oracle.X_STALENESS)
    o.close()
    return hist, user, item


@pytest.mark.parametrize("policy", [oracle.SSP_LAZY, oracle.SSP_WORST, oracle.ESSP])
def test_staleness_bsp_is_always_minus_one(policy):
    # Fig. 1 caption: on a BSP system the clock differential is always -1 (s = 0)
    hist, user, _ = staleness_run(policy, 0, 3, 5)
    assert hist.tolist() == [2 * user.size * 5]


@pytest.mark.parametrize("s", [1, 3, 7])
def test_staleness_essp_is_one_clock_regardless_of_s(s):
    # Section 4: reads observe staleness 1 regardless of s; clock 0 can only read version 0
    hist, user, _ = staleness_run(oracle.ESSP, s, 4, 9)
    want = np.zeros(s + 1, np.int64)
    want[0] = 2 * user.size
    want[1] = 2 * user.size * 8
    assert np.array_equal(hist, want)


@pytest.mark.parametrize("s", [1, 2, 4])
def test_staleness_worst_is_the_guaranteed_prewindow(s):
    # Section 3.2: the view holds every update of clocks <= c-s-1 and none of the window;
    # before clock s the view is version 0
    clocks = 2 * s + 3
    hist, user, _ = staleness_run(oracle.SSP_WORST, s, 5, clocks)
    want = np.zeros(s + 1, np.int64)
    for c in range(clocks):
        want[min(c, s)] += 2 * user.size
    assert np.array_equal(hist, want)


@pytest.mark.parametrize("s", [1, 3])
def test_staleness_lazy_is_uniform_in_steady_state(s):
    # Section 2.2: under SSP the distribution of clock differentials is (nearly) uniform.
    # P = s+1 workers with one user each and equal shards: every full period of s+1 clocks
    # after the first s adds the same count to every delay 0..s
    P = s + 1
    N, M = P, 50
    user = np.repeat(np.arange(P, dtype=np.int32), M)
    item = np.tile(np.arange(M, dtype=np.int32), P)
    val = np.ones(user.size, np.float32)
    rng = np.random.default_rng(1)
    L0 = (0.1 * rng.standard_normal((N, 4))).astype(np.float32)
    R0 = (0.1 * rng.standard_normal((M, 4))).astype(np.float32)

    def hist_after(clocks):
        o = oracle.Oracle(N, M, 4, P, s, 0.01, 0.05, oracle.SSP_LAZY, oracle.ROWMEAN, 1, 0)
        o.load(user, item, val)
        o.set_factors(L0, R0)
        o.clock(clocks)
        h = o.export(oracle.X_STALENESS)
        o.close()
        return h

    # each of the P workers reads its 2M rows once at every delay per period
    a, b = hist_after(s), hist_after(s + 3 * (s + 1))
    assert np.array_equal(b - a, np.full(s + 1, 3 * P * 2 * M, np.int64))


@pytest.mark.parametrize("policy", [oracle.SSP_LAZY, oracle.SSP_WORST, oracle.ESSP])
@pytest.mark.parametrize("B", [1, 3])
def test_staleness_counts_two_reads_per_processed_rating(policy, B):
    # every rating of the clock's block is processed once and reads two rows
    N, M, clocks = 40, 30, 7
    hist, user, item = staleness_run(policy, 3, 4, clocks, B=B)
    blocks = np.array([block_of(int(u), int(i), 7, B) for u, i in zip(user, item)])
    processed = sum(int((blocks == c % B).sum()) for c in range(clocks))
    assert hist.sum() == 2 * processed


# ---------------------------------------------------------------- per-row caches (Section 4)
@pytest.mark.parametrize("s", [1, 2, 3])
@pytest.mark.parametrize("P", [1, 3])
def test_ssp_row_with_every_row_read_each_clock_is_phase_zero_lazy(s, P):
    # B = 1: every client reads all of its rows at every clock, so every cached row is
    # fetched at clock 0 and refreshed together at s+1, 2(s+1), ...: the view of every read
    # is c - (c mod (s+1)), i.e. SSP_LAZY with every worker in phase 0 (all users on worker 0)
    rng = np.random.default_rng(10 * s + P)
    N, M, K = 30, 20, 3
    user, item, val, L0, R0 = rand_problem(rng, N, M, 300, K, dup=5)
    got = oracle.run(user, item, val, L0, R0, N=N, M=M, K=K, P=P, s=s, eta=0.05, lam=0.05, clocks=3 * s + 4,
                     policy=oracle.SSP_ROW)
    want = oracle.run(user, item, val, L0, R0, N=N, M=M, K=K, P=P, s=s, eta=0.05, lam=0.05, clocks=3 * s + 4,
                      policy=oracle.SSP_LAZY, owner=np.zeros(N, np.int32))
    assert np.array_equal(got[0], want[0]) and np.array_equal(got[1], want[1])


@pytest.mark.parametrize("s", [1, 3])
def test_essp_row_with_every_row_read_each_clock_is_essp(s):
    # B = 1: every row is first read at clock 0 (version 0), then pushed versions c - 1
    rng = np.random.default_rng(s)
    N, M, K = 30, 20, 3
    user, item, val, L0, R0 = rand_problem(rng, N, M, 300, K)
    got = oracle.run(user, item, val, L0, R0, N=N, M=M, K=K, P=4, s=s, eta=0.05, lam=0.05, clocks=7,
                     policy=oracle.ESSP_ROW)
    want = oracle.run(user, item, val, L0, R0, N=N, M=M, K=K, P=4, s=s, eta=0.05, lam=0.05, clocks=7,
                      policy=oracle.ESSP)
    assert np.array_equal(got[0], want[0]) and np.array_equal(got[1], want[1])


# W4: users 0, 1 on workers (and clients) 0, 1; ratings (0,0)=3 in block 0, (1,0)=1 and
# (0,1)=2 in block 1 (B = 2, seed 6), s = 1.  Versions read at each clock, by hand from
# the freshness rules: [user rows], [client 0's item rows], [client 1's item rows]
W4_VIEWS = {
    oracle.SSP_ROW: [([0, -1], [0, -1], [-1, -1]), ([0, 1], [-1, 1], [1, -1]),
                     ([2, -1], [2, -1], [-1, -1]), ([2, 3], [-1, 3], [3, -1])],
    oracle.ESSP_ROW: [([0, -1], [0, -1], [-1, -1]), ([0, 1], [-1, 1], [1, -1]),
                      ([1, -1], [1, -1], [-1, -1]), ([2, 2], [-1, 2], [2, -1])],
}
W4_CACHE_AFTER_4 = {oracle.SSP_ROW: [2, 3, 2, 3, 3, -1], oracle.ESSP_ROW: [2, 2, 1, 2, 2, -1]}
W4_STALENESS = {oracle.SSP_ROW: [10, 2], oracle.ESSP_ROW: [5, 7]}


@pytest.mark.parametrize("policy", [oracle.SSP_ROW, oracle.ESSP_ROW])
def test_per_row_hand_example_w4(policy):
    from dense_ref import run_dense_rowviews
    assert [block_of(0, 0, 6, 2), block_of(1, 0, 6, 2), block_of(0, 1, 6, 2)] == [0, 1, 1]
    user = np.array([0, 1, 0], np.int32)
    item = np.array([0, 0, 1], np.int32)
    val = np.array([3.0, 1.0, 2.0], np.float32)
    L0 = np.array([[0.5, -0.25], [0.25, 0.5]], np.float32)
    R0 = np.array([[1.0, 0.5], [0.75, -0.5]], np.float32)
    o = oracle.Oracle(2, 2, 2, 2, 1, 0.1, 0.05, policy, oracle.ROWMEAN, 2, 6)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    o.clock(4)
    assert o.export(oracle.X_ROW_VERSIONS).tolist() == W4_CACHE_AFTER_4[policy]
    assert o.export(oracle.X_STALENESS).tolist() == W4_STALENESS[policy]
    assert o.export(oracle.X_VERSION_LOG).size == 0
    views = [(vL, [v0, v1]) for vL, v0, v1 in W4_VIEWS[policy]]
    hist = run_dense_rowviews(user, item, val, L0, R0, N=2, M=2, K=2, P=2, C=2, eta=0.1, lam=0.05, views=views,
                              B=2, seed=6)
    L, R = o.get_factors()
    np.testing.assert_allclose(L, hist[4][0], rtol=0, atol=1e-6)
    np.testing.assert_allclose(R, hist[4][1], rtol=0, atol=1e-6)
    o.close()


@pytest.mark.parametrize("policy", [oracle.SSP_ROW, oracle.ESSP_ROW])
@pytest.mark.parametrize("s", [1, 3])
def test_per_row_staleness_stays_in_the_window(policy, s):
    # every read sees a version in [c - s, c]; ESSP_ROW reads are fresh (first reads) or
    # one clock old; every processed rating reads two rows
    N, M, clocks, B = 60, 40, 12, 4
    rng = np.random.default_rng(s)
    user, item, val, L0, R0 = rand_problem(rng, N, M, 900, 3)
    o = oracle.Oracle(N, M, 3, 5, s, 0.05, 0.05, policy, oracle.ROWMEAN, B, 9)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    o.clock(clocks)
    hist = o.export(oracle.X_STALENESS)
    cache = o.export(oracle.X_ROW_VERSIONS)
    o.close()
    blocks = np.array([block_of(int(u), int(i), 9, B) for u, i in zip(user, item)])
    assert hist.sum() == 2 * sum(int((blocks == c % B).sum()) for c in range(clocks))
    if policy == oracle.ESSP_ROW:
        assert hist[2:].sum() == 0 and hist[0] > 0 and hist[1] > 0
    else:
        assert hist[1:].sum() > 0  # intermittent reads keep rows cached across clocks
    assert cache.min() >= -1 and cache.max() <= clocks - 1


# ---------------------------------------------------------------- sequential steps inside a worker (SEQ)
def seq_order_by_definition(user, item, owner, P, G, B, seed):
    """Load indices of each block in the order the workers apply them, from the stated
    stratification: sub-epoch t = (j mod G - (i div P) mod G) mod G, then worker, user
    group, and canonical (user, item, load index) order."""
    blocks = np.array([block_of(int(u), int(i), seed, B) for u, i in zip(user, item)])
    out = []
    for b in range(B):
        idx = [t for t in range(user.size) if blocks[t] == b]
        key = lambda t: (((int(item[t]) % G) - (int(user[t]) // P) % G) % G, int(owner[user[t]]),
                         (int(user[t]) // P) % G, int(user[t]), int(item[t]), t)
        out.append(np.array(sorted(idx, key=key), np.int64))
    return out


@pytest.mark.parametrize("P,G,B", [(1, 1, 1), (1, 3, 1), (3, 2, 2), (4, 5, 3), (2, 64, 1)])
def test_seq_order_is_the_stratified_order(P, G, B):
    rng = np.random.default_rng(P * 100 + G)
    N, M = 23, 17
    user, item, val, L0, R0 = rand_problem(rng, N, M, 150, 2, dup=5)
    owner = rng.integers(0, P, size=N).astype(np.int32)
    o = oracle.Oracle(N, M, 2, P, 1, 0.01, 0.0, oracle.SSP_LAZY, oracle.SEQ, B, 11, owner, strata=G)
    o.load(user, item, val)
    want = seq_order_by_definition(user, item, owner, P, G, B, 11)
    for b in range(B):
        assert np.array_equal(o.export(oracle.X_SEQ_ORDER, b), want[b])
    o.close()


def matching_problem(rng, P, users_per_worker, M, K):
    """Every worker holds a matching: each of its users and each item at most once."""
    user, item = [], []
    for p in range(P):
        us = p + P * np.arange(users_per_worker)
        its = rng.choice(M, size=users_per_worker, replace=False)
        user += us.tolist()
        item += its.tolist()
    user, item = np.array(user, np.int32), np.array(item, np.int32)
    val = rng.integers(1, 6, size=user.size).astype(np.float32)
    N = P * users_per_worker
    L0 = (0.3 * rng.standard_normal((N, K))).astype(np.float32)
    R0 = (0.3 * rng.standard_normal((M, K))).astype(np.float32)
    return N, user, item, val, L0, R0


@pytest.mark.parametrize("policy,s", [(oracle.SSP_LAZY, 0), (oracle.SSP_LAZY, 2), (oracle.SSP_WORST, 1),
                                      (oracle.ESSP, 3)])
def test_seq_equals_sum_when_no_row_is_read_back(policy, s):
    # with a matching per worker no rating reads a row another rating of the same worker
    # wrote, so applying the ratings one by one is the summed step of the same view
    rng = np.random.default_rng(s + 10 * policy)
    P, M, K = 4, 9, 3
    N, user, item, val, L0, R0 = matching_problem(rng, P, 6, M, K)
    res = []
    for step in (oracle.SUM, oracle.SEQ):
        o = oracle.Oracle(N, M, K, P, s, 0.05, 0.1, policy, step, 1, 0, strata=4)
        o.load(user, item, val)
        o.set_factors(L0, R0)
        o.clock(6)
        res.append(o.get_factors() + (o.export(oracle.X_VERSION_LOG), o.export(oracle.X_STALENESS)))
        o.close()
    for a, b in zip(res[0][:2], res[1][:2]):
        np.testing.assert_allclose(a, b, rtol=1e-6, atol=1e-7)
    assert np.array_equal(res[0][2], res[1][2]) and np.array_equal(res[0][3], res[1][3])


@pytest.mark.parametrize("G,lam,dup", [(1, 0.0, 0), (1, 0.1, 4), (3, 0.05, 3), (7, 0.1, 0)])
def test_seq_p1_s0_clock_is_a_chain_of_single_rating_steps(G, lam, dup):
    # P = 1, s = 0: one SEQ clock applies the Section 3.1 rule once per rating, in the
    # stratified order, each step reading the previous one's result.  The same chain is
    # built from single-rating SUM clocks (each pinned by the closed form and finite
    # differences above), one fresh oracle per rating.
    rng = np.random.default_rng(G + dup)
    N, M, K, eta = 7, 6, 3, 0.05
    user, item, val, L0, R0 = rand_problem(rng, N, M, 25, K, dup=dup)
    o = oracle.Oracle(N, M, K, 1, 0, eta, lam, oracle.SSP_LAZY, oracle.SEQ, strata=G)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    o.clock(1)
    L_seq, R_seq = o.get_factors()
    order = o.export(oracle.X_SEQ_ORDER)
    o.close()
    assert np.array_equal(order, seq_order_by_definition(user, item, np.zeros(N, np.int32), 1, G, 1, 0)[0])
    L, R = L0.copy(), R0.copy()
    for t in order:
        one = oracle.Oracle(N, M, K, 1, 0, eta, lam, oracle.SSP_LAZY, oracle.SUM)
        one.load(user[t:t + 1], item[t:t + 1], val[t:t + 1])
        one.set_factors(L, R)
        one.clock(1)
        L, R = one.get_factors()
        one.close()
    # the chain rounds every step to fp32, the SEQ clock keeps the worker's copy in fp64
    np.testing.assert_allclose(L_seq, L, rtol=0, atol=2e-6)
    np.testing.assert_allclose(R_seq, R, rtol=0, atol=2e-6)


def test_seq_workers_commit_the_sum_of_their_own_chains():
    # s = 0, P = 3: each worker runs its chain from version c alone; the commit adds every
    # worker's (copy - view).  Each worker's chain is rebuilt by a P = 1 SEQ oracle that
    # holds only that worker's ratings, with the worker's users re-numbered so that they
    # keep their user groups.
    rng = np.random.default_rng(5)
    P, G, N, M, K, eta, lam = 3, 2, 12, 8, 2, 0.04, 0.05
    user, item, val, L0, R0 = rand_problem(rng, N, M, 60, K)
    o = oracle.Oracle(N, M, K, P, 0, eta, lam, oracle.SSP_LAZY, oracle.SEQ, strata=G)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    o.clock(1)
    L_all, R_all = o.get_factors()
    o.close()
    L_want, R_want = L0.astype(np.float64).copy(), R0.astype(np.float64).copy()
    for p in range(P):
        sel = (user % P) == p
        # user i = p + P k has user group k mod G; as user k of a P = 1 worker it keeps it
        Np = N // P
        one = oracle.Oracle(Np, M, K, 1, 0, eta, lam, oracle.SSP_LAZY, oracle.SEQ, strata=G)
        one.load(user[sel] // P, item[sel], val[sel])
        one.set_factors(L0[p::P], R0)
        one.clock(1)
        Lp, Rp = one.get_factors()
        one.close()
        L_want[p::P] = Lp
        R_want += Rp.astype(np.float64) - R0
    np.testing.assert_allclose(L_all, L_want, rtol=0, atol=1e-6)
    np.testing.assert_allclose(R_all, R_want, rtol=0, atol=1e-6)


@pytest.mark.parametrize("P,G", [(1, 1), (1, 4), (4, 4)])
def test_seq_descent_on_noiseless_planted_data(P, G):
    rng = np.random.default_rng(3)
    N, M, K = 30, 20, 3
    U = rng.standard_normal((N, K)) * 0.5
    V = rng.standard_normal((M, K)) * 0.5
    cells = rng.choice(N * M, size=300, replace=False)
    user, item = (cells // M).astype(np.int32), (cells % M).astype(np.int32)
    val = np.einsum("nk,nk->n", U[user], V[item]).astype(np.float32)
    o = oracle.Oracle(N, M, K, P, 0, 0.02, 0.0, oracle.SSP_LAZY, oracle.SEQ, strata=G)
    o.load(user, item, val)
    o.set_factors((0.3 * rng.standard_normal((N, K))).astype(np.float32),
                  (0.3 * rng.standard_normal((M, K))).astype(np.float32))
    losses = [o.loss()]
    for _ in range(25):
        o.clock(1)
        losses.append(o.loss())
    o.close()
    assert all(b < a for a, b in zip(losses, losses[1:]))


def test_seq_staleness_and_version_log_follow_the_table_policy():
    rng = np.random.default_rng(8)
    N, M, P, s, B = 20, 15, 3, 2, 2
    user, item, val, L0, R0 = rand_problem(rng, N, M, 120, 2)
    hist = {}
    for step in (oracle.ROWMEAN, oracle.SEQ):
        o = oracle.Oracle(N, M, 2, P, s, 0.01, 0.05, oracle.SSP_LAZY, step, B, 4)
        o.load(user, item, val)
        o.set_factors(L0, R0)
        o.clock(7)
        hist[step] = (o.export(oracle.X_STALENESS), o.export(oracle.X_VERSION_LOG))
        o.close()
    assert np.array_equal(hist[oracle.ROWMEAN][0], hist[oracle.SEQ][0])
    assert np.array_equal(hist[oracle.ROWMEAN][1], hist[oracle.SEQ][1])


@pytest.mark.parametrize("s,P", [(1, 2), (2, 3), (3, 1)])
def test_seq_under_ssp_row_with_every_row_read_each_clock_is_phase_zero_lazy(s, P):
    # B = 1: every client reads all its rows at every clock, so every row's view is
    # c - (c mod (s+1)).  Under SEQ a worker's chain depends on which users it owns, so the
    # comparison keeps the workers: worker q becomes worker (s+1) q of P(s+1) workers, all
    # in LAZY phase 0; G = 1 makes the order canonical inside each worker either way.
    rng = np.random.default_rng(5 * s + P)
    N, M, K = 24, 15, 3
    user, item, val, L0, R0 = rand_problem(rng, N, M, 200, K, dup=4)
    # eta small enough that the summed sequential progress stays finite over these clocks
    o = oracle.Oracle(N, M, K, P, s, 0.01, 0.05, oracle.SSP_ROW, oracle.SEQ, strata=1)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    o.clock(3 * s + 4)
    got = o.get_factors()
    o.close()
    owner = ((s + 1) * (np.arange(N) % P)).astype(np.int32)
    o = oracle.Oracle(N, M, K, P * (s + 1), s, 0.01, 0.05, oracle.SSP_LAZY, oracle.SEQ, owner=owner, strata=1)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    o.clock(3 * s + 4)
    want = o.get_factors()
    o.close()
    assert np.isfinite(got[0]).all() and np.isfinite(got[1]).all()
    assert np.array_equal(got[0], want[0]) and np.array_equal(got[1], want[1])


@pytest.mark.parametrize("s", [1, 3])
def test_seq_under_essp_row_with_every_row_read_each_clock_is_essp(s):
    rng = np.random.default_rng(s)
    N, M, K, P = 24, 15, 3, 4
    user, item, val, L0, R0 = rand_problem(rng, N, M, 200, K)
    res = []
    for policy in (oracle.ESSP_ROW, oracle.ESSP):
        o = oracle.Oracle(N, M, K, P, s, 0.01, 0.05, policy, oracle.SEQ, strata=3)
        o.load(user, item, val)
        o.set_factors(L0, R0)
        o.clock(7)
        res.append(o.get_factors() + (o.export(oracle.X_STALENESS),))
        o.close()
    assert np.isfinite(res[0][0]).all()
    for a, b in zip(res[0], res[1]):
        assert np.array_equal(a, b)


def test_seq_argument_errors():
    with pytest.raises(oracle.OracleError):
        oracle.Oracle(4, 4, 2, 2, 1, 0.1, 0.0, oracle.SSP_LAZY, oracle.SEQ, strata=0)
    o = oracle.Oracle(4, 4, 2, 2, 1, 0.1, 0.0, oracle.SSP_LAZY, oracle.SUM)
    o.load(np.array([0], np.int32), np.array([1], np.int32), np.array([1.0], np.float32))
    with pytest.raises(oracle.OracleError):
        o.export(oracle.X_SEQ_ORDER)
    o.close()


# ---------------------------------------------------------------- value-bounded views (VAP) and eta / sqrt(t)
def run_oracle(user, item, val, L0, R0, N, M, K, P, s, clocks, policy, step=oracle.ROWMEAN, B=1, seed=0, **kw):
    o = oracle.Oracle(N, M, K, P, s, 0.05, 0.05, policy, step, B, seed, **kw)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    o.clock(clocks)
    L, R = o.get_factors()
    out = (L, R, o.export(oracle.X_VERSION_LOG), o.export(oracle.X_STALENESS))
    o.close()
    return out


@pytest.mark.parametrize("step,B", [(oracle.ROWMEAN, 1), (oracle.SUM, 3), (oracle.SEQ, 2)])
@pytest.mark.parametrize("s", [1, 3])
def test_vap_unbounded_is_ssp_worst_and_zero_bound_is_bsp(step, B, s):
    # Section 3 (VAP): with no bound every view may miss the whole window, i.e. the oldest
    # version the ring holds (SSP_WORST); with bound 0 no update may be in transit (BSP)
    rng = np.random.default_rng(s + 7 * B)
    N, M, K, P = 30, 20, 3, 4
    user, item, val, L0, R0 = rand_problem(rng, N, M, 250, K)
    args = (user, item, val, L0, R0, N, M, K, P)
    wide = run_oracle(*args, s, 8, oracle.VAP, step, B, 3, value_bound=float("inf"))
    worst = run_oracle(*args, s, 8, oracle.SSP_WORST, step, B, 3)
    tight = run_oracle(*args, s, 8, oracle.VAP, step, B, 3, value_bound=0.0)
    bsp = run_oracle(*args, 0, 8, oracle.SSP_WORST, step, B, 3)
    for a, b in zip(wide, worst):
        assert np.array_equal(a, b)
    for a, b in zip(tight[:3], bsp[:3]):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("v0,s,P,step", [(0.1, 3, 3, oracle.ROWMEAN), (0.5, 2, 1, oracle.SUM),
                                         (0.2, 4, 5, oracle.ROWMEAN)])
def test_vap_matches_the_dense_brute_force(v0, s, P, step):
    # the dense matrix-algebra form, choosing each clock's view from its own history
    rng = np.random.default_rng(int(v0 * 1000) + s)
    N, M, K = 12, 9, 3
    user, item, val, L0, R0 = rand_problem(rng, N, M, 70, K)
    o = oracle.Oracle(N, M, K, P, s, 0.05, 0.05, oracle.VAP, step, value_bound=v0)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    o.clock(10)
    L, R = o.get_factors()
    vlog = o.export(oracle.X_VERSION_LOG).reshape(10, P)
    hist = run_dense(user, item, val, L0, R0, N=N, M=M, K=K, P=P, s=s, eta=0.05, lam=0.05, clocks=10, step=step,
                     vap_v0=v0)
    np.testing.assert_allclose(L, hist[10][0], rtol=0, atol=1e-6)
    np.testing.assert_allclose(R, hist[10][1], rtol=0, atol=1e-6)
    # the views really vary: some clocks read stale versions, some fresh
    d = np.arange(10)[:, None] - vlog
    assert (d > 0).any() and (d[1:] == 0).any()
    o.close()


def test_vap_views_satisfy_the_value_bound_and_are_the_stalest_that_do():
    rng = np.random.default_rng(12)
    N, M, K, P, s, v0 = 25, 15, 2, 3, 3, 0.03
    user, item, val, L0, R0 = rand_problem(rng, N, M, 150, K)
    o = oracle.Oracle(N, M, K, P, s, 0.05, 0.05, oracle.VAP, oracle.ROWMEAN, value_bound=v0)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    for c in range(12):
        vers = {k: o.get_version(c - k) for k in range(0, min(c, s) + 1)}
        o.clock(1)
        v = int(o.export(oracle.X_VERSION_LOG)[-1])
        norm = lambda k: max(np.abs(vers[0][0] - vers[k][0]).max(), np.abs(vers[0][1] - vers[k][1]).max())
        bound = v0 / np.sqrt(c + 1.0)
        assert norm(c - v) <= bound
        assert all(norm(k) > bound for k in vers if k > c - v)
        norms = o.export(oracle.X_VAP_NORMS).reshape(-1, s + 1)[c]
        assert all(norms[k] == norm(k) for k in vers)
    o.close()


@pytest.mark.parametrize("step,policy,s", [(oracle.ROWMEAN, oracle.SSP_LAZY, 0), (oracle.SUM, oracle.SSP_WORST, 2)])
def test_eta_decay_matches_the_dense_brute_force(step, policy, s):
    # the step schedule of Section 3's theorems, eta_t = eta / sqrt(t), t = c + 1
    rng = np.random.default_rng(4)
    N, M, K = 10, 8, 3
    user, item, val, L0, R0 = rand_problem(rng, N, M, 50, K)
    o = oracle.Oracle(N, M, K, 2, s, 0.05, 0.05, policy, step, eta_decay=True)
    o.load(user, item, val)
    o.set_factors(L0, R0)
    o.clock(6)
    L, R = o.get_factors()
    o.close()
    hist = run_dense(user, item, val, L0, R0, N=N, M=M, K=K, P=2, s=s, eta=0.05, lam=0.05, clocks=6, step=step,
                     policy=policy, eta_decay=True)
    np.testing.assert_allclose(L, hist[6][0], rtol=0, atol=1e-6)
    np.testing.assert_allclose(R, hist[6][1], rtol=0, atol=1e-6)


def test_vap_argument_errors():
    with pytest.raises(oracle.OracleError):
        oracle.Oracle(4, 4, 2, 2, 1, 0.1, 0.0, oracle.VAP, oracle.ROWMEAN, value_bound=-1.0)
    o = oracle.Oracle(4, 4, 2, 2, 1, 0.1, 0.0, oracle.SSP_LAZY, oracle.ROWMEAN)
    with pytest.raises(oracle.OracleError):
        o.export(oracle.X_VAP_NORMS)
    o.close()
