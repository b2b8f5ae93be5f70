"""HIP path vs the CPU oracle, through the C ABI, on the same seeded inputs (MI355X).

Tolerances (stated for the method): factors max |GPU - oracle| <= 1e-4 and loss relative
error <= 1e-5 after the config's clocks; integer work (layout, version log) bit-exact.
"""
import sys

import numpy as np
import pytest

import oracle
from golden_cases import load_cases
from paper_1410_8043_amd import synth

pytestmark = pytest.mark.gpu

FACTOR_TOL = 1e-4
LOSS_RTOL = 1e-5
UPDATE_RTOL = 1e-2   # of the oracle's largest accumulated update of the factor
UPDATE_FLOOR = 1e-6  # for cases whose updates are themselves near fp32 rounding


@pytest.fixture(scope="module")
def gpu():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_1410_8043_amd import ps_mf

    return ps_mf


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def run_both(ps_mf, w_user, w_item, w_val, L0, R0, *, N, M, K, P, s, eta, lam, clocks, policy=0, step=0, B=1,
             seed=0, owner=None, check_versions=False, min_dense=0, strata=None, value_bound=None, eta_decay=False,
             **handle_opts):
    say(f"case N={N} M={M} K={K} P={P} s={s} policy={policy} step={step} B={B} nnz={len(w_user)} clocks={clocks} "
        f"strata={strata} v0={value_bound} eta_decay={eta_decay} {handle_opts}")
    o = oracle.Oracle(N, M, K, P, s, eta, lam, policy, step, B, seed, owner, strata=strata, value_bound=value_bound,
                      eta_decay=eta_decay)
    o.load(w_user, w_item, w_val)
    o.set_factors(L0, R0)
    with ps_mf.PsMf(N, M, K, P, s, eta, lam, policy=policy, step=step, B=B, mb_seed=seed, owner=owner,
                    strata=strata, value_bound=value_bound, eta_decay=eta_decay, **handle_opts) as g:
        g.load_ratings(w_user, w_item, w_val)
        if step == oracle.SEQ:
            for b in range(B):
                assert np.array_equal(g.export_index(ps_mf.IDX_SEQ_ORDER, b), o.export(oracle.X_SEQ_ORDER, b))
        if min_dense:
            # the case must put at least min_dense ratings into dense (MFMA) tiles
            split = sum(g.export_index(ps_mf.IDX_SPLIT, b) for b in range(B))
            say(f"  split (dense, cells, units) x (user-major, item-major): {split.tolist()}")
            assert split[0] >= min_dense and split[3] == split[0]
        g.set_factors(L0, R0)
        g.clock(clocks)
        o.clock(clocks)
        L, R = g.get_factors()
        Lo, Ro = o.get_factors()
        err = max(np.abs(L - Lo).max(initial=0), np.abs(R - Ro).max(initial=0))
        loss, loss_o = g.loss(), o.loss()
        assert err <= FACTOR_TOL, err
        # scale-aware: each factor's deviation from the oracle is small next to the oracle's
        # own accumulated update of that factor, so a dropped term (an R commit, the lambda
        # part) cannot hide under the absolute tolerance when the updates are small
        for V, Vo, V0 in ((L, Lo, L0), (R, Ro, R0)):
            if V.size:
                upd = np.abs(Vo.astype(np.float64) - np.asarray(V0, np.float64)).max()
                dev = np.abs(V.astype(np.float64) - Vo).max()
                assert dev <= max(UPDATE_RTOL * upd, UPDATE_FLOOR), (dev, upd)
        assert abs(loss - loss_o) <= LOSS_RTOL * max(loss_o, 1e-30), (loss, loss_o)
        assert np.array_equal(g.export_index(gpu_mod().IDX_VERSION_LOG), o.export(oracle.X_VERSION_LOG))
        assert np.array_equal(g.export_index(gpu_mod().IDX_STALENESS), o.export(oracle.X_STALENESS))
        if policy in (oracle.SSP_ROW, oracle.ESSP_ROW):
            assert np.array_equal(g.export_index(gpu_mod().IDX_ROW_VERSIONS), o.export(oracle.X_ROW_VERSIONS))
        if policy == oracle.VAP:
            gn, on = g.export_index(gpu_mod().IDX_VAP_NORMS), o.export(oracle.X_VAP_NORMS)
            assert gn.shape == on.shape and np.array_equal(gn < 0, on < 0)
            assert np.abs(gn - on).max(initial=0) <= 2 * FACTOR_TOL
        if check_versions:
            for v in range(max(0, clocks - s), clocks + 1):
                Lv, Rv = g.get_version(v)
                Lov, Rov = o.get_version(v)
                assert max(np.abs(Lv - Lov).max(), np.abs(Rv - Rov).max()) <= FACTOR_TOL
    return err


def gpu_mod():
    from paper_1410_8043_amd import ps_mf
    return ps_mf


# ---------------------------------------------------------------- hand-worked values
@pytest.mark.parametrize("case", load_cases(), ids=lambda c: c["name"])
def test_hand_examples_through_abi(gpu, case):
    u = np.array([r[0] for r in case["ratings"]], np.int32)
    i = np.array([r[1] for r in case["ratings"]], np.int32)
    v = np.array([r[2] for r in case["ratings"]], np.float32)
    say(f"hand example {case['name']}")
    with gpu.PsMf(case["N"], case["M"], case["K"], case["P"], case["s"], case["eta"], case["lam"],
                  policy=case["policy"], step=case["step"], owner=case["owner"], strata=case["strata"],
                  value_bound=case["v0"]) as g:
        g.load_ratings(u, i, v)
        g.set_factors(case["L0"], case["R0"])
        for ex in sorted(case["expect"], key=lambda e: e["clock"]):
            g.clock(ex["clock"] - g.clock_value)
            L, R = g.get_factors()
            np.testing.assert_allclose(L.ravel(), ex["L"], atol=1e-6, rtol=0)
            np.testing.assert_allclose(R.ravel(), ex["R"], atol=1e-6, rtol=0)
            if ex["loss"] is not None:
                assert abs(g.loss() - ex["loss"]) <= 1e-5 * ex["loss"]


# ---------------------------------------------------------------- configured workloads
@pytest.mark.parametrize("s", [0, 2])
@pytest.mark.parametrize("policy", [oracle.SSP_LAZY, oracle.SSP_WORST, oracle.ESSP])
def test_tiny_config(gpu, s, policy):
    spec = synth.CONFIGS["tiny"]
    w = synth.generate(spec)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=s, eta=spec.eta,
             lam=spec.lam, clocks=spec.clocks, policy=policy, check_versions=True)


@pytest.mark.parametrize("step", [oracle.ROWMEAN, oracle.SUM])
def test_tiny_config_step_modes(gpu, step):
    spec = synth.CONFIGS["tiny"]
    w = synth.generate(spec)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=2, eta=spec.eta,
             lam=spec.lam, clocks=spec.clocks, step=step)


@pytest.mark.parametrize("s", [0, 1, 3, 7])
def test_full_shape_scaled(gpu, s):
    """The 100M-rating K=128 workload's degree laws at 2% of its size (several tiles, ragged tails)."""
    spec = synth.scaled(synth.CONFIGS["full"], 0.02)
    w = synth.generate(spec)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=s, eta=spec.eta,
             lam=spec.lam, clocks=10, check_versions=True)


@pytest.mark.parametrize("cells,heavy_min,hot_steps", [(False, -1, 0), (True, 1, 0), (True, 100, 0), (True, -1, 0),
                                                       (True, -1, 2), (True, 100, 1), (True, 1, 3),
                                                       (True, 10 ** 9, 2)])
@pytest.mark.parametrize("K", [32, 128, 512])
def test_lds_cells_and_units_agree_with_oracle(gpu, cells, heavy_min, hot_steps, K):
    """The LDS-staged cells (users with at least heavy_min ratings; with hot_steps > 0 also the
    other users' ratings of the most rated items) and the L2 unit path, alone and mixed, on
    the full workload's laws at 2% size, s=3 (four worker classes)."""
    spec = synth.scaled(synth.CONFIGS["full"], 0.02)
    w = synth.generate(spec, K=K)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=K, P=spec.P, s=3, eta=spec.eta,
             lam=spec.lam, clocks=6, check_versions=True, cells=cells, heavy_min=heavy_min, hot_steps=hot_steps)


@pytest.mark.parametrize("policy", [oracle.SSP_WORST, oracle.ESSP])
def test_full_shape_scaled_policies(gpu, policy):
    spec = synth.scaled(synth.CONFIGS["full"], 0.02)
    w = synth.generate(spec)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=7, eta=spec.eta,
             lam=spec.lam, clocks=10, policy=policy)


def test_medium_shape_scaled_minibatch_blocks(gpu):
    spec = synth.scaled(synth.CONFIGS["medium"], 0.05)
    w = synth.generate(spec)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=3, eta=spec.eta,
             lam=spec.lam, clocks=spec.clocks, B=spec.B, seed=spec.seed, check_versions=True)


def test_contention_shape_scaled(gpu):
    spec = synth.scaled(synth.CONFIGS["contention"], 0.03)
    w = synth.generate(spec)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=15, eta=spec.eta,
             lam=spec.lam, clocks=20)


def test_large_shape_scaled(gpu):
    spec = synth.scaled(synth.CONFIGS["large"], 0.005)
    w = synth.generate(spec)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=3, eta=spec.eta,
             lam=spec.lam, clocks=10)


@pytest.mark.parametrize("dense_min", [1, 200])
def test_large_shape_scaled_dense_tiles_at_k256(gpu, dense_min):
    """Rank 256: dense tiles with one workgroup per CU, next to cells and units."""
    spec = synth.scaled(synth.CONFIGS["large"], 0.01)
    w = synth.generate(spec)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=3, eta=spec.eta,
             lam=spec.lam, clocks=6, dense_min=dense_min, heavy_min=40, min_dense=4096)


@pytest.mark.parametrize("s", [0, 3])
def test_long_rows_take_the_workgroup_path(gpu, s):
    """Users with thousands of ratings (the capped Zipf head) exercise the long-row kernel."""
    spec = synth.ConfigSpec("heavy", 9, 40, 9000, 60_000, 1.1, 0.9, 8, 0.5, 64, 4, (s,), 0.01, 0.05, 5, 1)
    w = synth.generate(spec)
    assert np.bincount(w.user).max() >= 4096
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=s, eta=0.01,
             lam=0.05, clocks=5)


# ---------------------------------------------------------------- ragged rank and edge cases
def small_problem(seed, N, M, nnz, K, dup=0):
    rng = np.random.default_rng(seed)
    cells = rng.choice(N * M, size=nnz, replace=False)
    user = (cells // M).astype(np.int32)
    item = (cells % M).astype(np.int32)
    if dup:
        extra = rng.integers(0, nnz, size=dup)
        user = np.concatenate([user, user[extra]])
        item = np.concatenate([item, item[extra]])
    val = rng.integers(1, 6, size=user.shape[0]).astype(np.float32)
    L0 = (0.1 * rng.standard_normal((N, K))).astype(np.float32)
    R0 = (0.1 * rng.standard_normal((M, K))).astype(np.float32)
    return user, item, val, L0, R0


@pytest.mark.parametrize("K", [1, 7, 16, 33, 100, 128, 200, 256, 512])
def test_ragged_rank(gpu, K):
    N, M = 300, 90
    user, item, val, L0, R0 = small_problem(K, N, M, 3000, K, dup=20)
    run_both(gpu, user, item, val, L0, R0, N=N, M=M, K=K, P=5, s=2, eta=0.05, lam=0.05, clocks=6)


def test_zero_degree_rows_and_custom_owner(gpu):
    N, M, K = 200, 80, 16
    user, item, val, L0, R0 = small_problem(3, N, M, 1500, K)
    keep = (user % 3 != 0) & (item % 4 != 0)  # many users and items with no rating
    owner = np.random.default_rng(4).integers(0, 6, N).astype(np.int32)
    run_both(gpu, user[keep], item[keep], val[keep], L0, R0, N=N, M=M, K=K, P=6, s=3, eta=0.05, lam=0.05,
             clocks=8, owner=owner, check_versions=True)


def test_single_rating_and_empty(gpu):
    L0 = np.full((3, 4), 0.5, np.float32)
    R0 = np.full((2, 4), 0.25, np.float32)
    run_both(gpu, np.array([2], np.int32), np.array([1], np.int32), np.array([3.0], np.float32), L0, R0,
             N=3, M=2, K=4, P=2, s=1, eta=0.1, lam=0.1, clocks=4)
    run_both(gpu, np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32), L0, R0,
             N=3, M=2, K=4, P=2, s=1, eta=0.1, lam=0.1, clocks=3)


def test_device_handle_exports_match_oracle_layout(gpu):
    spec = synth.scaled(synth.CONFIGS["medium"], 0.02)
    w = synth.generate(spec, K=8)
    with gpu.PsMf(spec.N, spec.M, 8, spec.P, 3, 0.01, 0.05, B=spec.B, mb_seed=spec.seed) as g:
        g.load_ratings(w.user, w.item, w.val)
        o = oracle.Oracle(spec.N, spec.M, 8, spec.P, 3, 0.01, 0.05, oracle.SSP_LAZY, oracle.ROWMEAN, spec.B,
                          spec.seed)
        o.load(w.user, w.item, w.val)
        for b in range(spec.B):
            assert np.array_equal(g.export_index(gpu.IDX_PERM, b), o.export(oracle.X_PERM, b))
            assert np.array_equal(g.export_index(gpu.IDX_ROW_PTR, b), o.export(oracle.X_ROW_PTR, b))


def test_checkpoint_resume_at_s0(gpu):
    spec = synth.CONFIGS["tiny"]
    w = synth.generate(spec)
    args = (spec.N, spec.M, spec.K, spec.P, 0, spec.eta, spec.lam)
    with gpu.PsMf(*args) as a:
        a.load_ratings(w.user, w.item, w.val)
        a.set_factors(w.L0, w.R0)
        a.clock(10)
        L10, R10 = a.get_factors()
    with gpu.PsMf(*args) as b:
        b.load_ratings(w.user, w.item, w.val)
        b.set_factors(w.L0, w.R0)
        b.clock(5)
        L5, R5 = b.get_factors()
        b.set_factors(L5, R5)
        b.clock(5)
        Lr, Rr = b.get_factors()
    assert max(np.abs(L10 - Lr).max(), np.abs(R10 - Rr).max()) <= FACTOR_TOL


# ---------------------------------------------------------------- dense (MFMA) tiles
@pytest.mark.parametrize("s,policy", [(0, oracle.SSP_LAZY), (2, oracle.SSP_LAZY), (2, oracle.SSP_WORST),
                                      (2, oracle.ESSP)])
@pytest.mark.parametrize("dense_min", [1, 150])
def test_tiny_config_dense_tiles(gpu, s, policy, dense_min):
    """The tiny workload with every 64 x 64 tile (dense_min = 1) or about half of them swept
    by the matrix-core cells, the rest by cells and units."""
    spec = synth.CONFIGS["tiny"]
    w = synth.generate(spec)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=s, eta=spec.eta,
             lam=spec.lam, clocks=spec.clocks, policy=policy, check_versions=True, dense_min=dense_min,
             min_dense=spec.nnz // 4)


@pytest.mark.parametrize("K", [16, 32, 64, 100, 128])
@pytest.mark.parametrize("dense_min", [1, 300, 1229])
def test_dense_tiles_mixed_with_cells_and_units(gpu, K, dense_min):
    """The 100M-rating workload's laws at 5% size, s=3 (four worker classes): dense tiles of
    heavy users x popular items next to LDS cells and L2 units, ragged tile edges."""
    spec = synth.scaled(synth.CONFIGS["full"], 0.05)
    w = synth.generate(spec, K=K)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=K, P=spec.P, s=3, eta=spec.eta,
             lam=spec.lam, clocks=6, check_versions=True, dense_min=dense_min, heavy_min=100, hot_steps=1,
             min_dense=4096)


@pytest.mark.parametrize("K", [16, 33, 100, 128, 200, 256])
def test_dense_tiles_ragged_rank_duplicates_and_empty_rows(gpu, K):
    """Every tile dense: padded ranks, duplicate (user, item) pairs (the repeats stay
    sparse), users and items without ratings and a scattering owner map."""
    N, M = 300, 90
    user, item, val, L0, R0 = small_problem(K + 1, N, M, 6000, K, dup=40)
    keep = (user % 7 != 0) & (item % 5 != 0)
    owner = np.random.default_rng(K).integers(0, 5, N).astype(np.int32)
    run_both(gpu, user[keep], item[keep], val[keep], L0, R0, N=N, M=M, K=K, P=5, s=2, eta=0.05, lam=0.05,
             clocks=6, owner=owner, check_versions=True, dense_min=1, min_dense=1000)


@pytest.mark.parametrize("step", [oracle.ROWMEAN, oracle.SUM])
def test_dense_tiles_medium_minibatch_blocks(gpu, step):
    spec = synth.scaled(synth.CONFIGS["medium"], 0.05)
    w = synth.generate(spec)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=3,
             eta=spec.eta if step == oracle.ROWMEAN else 1e-4, lam=spec.lam, clocks=8, B=spec.B, seed=spec.seed,
             step=step, dense_min=64, min_dense=4096)


# ---------------------------------------------------------------- per-row caches (Section 4)
@pytest.mark.parametrize("config,policy,s,B", [("full", oracle.SSP_LAZY, 3, 1), ("full", oracle.SSP_LAZY, 0, 1),
                                                ("full", oracle.ESSP, 2, 1), ("full", oracle.SSP_ROW, 1, 1),
                                                ("full", oracle.VAP, 3, 1), ("medium", oracle.SSP_LAZY, 3, 4),
                                                ("medium", oracle.SSP_WORST, 2, 4), ("medium", oracle.ESSP_ROW, 2, 4)])
def test_unit_written_rows_equal_commit_written_rows(gpu, config, policy, s, B):
    """PS_MF_OPT_UNIT_COMMIT: the work unit of a user whose ratings all lie in it writes the
    user's new version itself (when the user's view is not the new version's slot) and the
    commit skips the user.  Every clock's factors, loss and version log must equal the commit
    writing every row, bit for bit, and stay within the oracle's tolerances; the poisoned
    commit (rows the commit does not write are NaN before it) must stay finite."""
    spec = synth.scaled(synth.CONFIGS[config], 0.05)
    K = 64 if config == "full" else spec.K
    w = synth.generate(spec, K=K)
    opts = dict(dense_min=300, heavy_min=64, hot_steps=0) if config == "full" else {}
    vb = 0.003 if policy == oracle.VAP else None
    clocks = 2 * s + 3
    say(f"unit commit: {config}@0.05 nnz={w.nnz} policy={policy} s={s} B={B} clocks={clocks}")
    out = []
    for unit_commit, poison in ((True, True), (False, False)):
        with gpu.PsMf(spec.N, spec.M, K, spec.P, s, spec.eta, spec.lam, policy=policy, B=B, mb_seed=spec.seed,
                      value_bound=vb, unit_commit=unit_commit, poison=poison, **opts) as g:
            g.load_ratings(w.user, w.item, w.val)
            g.set_factors(w.L0, w.R0)
            hist = []
            for _ in range(clocks):
                g.clock(1)
                hist.append(g.loss())
                hist.append(g.get_factors())
            out.append((hist, g.export_index(gpu.IDX_VERSION_LOG)))
    (ha, va), (hb, vb_) = out
    assert np.array_equal(va, vb_)
    for x, y in zip(ha, hb):
        if isinstance(x, tuple):
            assert np.isfinite(x[0]).all() and np.isfinite(x[1]).all()
            assert np.array_equal(x[0], y[0]) and np.array_equal(x[1], y[1])
        else:
            assert x == y
    o = oracle.Oracle(spec.N, spec.M, K, spec.P, s, spec.eta, spec.lam, policy, oracle.ROWMEAN, B, spec.seed,
                      value_bound=vb)
    o.load(w.user, w.item, w.val)
    o.set_factors(w.L0, w.R0)
    o.clock(clocks)
    Lo, Ro = o.get_factors()
    loss_o = o.loss()
    o.close()
    L, R = ha[-1]
    assert max(np.abs(L - Lo).max(), np.abs(R - Ro).max()) <= FACTOR_TOL
    assert abs(ha[-2] - loss_o) <= LOSS_RTOL * loss_o


@pytest.mark.parametrize("policy", [oracle.SSP_ROW, oracle.ESSP_ROW])
@pytest.mark.parametrize("s,B", [(0, 1), (1, 1), (1, 4), (3, 4), (7, 3)])
def test_tiny_config_per_row_policies(gpu, policy, s, B):
    """Per-row cached versions on the tiny workload, whole shards (B = 1) and minibatches
    (rows read intermittently, so their cached versions differ row by row)."""
    spec = synth.CONFIGS["tiny"]
    w = synth.generate(spec)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=s, eta=spec.eta,
             lam=spec.lam, clocks=12, policy=policy, B=B, seed=spec.seed, check_versions=True)


@pytest.mark.parametrize("policy", [oracle.SSP_ROW, oracle.ESSP_ROW])
@pytest.mark.parametrize("K", [32, 128])
def test_per_row_policies_with_dense_tiles_cells_and_units(gpu, policy, K):
    """The 100M-rating workload's laws at 5% size in 4 minibatch blocks, s = 3: per-row
    slots through the dense tiles, the LDS cells, the L2 units and the commit."""
    spec = synth.scaled(synth.CONFIGS["full"], 0.05)
    w = synth.generate(spec, K=K)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=K, P=spec.P, s=3, eta=spec.eta,
             lam=spec.lam, clocks=9, policy=policy, B=4, seed=spec.seed, check_versions=True, dense_min=300,
             heavy_min=30, hot_steps=1, min_dense=4096)


@pytest.mark.parametrize("policy", [oracle.SSP_ROW, oracle.ESSP_ROW])
def test_per_row_policies_medium_minibatches_ragged_rank(gpu, policy):
    spec = synth.scaled(synth.CONFIGS["medium"], 0.05)
    w = synth.generate(spec, K=33)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=33, P=spec.P, s=3, eta=spec.eta,
             lam=spec.lam, clocks=10, policy=policy, B=spec.B, seed=spec.seed)


def test_timing_option_counts_launches(gpu):
    spec = synth.CONFIGS["tiny"]
    w = synth.generate(spec)
    with gpu.PsMf(spec.N, spec.M, spec.K, spec.P, 2, spec.eta, spec.lam, timing=True) as g:
        g.load_ratings(w.user, w.item, w.val)
        g.set_factors(w.L0, w.R0)
        g.clock(7)
        ms, n = g.kernel_time(gpu.KERNEL_SWEEP)
        assert n == 7 and ms > 0
        ms, n = g.kernel_time(gpu.KERNEL_COMMIT)
        assert n == 7 and ms > 0


# ---------------------------------------------------------------- sequential steps inside a worker (STEP_SEQ)
@pytest.mark.parametrize("s", [0, 2])
@pytest.mark.parametrize("policy", [oracle.SSP_LAZY, oracle.SSP_WORST, oracle.ESSP])
@pytest.mark.parametrize("G", [1, 8, 64])
def test_tiny_config_seq(gpu, s, policy, G):
    """Each worker applies its ratings one by one to its own rows (G sub-epochs of
    row-disjoint strata), on the 20,000-rating K=16 workload, 10 clocks."""
    spec = synth.CONFIGS["tiny"]
    w = synth.generate(spec)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=s, eta=spec.eta,
             lam=spec.lam, clocks=spec.clocks, policy=policy, step=oracle.SEQ, strata=G, check_versions=True)


@pytest.mark.parametrize("s,G", [(0, 64), (3, 64), (7, 16)])
def test_full_shape_scaled_seq(gpu, s, G):
    spec = synth.scaled(synth.CONFIGS["full"], 0.02)
    w = synth.generate(spec)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=s, eta=spec.eta,
             lam=spec.lam, clocks=10, step=oracle.SEQ, strata=G, check_versions=True)


def test_medium_shape_scaled_seq_minibatch_blocks(gpu):
    spec = synth.scaled(synth.CONFIGS["medium"], 0.05)
    w = synth.generate(spec)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=3, eta=spec.eta,
             lam=spec.lam, clocks=spec.clocks, B=spec.B, seed=spec.seed, step=oracle.SEQ, strata=32)


def test_contention_and_large_shapes_scaled_seq(gpu):
    spec = synth.scaled(synth.CONFIGS["contention"], 0.03)
    w = synth.generate(spec)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=15, eta=spec.eta,
             lam=spec.lam, clocks=8, step=oracle.SEQ, strata=64)
    spec = synth.scaled(synth.CONFIGS["large"], 0.005)
    w = synth.generate(spec)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=3, eta=spec.eta,
             lam=spec.lam, clocks=4, step=oracle.SEQ, strata=64)


@pytest.mark.parametrize("K", [1, 7, 33, 100, 200, 512])
def test_ragged_rank_seq(gpu, K):
    N, M = 300, 90
    user, item, val, L0, R0 = small_problem(K, N, M, 3000, K, dup=20)
    run_both(gpu, user, item, val, L0, R0, N=N, M=M, K=K, P=5, s=2, eta=0.05, lam=0.05, clocks=6, step=oracle.SEQ,
             strata=6)


def test_seq_zero_degree_rows_custom_owner_single_and_empty(gpu):
    N, M, K = 200, 80, 16
    user, item, val, L0, R0 = small_problem(3, N, M, 1500, K)
    keep = (user % 3 != 0) & (item % 4 != 0)
    owner = np.random.default_rng(4).integers(0, 6, N).astype(np.int32)
    run_both(gpu, user[keep], item[keep], val[keep], L0, R0, N=N, M=M, K=K, P=6, s=3, eta=0.05, lam=0.05,
             clocks=8, owner=owner, step=oracle.SEQ, strata=5, B=3, seed=2, check_versions=True)
    L0 = np.full((3, 4), 0.5, np.float32)
    R0 = np.full((2, 4), 0.25, np.float32)
    run_both(gpu, np.array([2], np.int32), np.array([1], np.int32), np.array([3.0], np.float32), L0, R0,
             N=3, M=2, K=4, P=2, s=1, eta=0.1, lam=0.1, clocks=4, step=oracle.SEQ, strata=3)
    run_both(gpu, np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32), L0, R0,
             N=3, M=2, K=4, P=2, s=1, eta=0.1, lam=0.1, clocks=3, step=oracle.SEQ)


# ---------------------------------------------------------------- value-bounded views (VAP) and eta / sqrt(t)
VAP_MARGIN = 1e-5  # decisions are compared only where the oracle's norm is this far from the bound (the
                  # factors of the two sides agree to about 1e-6 over these runs)


def pick_value_bound(user, item, val, L0, R0, candidates, *, N, M, K, P, s, eta, lam, clocks, step=0, B=1, seed=0,
                     strata=None, eta_decay=False):
    """The first candidate bound under which the oracle's every view decision (norm vs bound)
    keeps VAP_MARGIN, so that fp32 differences cannot flip it, and which mixes stale and
    fresh views."""
    for v0 in candidates:
        o = oracle.Oracle(N, M, K, P, s, eta, lam, oracle.VAP, step, B, seed, strata=strata, value_bound=v0,
                          eta_decay=eta_decay)
        o.load(user, item, val)
        o.set_factors(L0, R0)
        o.clock(clocks)
        norms = o.export(oracle.X_VAP_NORMS).reshape(clocks, s + 1)
        d = np.arange(clocks) - o.export(oracle.X_VERSION_LOG).reshape(clocks, P)[:, 0]
        o.close()
        bound = v0 / np.sqrt(np.arange(clocks) + 1.0)
        gap = np.abs(norms[:, 1:] - bound[:, None])[norms[:, 1:] >= 0]
        if (gap.size == 0 or gap.min() > VAP_MARGIN) and (d[1:] > 0).any() and (d[1:] == 0).any():
            say(f"  value bound {v0}: delays {d.tolist()}, smallest margin {gap.min(initial=np.inf):.3g}")
            return v0
    raise AssertionError("no candidate bound keeps the decision margin")


@pytest.mark.parametrize("s,step", [(1, oracle.ROWMEAN), (2, oracle.SUM), (3, oracle.SEQ)])
def test_tiny_config_vap(gpu, s, step):
    spec = synth.CONFIGS["tiny"]
    w = synth.generate(spec)
    kw = dict(N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=s, eta=spec.eta, lam=spec.lam, clocks=spec.clocks, step=step,
              strata=8 if step == oracle.SEQ else None)
    v0 = pick_value_bound(w.user, w.item, w.val, w.L0, w.R0, [1e-4 * 1.25 ** k for k in range(80)], **kw)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, policy=oracle.VAP, value_bound=v0, check_versions=True, **kw)


def test_vap_limits_and_eta_decay(gpu):
    spec = synth.CONFIGS["tiny"]
    w = synth.generate(spec)
    kw = dict(N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=2, eta=spec.eta, lam=spec.lam, clocks=spec.clocks)
    for v0 in (0.0, float("inf")):
        run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, policy=oracle.VAP, value_bound=v0, **kw)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, policy=oracle.SSP_LAZY, eta_decay=True, **kw)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, policy=oracle.SSP_WORST, step=oracle.SEQ, strata=16,
             eta_decay=True, **kw)


def test_full_shape_scaled_vap(gpu):
    spec = synth.scaled(synth.CONFIGS["full"], 0.02)
    w = synth.generate(spec)
    kw = dict(N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=3, eta=spec.eta, lam=spec.lam, clocks=8)
    v0 = pick_value_bound(w.user, w.item, w.val, w.L0, w.R0, [1e-4 * 1.25 ** k for k in range(80)], **kw)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, policy=oracle.VAP, value_bound=v0, check_versions=True, **kw)


def test_medium_shape_scaled_vap_minibatch_blocks_and_eta_decay(gpu):
    spec = synth.scaled(synth.CONFIGS["medium"], 0.05)
    w = synth.generate(spec)
    kw = dict(N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=3, eta=spec.eta, lam=spec.lam, clocks=12, B=spec.B,
              seed=spec.seed, eta_decay=True)
    v0 = pick_value_bound(w.user, w.item, w.val, w.L0, w.R0, [1e-4 * 1.25 ** k for k in range(80)], **kw)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, policy=oracle.VAP, value_bound=v0, **kw)


@pytest.mark.parametrize("policy,s,B", [(oracle.SSP_LAZY, 2, 3), (oracle.VAP, 2, 2), (oracle.ESSP, 1, 1)])
def test_seq_graph_replays_equal_eager_launches(gpu, policy, s, B):
    """The sequential step replays a captured HIP graph per (block, view schedule); every
    replay, with the program's own work and synchronizations between clocks, must equal
    launching the sub-epochs one by one, bit for bit."""
    N, M, K = 400, 150, 33
    user, item, val, L0, R0 = small_problem(11, N, M, 6000, K, dup=30)
    out = []
    for graphs in (True, False):
        with gpu.PsMf(N, M, K, 5, s, 0.02, 0.05, policy=policy, step=gpu.STEP_SEQ, strata=7, B=B, mb_seed=3,
                      value_bound=0.05 if policy == oracle.VAP else None, seq_graphs=graphs) as g:
            g.load_ratings(user, item, val)
            g.set_factors(L0, R0)
            hist = []
            for _ in range(3 * (2 * s + 1) * B):
                g.clock(1)
                hist.append(g.loss())
                hist.append(g.get_factors())
            out.append((hist, g.export_index(gpu.IDX_VERSION_LOG)))
    (ha, va), (hb, vb) = out
    assert np.array_equal(va, vb)
    for x, y in zip(ha, hb):
        if isinstance(x, tuple):
            assert np.array_equal(x[0], y[0]) and np.array_equal(x[1], y[1])
        else:
            assert x == y


@pytest.mark.parametrize("policy,s,B", [(oracle.SSP_LAZY, 2, 3), (oracle.VAP, 2, 2), (oracle.SSP_ROW, 1, 2),
                                      (oracle.SSP_WORST, 0, 1)])
def test_sweep_graph_replays_equal_eager_launches(gpu, policy, s, B):
    """With PS_MF_OPT_SWEEP_GRAPHS each clock's sweep (units, LDS cells and dense tiles on
    their three streams) is replayed from a HIP graph per (block, view schedule); every
    replay, with the program's own work and synchronizations between clocks, must equal
    launching the sweep one kernel at a time, bit for bit, and stay within the tolerances
    of the oracle."""
    spec = synth.scaled(synth.CONFIGS["full"], 0.05)
    w = synth.generate(spec, K=64)
    opts = dict(dense_min=300, heavy_min=64, hot_steps=0)
    clocks = (2 * s + 1) * B + 2  # every (block, view schedule) graph, some replayed
    say(f"sweep graphs: full@0.05 nnz={w.nnz} policy={policy} s={s} B={B} clocks={clocks}")
    out = []
    for graphs in (True, False):
        with gpu.PsMf(spec.N, spec.M, 64, spec.P, s, spec.eta, spec.lam, policy=policy, B=B, mb_seed=spec.seed,
                      value_bound=0.003 if policy == oracle.VAP else None, sweep_graphs=graphs, **opts) as g:
            g.load_ratings(w.user, w.item, w.val)
            split = g.export_index(gpu.IDX_SPLIT)
            assert split[0] > 0 and split[1] > 0 and split[2] > 0, split
            g.set_factors(w.L0, w.R0)
            hist = []
            for _ in range(clocks):
                g.clock(1)
                hist.append(g.loss())
                hist.append(g.get_factors())
            out.append((hist, g.export_index(gpu.IDX_VERSION_LOG)))
    (ha, va), (hb, vb) = out
    assert np.array_equal(va, vb)
    for x, y in zip(ha, hb):
        if isinstance(x, tuple):
            assert np.array_equal(x[0], y[0]) and np.array_equal(x[1], y[1])
        else:
            assert x == y
    o = oracle.Oracle(spec.N, spec.M, 64, spec.P, s, spec.eta, spec.lam, policy, oracle.ROWMEAN, B, spec.seed,
                      value_bound=0.003 if policy == oracle.VAP else None)
    o.load(w.user, w.item, w.val)
    o.set_factors(w.L0, w.R0)
    o.clock(clocks)
    Lo, Ro = o.get_factors()
    loss_o = o.loss()
    o.close()
    L, R = ha[-1]
    assert max(np.abs(L - Lo).max(), np.abs(R - Ro).max()) <= FACTOR_TOL
    assert abs(ha[-2] - loss_o) <= LOSS_RTOL * loss_o


@pytest.mark.parametrize("policy", [oracle.SSP_ROW, oracle.ESSP_ROW])
@pytest.mark.parametrize("s,B", [(1, 1), (3, 4), (2, 3)])
def test_tiny_config_seq_per_row_policies(gpu, policy, s, B):
    """The sequential step under the per-row caches: each worker's copy starts from the
    versions its client's cache holds; cached versions, staleness and factors against the
    oracle."""
    spec = synth.CONFIGS["tiny"]
    w = synth.generate(spec)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=spec.K, P=spec.P, s=s, eta=spec.eta,
             lam=spec.lam, clocks=spec.clocks, policy=policy, step=oracle.SEQ, strata=8, B=B, seed=5)


def test_medium_shape_scaled_seq_per_row_ragged_rank(gpu):
    spec = synth.scaled(synth.CONFIGS["medium"], 0.05)
    w = synth.generate(spec, K=33)
    run_both(gpu, w.user, w.item, w.val, w.L0, w.R0, N=spec.N, M=spec.M, K=33, P=spec.P, s=3, eta=spec.eta,
             lam=spec.lam, clocks=8, policy=oracle.SSP_ROW, step=oracle.SEQ, strata=32, B=spec.B, seed=spec.seed)


def test_seq_clock_inside_a_callers_graph_capture(gpu):
    """A caller may capture a sequential clock into its own HIP graph (torch.cuda.graph on
    the handle's stream): the library then launches the sub-epochs one by one into the
    caller's capture.  With s = 0 and one block every clock runs the same launches, so every
    replay advances the factors exactly like an eager clock."""
    import torch

    N, M, K = 300, 120, 16
    user, item, val, L0, R0 = small_problem(21, N, M, 4000, K)
    side = torch.cuda.Stream()
    res = []
    for captured in (False, True):
        with gpu.PsMf(N, M, K, 4, 0, 0.02, 0.05, step=gpu.STEP_SEQ, strata=5, stream=side) as g:
            g.load_ratings(user, item, val)
            g.set_factors(L0, R0)
            torch.cuda.synchronize()
            if captured:
                graph = torch.cuda.CUDAGraph()
                with torch.cuda.graph(graph, stream=side):
                    g.clock(1)
                for _ in range(4):  # the capture itself ran nothing; each replay is one clock
                    graph.replay()
                    torch.cuda.synchronize()
                    res.append(g.get_factors())  # s = 0: the one ring slot
            else:
                for _ in range(4):
                    g.clock(1)
                    torch.cuda.synchronize()
                    res.append(g.get_factors())
    for (La, Ra), (Lb, Rb) in zip(res[:4], res[4:]):
        assert np.array_equal(La, Lb) and np.array_equal(Ra, Rb)
