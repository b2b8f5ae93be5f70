"""The C-ABI library: symbols, argument checks and the host-side integer layout (no GPU).

Host-only handles (PS_MF_OPT_HOST_ONLY) build and export the integer layout without
touching a device; their exports must equal the oracle's, bit for bit.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ps_mf = pytest.importorskip("paper_1410_8043_amd.ps_mf", reason="libps_mf.so not built")


def declared_functions():
    text = open(os.path.join(ROOT, "include", "ps_mf.h")).read()
    return sorted(set(re.findall(r"\b(ps_mf_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(ps_mf.LIB_PATH)
    names = declared_functions()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(ps_mf.SYMBOLS)


def test_every_header_constant_matches_the_binding():
    """Every #define PS_MF_<NAME> <value> of include/ps_mf.h (error codes, option keys,
    policies, steps, exports, timing kinds) has the same value in the Python binding."""
    text = open(os.path.join(ROOT, "include", "ps_mf.h")).read()
    consts = dict(re.findall(r"#define PS_MF_([A-Z_0-9]+) \(?(-?\d+)\)?", text))
    assert len(consts) == 50, len(consts)
    for name, value in consts.items():
        assert getattr(ps_mf, name) == int(value), name


@pytest.mark.parametrize("args", [
    (0, 1, 1, 1, 0, 0.1, 0.1), (1, 0, 1, 1, 0, 0.1, 0.1), (1, 1, 0, 1, 0, 0.1, 0.1), (1, 1, 513, 1, 0, 0.1, 0.1),
    (1, 1, 1, 0, 0, 0.1, 0.1), (1, 1, 1, 1, -1, 0.1, 0.1), (1, 1, 1, 1, 0, float("nan"), 0.1),
    (1, 1, 1, 1, 0, 0.1, float("inf")), (2**31, 1, 1, 1, 0, 0.1, 0.1)])
def test_create_rejects_bad_arguments(args):
    with pytest.raises(ps_mf.PsMfError) as e:
        ps_mf.ps_mf_create(*args)
    assert e.value.code == ps_mf.EINVAL


def test_option_and_state_errors():
    h = ps_mf.ps_mf_create(4, 3, 2, 2, 1, 0.1, 0.1)
    try:
        for key, val in [(99, 0), (ps_mf.OPT_POLICY, 7), (ps_mf.OPT_STEP, 5), (ps_mf.OPT_MB_BLOCKS, 0)]:
            with pytest.raises(ps_mf.PsMfError) as e:
                ps_mf.ps_mf_set_option(h, key, val)
            assert e.value.code == ps_mf.EINVAL
        with pytest.raises(ps_mf.PsMfError) as e:
            ps_mf.ps_mf_set_owner_map(h, np.array([0, 1, 2, 0]))
        assert e.value.code == ps_mf.EINVAL
        for f in (lambda: ps_mf.ps_mf_clock(h, 1), lambda: ps_mf.ps_mf_loss(h),
                  lambda: ps_mf.ps_mf_set_factors(h, np.zeros((4, 2)), np.zeros((3, 2)))):
            with pytest.raises(ps_mf.PsMfError) as e:
                f()
            assert e.value.code == ps_mf.ESTATE
        ps_mf.ps_mf_set_option(h, ps_mf.OPT_HOST_ONLY, 1)
        ps_mf.ps_mf_load_ratings(h, np.array([0, 3]), np.array([2, 0]), np.array([1.0, 5.0]))
        with pytest.raises(ps_mf.PsMfError) as e:
            ps_mf.ps_mf_load_ratings(h, np.array([0]), np.array([0]), np.array([1.0]))
        assert e.value.code == ps_mf.ESTATE
        with pytest.raises(ps_mf.PsMfError) as e:
            ps_mf.ps_mf_set_option(h, ps_mf.OPT_POLICY, ps_mf.ESSP)
        assert e.value.code == ps_mf.ESTATE
        with pytest.raises(ps_mf.PsMfError) as e:
            ps_mf.ps_mf_export_index(h, ps_mf.IDX_COL, 1)
        assert e.value.code == ps_mf.EINVAL
        assert "block" in ps_mf.ps_mf_last_error(h)
    finally:
        ps_mf.ps_mf_destroy(h)
    ps_mf.ps_mf_destroy(None)  # NULL-safe


@pytest.mark.parametrize("bad", [dict(user=[0, 4]), dict(user=[-1, 0]), dict(item=[0, 3]),
                                 dict(value=[1.0, float("nan")]), dict(value=[float("inf"), 1.0])])
def test_load_rejects_bad_ratings(bad):
    coo = dict(user=[0, 1], item=[0, 2], value=[1.0, 2.0])
    coo.update(bad)
    with ps_mf.PsMf(4, 3, 2, 1, 0, 0.1, 0.1, host_only=True) as g:
        with pytest.raises(ps_mf.PsMfError) as e:
            g.load_ratings(np.array(coo["user"]), np.array(coo["item"]), np.array(coo["value"]))
        assert e.value.code == ps_mf.EINVAL


def compare_layout(g, o, B, N, M):
    assert np.array_equal(g.export_index(ps_mf.IDX_OWNER), o.export(oracle.X_OWNER))
    for b in range(B):
        for kind_g, kind_o in [(ps_mf.IDX_ROW_PTR, oracle.X_ROW_PTR), (ps_mf.IDX_COL, oracle.X_COL),
                               (ps_mf.IDX_PERM, oracle.X_PERM), (ps_mf.IDX_USER_COUNT, oracle.X_USER_COUNT),
                               (ps_mf.IDX_ITEM_COUNT, oracle.X_ITEM_COUNT)]:
            a, e = g.export_index(kind_g, b), o.export(kind_o, b)
            assert a.dtype == e.dtype and np.array_equal(a, e), (b, kind_g)


@pytest.mark.parametrize("B", [1, 3, 8])
@pytest.mark.parametrize("custom_owner", [False, True])
def test_host_layout_is_bit_exact_with_oracle(B, custom_owner):
    rng = np.random.default_rng(B)
    N, M, P, n = 300, 120, 7, 5000
    user = rng.integers(0, N, n).astype(np.int32)
    item = rng.integers(0, M, n).astype(np.int32)  # duplicates included on purpose
    val = rng.integers(1, 6, n).astype(np.float32)
    owner = rng.integers(0, P, N).astype(np.int32) if custom_owner else None
    seed = 0x14108043 + B
    with ps_mf.PsMf(N, M, 4, P, 2, 0.01, 0.05, B=B, mb_seed=seed, owner=owner, host_only=True) as g:
        g.load_ratings(user, item, val)
        o = oracle.Oracle(N, M, 4, P, 2, 0.01, 0.05, oracle.SSP_LAZY, oracle.ROWMEAN, B, seed, owner)
        o.load(user, item, val)
        compare_layout(g, o, B, N, M)


def test_host_layout_on_generated_workload():
    from paper_1410_8043_amd import synth
    spec = synth.scaled(synth.CONFIGS["medium"], 0.05)
    w = synth.generate(spec, K=8)
    with ps_mf.PsMf(spec.N, spec.M, 8, spec.P, 3, 0.01, 0.05, B=spec.B, mb_seed=spec.seed, host_only=True) as g:
        g.load_ratings(w.user, w.item, w.val)
        o = oracle.Oracle(spec.N, spec.M, 8, spec.P, 3, 0.01, 0.05, oracle.SSP_LAZY, oracle.ROWMEAN, spec.B, spec.seed)
        o.load(w.user, w.item, w.val)
        compare_layout(g, o, spec.B, spec.N, spec.M)


def test_empty_and_single_rating_layouts():
    with ps_mf.PsMf(5, 4, 3, 2, 0, 0.1, 0.1, host_only=True) as g:
        g.load_ratings(np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32))
        assert g.export_index(ps_mf.IDX_COL).size == 0
        assert np.array_equal(g.export_index(ps_mf.IDX_ROW_PTR), np.zeros(6, np.int64))
    with ps_mf.PsMf(5, 4, 3, 2, 0, 0.1, 0.1, host_only=True) as g:
        g.load_ratings(np.array([4]), np.array([3]), np.array([2.0]))
        assert np.array_equal(g.export_index(ps_mf.IDX_ROW_PTR), [0, 0, 0, 0, 0, 1])
        assert np.array_equal(g.export_index(ps_mf.IDX_ITEM_COUNT), [0, 0, 0, 1])


@pytest.mark.parametrize("cells,heavy_min,hot_steps", [(False, -1, 0), (True, 1, 0), (True, 40, 0), (True, -1, 0),
                                                       (True, -1, 1), (True, 40, 3), (True, 1, 2), (True, -1, -1)])
@pytest.mark.parametrize("K", [8, 128, 512])
def test_host_layout_with_and_without_cells(cells, heavy_min, hot_steps, K):
    """The exported integer layout does not depend on how the sweeps are scheduled, and the
    library's self-check (run on every host-only load) accepts each schedule."""
    from paper_1410_8043_amd import synth
    spec = synth.scaled(synth.CONFIGS["full"], 0.01)
    w = synth.generate(spec, K=1)
    with ps_mf.PsMf(spec.N, spec.M, K, spec.P, 3, 0.01, 0.05, host_only=True, cells=cells,
                    heavy_min=heavy_min, hot_steps=hot_steps) as g:
        g.load_ratings(w.user, w.item, w.val)
        o = oracle.Oracle(spec.N, spec.M, 4, spec.P, 3, 0.01, 0.05)
        o.load(w.user, w.item, w.val)
        compare_layout(g, o, 1, spec.N, spec.M)


@pytest.mark.parametrize("policy,s", [(0, 0), (0, 2), (1, 3), (2, 4)])
@pytest.mark.parametrize("B", [1, 3])
def test_host_layout_self_check_with_hot_cells_and_custom_owner(policy, s, B):
    """Cells of both families with several worker classes, minibatch blocks and an owner map
    that scatters users over workers: the self-check holds and the exported layout is the
    oracle's."""
    rng = np.random.default_rng(100 * s + B)
    N, M, P, n = 700, 300, 6, 60000
    # a few dense users and items so that every cell family is populated
    user = np.concatenate([rng.integers(0, N, n // 2), rng.integers(0, 24, n // 2)]).astype(np.int32)
    item = np.concatenate([rng.integers(0, 40, n // 2), rng.integers(0, M, n // 2)]).astype(np.int32)
    val = rng.integers(1, 6, user.size).astype(np.float32)
    owner = rng.integers(0, P, N).astype(np.int32)
    seed = 0x14108043 + 17 * B
    with ps_mf.PsMf(N, M, 16, P, s, 0.01, 0.05, policy=policy, B=B, mb_seed=seed, owner=owner, host_only=True,
                    cells=True, heavy_min=64, hot_steps=2) as g:
        g.load_ratings(user, item, val)
        o = oracle.Oracle(N, M, 16, P, s, 0.01, 0.05, policy, oracle.ROWMEAN, B, seed, owner)
        o.load(user, item, val)
        compare_layout(g, o, B, N, M)


def split_of(g, b=0):
    s = g.export_index(ps_mf.IDX_SPLIT, b)
    assert s.shape == (8,)
    return s


@pytest.mark.parametrize("dense_min", [1, 9, 200])
@pytest.mark.parametrize("policy,s,B", [(0, 0, 1), (0, 3, 1), (1, 2, 3), (2, 5, 2)])
@pytest.mark.parametrize("K", [16, 100])
def test_host_layout_self_check_with_dense_tiles(dense_min, policy, s, B, K):
    """Dense (matrix-core) tiles next to cells and units: every rating is swept exactly once
    per direction (self-check on load), duplicates of a (user, item) pair included, and the
    exported canonical layout is still the oracle's."""
    rng = np.random.default_rng(1000 * dense_min + 10 * s + B)
    N, M, P, n = 900, 400, 6, 80000
    # a block of heavy users x popular items (dense), plus scattered ratings and duplicates
    user = np.concatenate([rng.integers(0, 150, n // 2), rng.integers(0, N, n // 2)]).astype(np.int32)
    item = np.concatenate([rng.integers(0, 130, n // 2), rng.integers(0, M, n // 2)]).astype(np.int32)
    val = rng.integers(1, 6, user.size).astype(np.float32)
    owner = rng.integers(0, P, N).astype(np.int32)
    seed = 0x14108043 + 31 * B
    with ps_mf.PsMf(N, M, K, P, s, 0.01, 0.05, policy=policy, B=B, mb_seed=seed, owner=owner, host_only=True,
                    cells=True, heavy_min=64, hot_steps=1, dense_min=dense_min) as g:
        g.load_ratings(user, item, val)
        o = oracle.Oracle(N, M, K, P, s, 0.01, 0.05, policy, oracle.ROWMEAN, B, seed, owner)
        o.load(user, item, val)
        compare_layout(g, o, B, N, M)
        for b in range(B):
            sp = split_of(g, b)
            nb = g.export_index(ps_mf.IDX_COL, b).size
            assert sp[:3].sum() == nb and sp[3:6].sum() == nb
            assert sp[0] == sp[3] and sp[0] > 0
            if dense_min == 1 and B == 1:
                # every tile with a rating is dense: only the repeats of a (user, item) pair
                # stay sparse
                assert sp[0] == np.unique(user.astype(np.int64) * M + item).size


def test_dense_tiles_need_a_supported_rank():
    for K, ok in [(8, False), (16, True), (128, True), (129, True), (256, True), (257, False)]:
        with ps_mf.PsMf(40, 30, K, 2, 1, 0.01, 0.05, host_only=True, dense_min=5) as g:
            u = np.arange(40, dtype=np.int32).repeat(30)
            i = np.tile(np.arange(30, dtype=np.int32), 40)
            if ok:
                g.load_ratings(u, i, np.ones(u.size, np.float32))
                assert split_of(g)[0] == u.size
            else:
                with pytest.raises(ps_mf.PsMfError) as e:
                    g.load_ratings(u, i, np.ones(u.size, np.float32))
                assert e.value.code == ps_mf.EINVAL
    # the automatic threshold never fails: it leaves unsupported ranks without dense tiles
    with ps_mf.PsMf(40, 30, 8, 2, 1, 0.01, 0.05, host_only=True) as g:
        g.load_ratings(np.arange(40, dtype=np.int32).repeat(30), np.tile(np.arange(30, dtype=np.int32), 40),
                       np.ones(1200, np.float32))
        assert split_of(g)[0] == 0
    h = ps_mf.ps_mf_create(4, 3, 16, 1, 0, 0.1, 0.1)
    try:
        for bad in (-2, 4097):
            with pytest.raises(ps_mf.PsMfError) as e:
                ps_mf.ps_mf_set_option(h, ps_mf.OPT_DENSE_MIN, bad)
            assert e.value.code == ps_mf.EINVAL
    finally:
        ps_mf.ps_mf_destroy(h)


@pytest.mark.parametrize("policy", [ps_mf.SSP_ROW, ps_mf.ESSP_ROW])
def test_per_row_policies_on_a_host_only_handle(policy):
    """The per-row policies build the same integer layout (their clients are the worker
    classes p mod (s+1)); before any clock no row is cached and no read is counted."""
    from paper_1410_8043_amd import synth
    spec = synth.scaled(synth.CONFIGS["medium"], 0.03)
    w = synth.generate(spec, K=1)
    with ps_mf.PsMf(spec.N, spec.M, 16, spec.P, 3, 0.01, 0.05, policy=policy, B=spec.B, mb_seed=spec.seed,
                    host_only=True) as g:
        g.load_ratings(w.user, w.item, w.val)
        o = oracle.Oracle(spec.N, spec.M, 16, spec.P, 3, 0.01, 0.05, policy, oracle.ROWMEAN, spec.B, spec.seed)
        o.load(w.user, w.item, w.val)
        compare_layout(g, o, spec.B, spec.N, spec.M)
        rv = g.export_index(ps_mf.IDX_ROW_VERSIONS)
        assert rv.size == spec.N + min(spec.P, 4) * spec.M and np.all(rv == -1)
        assert g.export_index(ps_mf.IDX_STALENESS).tolist() == [0, 0, 0, 0]
    h = ps_mf.ps_mf_create(4, 3, 2, 1, 0, 0.1, 0.1)
    try:
        with pytest.raises(ps_mf.PsMfError) as e:
            ps_mf.ps_mf_set_option(h, ps_mf.OPT_POLICY, 6)
        assert e.value.code == ps_mf.EINVAL
    finally:
        ps_mf.ps_mf_destroy(h)


# ---------------------------------------------------------------- sequential step (STEP_SEQ)
@pytest.mark.parametrize("P,G,B,policy,custom_owner", [(1, 1, 1, ps_mf.SSP_LAZY, False), (3, 4, 2, ps_mf.SSP_WORST, False),
                                                       (5, 7, 3, ps_mf.ESSP, True), (4, 64, 1, ps_mf.SSP_LAZY, True)])
def test_seq_order_is_bit_exact_with_oracle(P, G, B, policy, custom_owner):
    """Host-only SEQ handle: the library's self-check of the order, chains and flags passes,
    and its export of the order equals the oracle's, bit for bit."""
    rng = np.random.default_rng(P * 7 + G)
    N, M, n = 61, 37, 900
    user = rng.integers(0, N, n).astype(np.int32)
    item = rng.integers(0, M, n).astype(np.int32)
    val = rng.integers(1, 6, n).astype(np.float32)
    owner = rng.integers(0, P, N).astype(np.int32) if custom_owner else None
    with ps_mf.PsMf(N, M, 8, P, 2, 0.01, 0.05, policy=policy, step=ps_mf.STEP_SEQ, strata=G, B=B, mb_seed=5,
                    owner=owner, host_only=True) as g:
        g.load_ratings(user, item, val)
        o = oracle.Oracle(N, M, 8, P, 2, 0.01, 0.05, policy, oracle.SEQ, B, 5, owner, strata=G)
        o.load(user, item, val)
        compare_layout(g, o, B, N, M)
        for b in range(B):
            assert np.array_equal(g.export_index(ps_mf.IDX_SEQ_ORDER, b), o.export(oracle.X_SEQ_ORDER, b))
        o.close()


def test_seq_order_on_generated_workload():
    from paper_1410_8043_amd import synth
    spec = synth.scaled(synth.CONFIGS["medium"], 0.02)
    w = synth.generate(spec, K=1)
    with ps_mf.PsMf(spec.N, spec.M, 16, spec.P, 3, 0.01, 0.05, step=ps_mf.STEP_SEQ, strata=16, B=spec.B,
                    mb_seed=spec.seed, host_only=True) as g:
        g.load_ratings(w.user, w.item, w.val)
        o = oracle.Oracle(spec.N, spec.M, 16, spec.P, 3, 0.01, 0.05, oracle.SSP_LAZY, oracle.SEQ, spec.B, spec.seed,
                          strata=16)
        o.load(w.user, w.item, w.val)
        for b in range(spec.B):
            assert np.array_equal(g.export_index(ps_mf.IDX_SEQ_ORDER, b), o.export(oracle.X_SEQ_ORDER, b))
        # block 0: its ratings, one user run per (user, sub-epoch) pair with ratings
        split = g.export_index(ps_mf.IDX_SPLIT, 0).tolist()
        sel = o.export(oracle.X_SEQ_ORDER, 0)
        u, i = w.user[sel].astype(np.int64), w.item[sel].astype(np.int64)
        runs = np.unique(u * 16 + ((i % 16) - (u // spec.P) % 16) % 16).size
        assert split[1] == runs and split[2] == sel.size
        assert 0 < split[0] <= split[1] <= split[2] and split[3:] == [0] * 5
        o.close()


def test_seq_option_errors():
    h = ps_mf.ps_mf_create(4, 3, 2, 2, 1, 0.1, 0.1)
    try:
        for v in (0, 4097):
            with pytest.raises(ps_mf.PsMfError) as e:
                ps_mf.ps_mf_set_option(h, ps_mf.OPT_SEQ_STRATA, v)
            assert e.value.code == ps_mf.EINVAL
        ps_mf.ps_mf_set_option(h, ps_mf.OPT_HOST_ONLY, 1)
        ps_mf.ps_mf_load_ratings(h, np.array([0, 3]), np.array([2, 0]), np.array([1.0, 5.0]))
        with pytest.raises(ps_mf.PsMfError) as e:
            ps_mf.ps_mf_export_index(h, ps_mf.IDX_SEQ_ORDER, 0)
        assert e.value.code == ps_mf.EINVAL
    finally:
        ps_mf.ps_mf_destroy(h)
    for policy in (ps_mf.SSP_ROW, ps_mf.ESSP_ROW):  # the per-row caches work with the sequential step
        with ps_mf.PsMf(4, 3, 2, 2, 1, 0.1, 0.1, policy=policy, step=ps_mf.STEP_SEQ, host_only=True) as g:
            g.load_ratings(np.array([0, 3]), np.array([0, 2]), np.array([1.0, 2.0]))
            assert g.export_index(ps_mf.IDX_SEQ_ORDER).size == 2


# ---------------------------------------------------------------- value-bounded views (PS_MF_VAP)
def test_vap_arguments_and_host_layout():
    h = ps_mf.ps_mf_create(4, 3, 2, 2, 1, 0.1, 0.1)
    try:
        for v0 in (-1.0, float("nan")):
            with pytest.raises(ps_mf.PsMfError) as e:
                ps_mf.ps_mf_set_value_bound(h, v0)
            assert e.value.code == ps_mf.EINVAL
        ps_mf.ps_mf_set_value_bound(h, float("inf"))
        ps_mf.ps_mf_set_option(h, ps_mf.OPT_HOST_ONLY, 1)
        ps_mf.ps_mf_load_ratings(h, np.array([0, 3]), np.array([2, 0]), np.array([1.0, 5.0]))
        with pytest.raises(ps_mf.PsMfError) as e:
            ps_mf.ps_mf_set_value_bound(h, 1.0)
        assert e.value.code == ps_mf.ESTATE
        with pytest.raises(ps_mf.PsMfError) as e:
            ps_mf.ps_mf_export_index(h, ps_mf.IDX_VAP_NORMS, 0)
        assert e.value.code == ps_mf.EINVAL
    finally:
        ps_mf.ps_mf_destroy(h)
    rng = np.random.default_rng(3)
    N, M, P = 40, 30, 3
    user, item = rng.integers(0, N, 500).astype(np.int32), rng.integers(0, M, 500).astype(np.int32)
    val = rng.integers(1, 6, 500).astype(np.float32)
    with ps_mf.PsMf(N, M, 8, P, 2, 0.01, 0.05, policy=ps_mf.VAP, value_bound=0.1, B=2, mb_seed=4,
                    host_only=True) as g:
        g.load_ratings(user, item, val)
        o = oracle.Oracle(N, M, 8, P, 2, 0.01, 0.05, oracle.VAP, oracle.ROWMEAN, 2, 4, value_bound=0.1)
        o.load(user, item, val)
        compare_layout(g, o, 2, N, M)
        assert g.export_index(ps_mf.IDX_VAP_NORMS).size == 0 and g.export_index(ps_mf.IDX_VERSION_LOG).size == 0
        o.close()


def test_noalloc_loss_rejects_inputs_beyond_its_static_scratch():
    # ps_mf_loss_noalloc keeps one fp64 partial sum per loss workgroup in a fixed array of
    # 2^18; at K <= 8 a workgroup takes 128 users' segments, so 2^25 + 64 users with one
    # rating each need 2^18 + 1 partials.  The check comes before any device work (a
    # host-only handle), and an input that fits only meets the missing device state.
    from paper_1410_8043_amd import ps_mf as m

    for n, code, text in (((1 << 25) + 64, m.EINVAL, "static scratch holds 262144"),
                          (1 << 12, m.ESTATE, "set factors")):
        h = m.ps_mf_create(n, 8, 8, 64, 0, 0.1, 0.1)
        try:
            m.ps_mf_set_option(h, m.OPT_HOST_ONLY, 1)
            u = np.arange(n, dtype=np.int32)
            m.ps_mf_load_ratings(h, u, u % 8, np.ones(n, np.float32))
            with pytest.raises(m.PsMfError) as e:
                m.ps_mf_loss_noalloc(h)
            assert e.value.code == code and text in str(e.value), str(e.value)
        finally:
            m._lib.ps_mf_destroy(h)


def test_tile_device_and_poison_options_are_checked():
    from paper_1410_8043_amd import ps_mf as m

    h = m.ps_mf_create(4, 3, 2, 2, 1, 0.1, 0.1)
    try:
        for key, val in [(m.OPT_ITEM_TILE_BYTES, 0), (m.OPT_ITEM_TILE_BYTES, -2), (m.OPT_DEVICE, -2),
                         (m.OPT_DEVICE, 4096)]:
            with pytest.raises(m.PsMfError) as e:
                m.ps_mf_set_option(h, key, val)
            assert e.value.code == m.EINVAL
        m.ps_mf_set_option(h, m.OPT_ITEM_TILE_BYTES, 1 << 20)
        m.ps_mf_set_option(h, m.OPT_ITEM_TILE_BYTES, -1)
        m.ps_mf_set_option(h, m.OPT_DEVICE, 0)
        m.ps_mf_set_option(h, m.OPT_DEVICE, -1)
    finally:
        m.ps_mf_destroy(h)
    # the poison check covers the fixed-view commit only: refused with the sequential step
    with m.PsMf(4, 3, 2, 2, 1, 0.1, 0.1, step=m.STEP_SEQ, poison=True, host_only=True) as g:
        with pytest.raises(m.PsMfError) as e:
            g.load_ratings(np.array([0, 3]), np.array([2, 0]), np.array([1.0, 5.0]))
        assert e.value.code == m.EINVAL and "poison" in str(e.value)
    with m.PsMf(4, 3, 2, 2, 1, 0.1, 0.1, poison=True, host_only=True) as g:
        g.load_ratings(np.array([0, 3]), np.array([2, 0]), np.array([1.0, 5.0]))


@pytest.mark.parametrize("item_tile_bytes", [256, 16384])
def test_user_major_item_tiles_split_the_units(item_tile_bytes):
    # smaller item tiles cut each user's units at item-range boundaries (tiles double while
    # units would average fewer than 16 ratings): more units and partial rows, the same
    # ratings; the layout's own self-check (host-only) passes
    from paper_1410_8043_amd import ps_mf as m

    N, M, K = 2000, 1000, 16
    rng = np.random.default_rng(17)
    cells = rng.choice(N * M, 400_000, replace=False)
    u, i = (cells // M).astype(np.int32), (cells % M).astype(np.int32)
    v = rng.integers(1, 6, cells.size).astype(np.float32)
    out = []
    for itb in (None, item_tile_bytes):
        with m.PsMf(N, M, K, 8, 3, 0.01, 0.05, host_only=True, item_tile_bytes=itb, dense_min=0, cells=0) as g:
            g.load_ratings(u, i, v)
            out.append(g.export_index(m.IDX_SPLIT))
    assert out[0][2] == out[1][2] == cells.size
    assert out[0][6] == N and out[1][6] >= 4 * N


def test_automatic_split_uses_dense_tiles_and_cells_only_on_large_blocks():
    """With the automatic thresholds, blocks of fewer than 2^24 ratings send every rating
    through the work units; larger blocks put their densest part into dense (matrix-core)
    tiles and LDS cells.  The same 17.6M ratings as one block and as two blocks."""
    from paper_1410_8043_amd import synth

    spec = synth.scaled(synth.CONFIGS["full"], 0.42)
    w = synth.generate(spec, K=1)
    assert w.nnz >= 1 << 24 > w.nnz // 2
    for B in (1, 2):
        with ps_mf.PsMf(spec.N, spec.M, 128, spec.P, 3, spec.eta, spec.lam, B=B, mb_seed=spec.seed,
                        host_only=True) as g:
            g.load_ratings(w.user, w.item, w.val)
            split = sum(g.export_index(ps_mf.IDX_SPLIT, b) for b in range(B))
        assert split[0] + split[1] + split[2] == w.nnz and split[3:6].tolist() == split[0:3].tolist()
        if B == 1:
            assert split[0] > 0 and split[1] > 0 and split[2] > 0, split
        else:
            assert split[0] == 0 and split[1] == 0 and split[2] == w.nnz, split
