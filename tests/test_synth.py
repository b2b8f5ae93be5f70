"""The seeded workload generator: determinism, distinct pairs, degree laws (no GPU)."""
import numpy as np
import pytest

from paper_1410_8043_amd import synth


def test_tiny_config_shape_and_determinism():
    a = synth.generate("tiny")
    b = synth.generate("tiny")
    assert a.nnz == 20_000
    for x, y in [(a.user, b.user), (a.item, b.item), (a.val, b.val), (a.L0, b.L0), (a.R0, b.R0)]:
        assert np.array_equal(x, y)
    key = a.user.astype(np.int64) * 500 + a.item
    assert np.unique(key).size == a.nnz
    assert a.user.min() >= 0 and a.user.max() < 1000 and a.item.min() >= 0 and a.item.max() < 500
    assert set(np.unique(a.val)) <= {1.0, 2.0, 3.0, 4.0, 5.0}
    assert a.L0.shape == (1000, 16) and a.R0.shape == (500, 16)
    assert abs(a.L0.std() - 0.1) < 0.005 and abs(a.L0.mean()) < 0.005


def test_degrees_water_fill_exact_sum_and_cap():
    w = synth.rank_weights(1000, 1.1, 7, 0)
    d = synth.degrees(w, 50_000, 300)
    assert d.sum() == 50_000 and d.max() == 300 and d.min() >= 0
    # monotone in the weight
    order = np.argsort(-w, kind="stable")
    assert np.all(np.diff(d[order]) <= 0)


def test_zipf_pairs_are_distinct_and_follow_degrees():
    spec = synth.scaled(synth.CONFIGS["full"], 0.02)
    w = synth.generate(spec, K=4)
    key = w.user.astype(np.int64) * spec.M + w.item
    assert np.unique(key).size == w.nnz == spec.nnz
    uw = synth.rank_weights(spec.N, spec.user_zipf, spec.seed, 0)
    d = synth.degrees(uw, spec.nnz, spec.M)
    assert np.array_equal(np.bincount(w.user, minlength=spec.N), d)
    # heavy-tailed item popularity: the most popular item is far above the mean
    idg = np.bincount(w.item, minlength=spec.M)
    assert idg.max() > 5 * idg.mean()


def test_normal_generator_moments():
    x = synth.normal((200_000,), 0.5, 3, 9).astype(np.float64)
    assert abs(x.mean()) < 0.005 and abs(x.std() - 0.5) < 0.005
    # counter-based: a prefix does not depend on the length asked for
    y = synth.normal((1000,), 0.5, 3, 9)
    assert np.array_equal(y, x[:1000].astype(np.float32))


def test_lda_corpus_is_seeded_and_in_range():
    from paper_1410_8043_amd.synth import lda_corpus as lc
    spec = lc.scaled(lc.CORPORA["small"], 0.01)
    a, b = lc.generate(spec), lc.generate(spec)
    for x, y in ((a.doc, b.doc), (a.word, b.word), (a.z0, b.z0)):
        np.testing.assert_array_equal(x, y)
    assert a.ntok == a.doc.shape[0] == a.word.shape[0] == a.z0.shape[0]
    assert a.doc.dtype == a.word.dtype == a.z0.dtype == np.int32
    assert (np.diff(a.doc) >= 0).all() and a.doc.max() < spec.D
    assert 0 <= a.word.min() and a.word.max() < spec.V
    assert 0 <= a.z0.min() and a.z0.max() < spec.K
    assert abs(a.ntok / spec.D - spec.mean_len) < 0.05 * spec.mean_len
    # Zipf-shaped word frequencies: the most frequent words take a large share
    cnt = np.sort(np.bincount(a.word, minlength=spec.V))[::-1]
    assert cnt[:spec.V // 100].sum() > 0.1 * a.ntok  # uniform words would give 1%
