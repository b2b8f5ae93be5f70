"""Pins of the LDA collapsed-Gibbs oracle (Section 5's topic-model workload under SSP/ESSP).

Each check rests on something other than the oracle's own code:
  - count invariants: the shared counts of the latest version and the doc-topic counts are
    exactly the tallies of the assignments (a sign or index slip in the in-clock changes
    or the commit breaks them);
  - the collapsed log p(w, z) equals the chain rule's sum of one-token predictive log
    probabilities, which needs no Gamma function (a dropped or misplaced term fails);
  - closed forms of the log-likelihood (one token; one word and one topic);
  - the exact posterior p(z | w) of a 16-state problem, by enumeration, is what one
    worker's sweeps (P = 1, s = 0: plain sequential collapsed Gibbs) visit in the long run
    (a count that does not exclude the token, a missing prior or a wrong normaliser moves it);
  - a brute-force reference that keeps every version and reads views from that history
    matches the oracle bit for bit under every policy (ring slots, views, block split,
    worker order, the commit);
  - the views the oracle logs are the ones the staleness bound admits.
"""
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_1410_8043_amd.synth import lda_corpus as lc
from tests.lda_dense_ref import run_lda_dense, token_block


POLICIES = [oracle.SSP_LAZY, oracle.SSP_WORST, oracle.ESSP]


def _tiny(**over):
    return lc.scaled(lc.CORPORA["tiny"], 1.0, **over)


def _run(spec, corpus, policy, clocks):
    o = oracle.LdaOracle(spec.D, spec.V, spec.K, spec.P, spec.s, spec.alpha, spec.beta, policy, spec.B, spec.seed)
    o.load(corpus.doc, corpus.word, corpus.z0)
    o.clock(clocks)
    return o


def _tallies(doc, word, z, D, V, K):
    ndk = np.zeros((D, K), np.int64)
    n = np.zeros((V + 1, K), np.int64)
    np.add.at(ndk, (doc, z), 1)
    np.add.at(n, (word, z), 1)
    np.add.at(n, (np.full_like(word, V), z), 1)
    return ndk, n


def chain_rule_loglik(doc, word, z, D, V, K, alpha, beta):
    """log p(w, z) = sum over tokens of log p(z_i, w_i | earlier tokens): the topic given the
    document's earlier topics times the word given the topic's earlier words."""
    ndk = np.zeros((D, K))
    nd = np.zeros(D)
    nwk = np.zeros((V, K))
    nk = np.zeros(K)
    ll = 0.0
    for d, w, k in zip(doc, word, z):
        ll += math.log((ndk[d, k] + alpha) / (nd[d] + K * alpha))
        ll += math.log((nwk[w, k] + beta) / (nk[k] + V * beta))
        ndk[d, k] += 1
        nd[d] += 1
        nwk[w, k] += 1
        nk[k] += 1
    return ll


@pytest.mark.parametrize("policy", POLICIES)
def test_counts_are_tallies_of_assignments(policy):
    spec = _tiny()
    corpus = lc.generate(spec)
    o = _run(spec, corpus, policy, 0)
    for c in range(6):
        z = o.z()
        assert z.min() >= 0 and z.max() < spec.K
        ndk, n = _tallies(corpus.doc, corpus.word, z, spec.D, spec.V, spec.K)
        np.testing.assert_array_equal(o.ndk(), ndk)
        np.testing.assert_array_equal(o.nwk(), n)
        assert int(o.nwk()[spec.V].sum()) == corpus.ntok
        o.clock(1)
    assert (o.z() != corpus.z0).mean() > 0.3  # the sampler moved


@pytest.mark.parametrize("policy", POLICIES)
def test_loglik_is_chain_rule(policy):
    spec = _tiny(D=40)
    corpus = lc.generate(spec)
    o = _run(spec, corpus, policy, 3)
    ref = chain_rule_loglik(corpus.doc, corpus.word, o.z(), spec.D, spec.V, spec.K, spec.alpha, spec.beta)
    assert o.loglik() == pytest.approx(ref, rel=1e-11)
    # the chain rule holds in any token order: the sum does not depend on it
    perm = np.random.default_rng(5).permutation(corpus.ntok)
    ref2 = chain_rule_loglik(corpus.doc[perm], corpus.word[perm], o.z()[perm], spec.D, spec.V, spec.K, spec.alpha,
                             spec.beta)
    assert ref2 == pytest.approx(ref, rel=1e-11)


def test_loglik_closed_forms():
    # one token: p(z) = alpha / (K alpha) = 1/K, p(w | z) = beta / (V beta) = 1/V
    o = oracle.LdaOracle(1, 7, 3, 1, 0, 0.3, 0.05, oracle.ESSP, 1, 1)
    o.load([0], [4], [2])
    assert o.loglik() == pytest.approx(-math.log(3) - math.log(7), rel=1e-14)
    # K = 1, V = 1, one document of n tokens: log p = 0 (every topic and word is forced)
    o = oracle.LdaOracle(1, 1, 1, 1, 0, 0.7, 0.2, oracle.ESSP, 1, 1)
    o.load([0] * 5, [0] * 5, [0] * 5)
    assert o.loglik() == pytest.approx(0.0, abs=1e-12)
    # K = 1, one document: p(w) is the Dirichlet-multinomial (Polya urn) of the word counts
    words = [0, 1, 1, 2, 1]
    V, beta = 3, 0.4
    o = oracle.LdaOracle(1, V, 1, 1, 0, 0.5, beta, oracle.ESSP, 1, 1)
    o.load([0] * 5, words, [0] * 5)
    urn, seen = 0.0, [0] * V
    for i, w in enumerate(words):
        urn += math.log((seen[w] + beta) / (i + V * beta))
        seen[w] += 1
    assert o.loglik() == pytest.approx(urn, rel=1e-13)


def _posterior(doc, word, D, V, K, alpha, beta):
    states = list(itertools.product(range(K), repeat=len(doc)))
    logp = np.array([chain_rule_loglik(doc, word, np.array(z), D, V, K, alpha, beta) for z in states])
    p = np.exp(logp - logp.max())
    return states, p / p.sum()


def test_sequential_sampler_reaches_the_exact_posterior():
    # 2 documents, 2 words, 2 topics, 4 tokens: 16 assignments, posterior by enumeration
    doc = np.array([0, 0, 1, 1])
    word = np.array([0, 1, 0, 0])
    D, V, K, alpha, beta = 2, 2, 2, 0.5, 0.5
    states, post = _posterior(doc, word, D, V, K, alpha, beta)
    index = {s: i for i, s in enumerate(states)}
    o = oracle.LdaOracle(D, V, K, 1, 0, alpha, beta, oracle.ESSP, 1, 77)
    o.load(doc, word, [0, 0, 0, 0])
    sweeps, burn = 60000, 100
    hits = np.zeros(len(states))
    for c in range(sweeps):
        o.clock(1)
        if c >= burn:
            hits[index[tuple(int(x) for x in o.z())]] += 1
    freq = hits / hits.sum()
    # 60k correlated sweeps: per-state standard error about 0.002
    assert np.abs(freq - post).max() < 0.012, (freq, post)
    assert 0.5 * np.abs(freq - post).sum() < 0.03


@pytest.mark.parametrize("policy", POLICIES)
@pytest.mark.parametrize("P,s,B", [(3, 2, 2), (4, 1, 3), (1, 0, 1), (5, 3, 1)])
def test_matches_brute_force_history(policy, P, s, B):
    spec = _tiny(D=30, V=40, K=5, P=P, s=s, B=B)
    corpus = lc.generate(spec)
    clocks = 7
    o = _run(spec, corpus, policy, clocks)
    z, ndk, n, vlog = run_lda_dense(corpus.doc, corpus.word, corpus.z0, D=spec.D, V=spec.V, K=spec.K, P=P, s=s,
                                    alpha=spec.alpha, beta=spec.beta, policy=policy, B=B, seed=spec.seed,
                                    clocks=clocks)
    np.testing.assert_array_equal(o.z(), z)
    np.testing.assert_array_equal(o.ndk(), ndk)
    np.testing.assert_array_equal(o.nwk(), n)
    np.testing.assert_array_equal(o.export(oracle.LDA_VERSION_LOG).reshape(clocks, P), vlog)


@pytest.mark.parametrize("alpha", [1e-6, 1e-9])
def test_matches_brute_force_with_extreme_weight_ratios(alpha):
    # one- and two-token documents with a tiny alpha: a lone token's topics weigh between
    # about alpha and 1, so the weights span six to nine decades and the scale is set by
    # the token's own topic
    spec = _tiny(D=120, V=10, K=6, P=3, s=1, B=2, mean_len=1, alpha=alpha, beta=0.5)
    corpus = lc.generate(spec)
    clocks = 6
    o = _run(spec, corpus, oracle.ESSP, clocks)
    z, ndk, n, _ = run_lda_dense(corpus.doc, corpus.word, corpus.z0, D=spec.D, V=spec.V, K=spec.K, P=spec.P,
                                 s=spec.s, alpha=alpha, beta=spec.beta, policy=oracle.ESSP, B=spec.B, seed=spec.seed,
                                 clocks=clocks)
    np.testing.assert_array_equal(o.z(), z)
    np.testing.assert_array_equal(o.ndk(), ndk)
    np.testing.assert_array_equal(o.nwk(), n)


def _paper_shape_token(rng, K, n_k, doc_topics, word_topics, k0):
    """Counts of one token at the 100M-token, V = 100k, K = 100 shape (each topic holds about
    1e6 tokens): a document of about 300 tokens over a few topics, a word used by a few
    topics, every count including the token itself (topic k0)."""
    nk = rng.integers(int(0.8 * n_k), int(1.2 * n_k), K).astype(np.int32)
    nd = np.zeros(K, np.int32)
    nd[doc_topics] = rng.integers(1, 120, len(doc_topics))
    nw = np.zeros(K, np.int32)
    nw[word_topics] = rng.integers(1, 3000, len(word_topics))
    nd[k0] = max(nd[k0], 1)
    nw[k0] = max(nw[k0], 1)
    return nd, nw, nk


def _exact_probabilities(nd, nw, nk, k0, alpha, beta, V):
    """The collapsed conditional in exact rational arithmetic (alpha and beta as the exact
    values of their doubles), the token excluded from every count."""
    a, b = Fraction(alpha), Fraction(beta)
    p = []
    for k in range(len(nd)):
        self_ = int(k == k0)
        p.append((int(nd[k]) - self_ + a) * (int(nw[k]) - self_ + b) / (int(nk[k]) - self_ + V * b))
    total = sum(p)
    return [x / total for x in p]


def test_draw_weights_at_the_paper_shape():
    # Section 5's topic-model shape: V = 100k words, K = 100 topics, 100M tokens, so every
    # topic total n_k is about 1e6.  A topic that neither the document nor the word uses
    # weighs only alpha beta / (n_k + V beta), about 1e-9 -- 3e-9 to 3e-5 of the token's total
    # weight here -- and must still keep its exact share.  Flooring loses less than one unit
    # per weight, so with pi_k the exact probability, |w_k / W - pi_k| <= (1 + K pi_k) / W,
    # W >= 2^(62 - c_K): every share is within 2^-40 of the exact one, every weight is
    # positive, and the smoothing-only topics are within 2^-24 of their own value (a fixed
    # absolute scale such as floor(p_k 2^24) floors them to zero)
    K, V, alpha, beta, n_k = 100, 100_000, 0.1, 0.01, 1_000_000
    o = oracle.LdaOracle(1, V, K, 1, 0, alpha, beta, oracle.ESSP, 1, 1)
    rng = np.random.default_rng(1410)
    ck = (K - 1).bit_length()
    for trial in range(40):
        doc_topics = rng.choice(K, int(rng.integers(1, 8)), replace=False)
        word_topics = rng.choice(K, int(rng.integers(1, 6)), replace=False)
        k0 = int(rng.choice(doc_topics))
        nd, nw, nk = _paper_shape_token(rng, K, n_k, doc_topics, word_topics, k0)
        w, total, _ = o.token_draw(nd, nw, nk, k0, int(rng.integers(0, 2**63)))
        assert total == sum(w) and total < 2**63
        assert 2 ** (62 - ck) <= max(w) < 2 ** (63 - ck)
        exact = _exact_probabilities(nd, nw, nk, k0, alpha, beta, V)
        smoothing_only = [k for k in range(K) if nd[k] - (k == k0) == 0 and nw[k] - (k == k0) == 0]
        assert smoothing_only, "the shape always leaves topics with neither document nor word counts"
        for k in range(K):
            err = abs(Fraction(w[k], total) - exact[k])
            assert err <= (1 + K * exact[k]) / total, (trial, k)
            assert err <= Fraction(1, 2**40), (trial, k)
            assert w[k] > 0, (trial, k)
        for k in smoothing_only:
            assert exact[k] < 1e-4
            assert abs(Fraction(w[k], total) - exact[k]) <= exact[k] / 2**24, (trial, k)


def test_draw_on_prefix_sum_boundaries():
    # the new topic is the first whose prefix sum of weights exceeds floor(r W / 2^64): a
    # random number that puts the target exactly on a prefix sum selects the next topic
    K, V = 7, 50
    o = oracle.LdaOracle(1, V, K, 1, 0, 0.3, 0.2, oracle.ESSP, 1, 1)
    nd = np.array([3, 0, 1, 0, 5, 2, 1], np.int32)
    nw = np.array([1, 2, 0, 0, 4, 1, 0], np.int32)
    nk = np.array([40, 31, 12, 9, 55, 20, 8], np.int32)
    w, total, _ = o.token_draw(nd, nw, nk, 0, 0)
    cum = np.cumsum(np.array(w, dtype=object))
    for k in range(K - 1):
        # the smallest r with floor(r W / 2^64) = cum[k]
        r = -((-int(cum[k]) << 64) // total)
        assert (r * total) >> 64 == cum[k]
        assert o.token_draw(nd, nw, nk, 0, r)[2] == k + 1, k
        # one below: the target is cum[k] - 1, still topic k
        assert o.token_draw(nd, nw, nk, 0, r - 1)[2] == k, k
    assert o.token_draw(nd, nw, nk, 0, 0)[2] == 0
    assert o.token_draw(nd, nw, nk, 0, 2**64 - 1)[2] == K - 1


def test_draw_matches_the_exact_conditional_in_frequency():
    # drawing with uniformly random r, topic frequencies follow the exact conditional
    # (including a topic the document does not use); 200k draws, standard error <= 0.0011
    K, V = 5, 30
    o = oracle.LdaOracle(1, V, K, 1, 0, 0.5, 0.1, oracle.ESSP, 1, 1)
    nd = np.array([4, 0, 2, 1, 3], np.int32)
    nw = np.array([2, 1, 0, 1, 5], np.int32)
    nk = np.array([30, 14, 22, 9, 41], np.int32)
    exact = [float(x) for x in _exact_probabilities(nd, nw, nk, 4, 0.5, 0.1, V)]
    rng = np.random.default_rng(3)
    hits = np.zeros(K)
    for r in rng.integers(0, 2**64, 200_000, dtype=np.uint64):
        hits[o.token_draw(nd, nw, nk, 4, int(r))[2]] += 1
    np.testing.assert_allclose(hits / hits.sum(), exact, atol=0.006)


def test_load_rejects_weights_outside_the_normal_range():
    # beta so small that the smoothing weight alpha beta / (n + V beta) is subnormal
    o = oracle.LdaOracle(2, 5, 2, 1, 0, 1e-200, 1e-200)
    with pytest.raises(oracle.OracleError):
        o.load([0, 1], [0, 1], [0, 1])


@pytest.mark.parametrize("policy", POLICIES)
def test_views_respect_the_staleness_bound(policy):
    spec = _tiny(P=6, s=3)
    corpus = lc.generate(spec)
    clocks = 12
    o = _run(spec, corpus, policy, clocks)
    vlog = o.export(oracle.LDA_VERSION_LOG).reshape(clocks, spec.P)
    c = np.arange(clocks)[:, None]
    assert (vlog <= c).all() and (vlog >= np.maximum(0, c - spec.s)).all()
    if policy == oracle.ESSP:
        assert (vlog == np.maximum(0, c - 1)).all()  # eager: every worker one clock behind
    if policy == oracle.SSP_WORST:
        assert (vlog == np.maximum(0, c - spec.s)).all()


def test_blocks_partition_the_tokens():
    spec = _tiny(B=3, P=5)
    corpus = lc.generate(spec)
    o = _run(spec, corpus, oracle.ESSP, 0)
    seen = np.concatenate([o.export(oracle.LDA_BLOCK_ORDER, b) for b in range(spec.B)])
    np.testing.assert_array_equal(np.sort(seen), np.arange(corpus.ntok))
    for b in range(spec.B):
        order = o.export(oracle.LDA_BLOCK_ORDER, b)
        assert all(token_block(int(t), spec.seed, spec.B) == b for t in order)
        key = np.stack([corpus.doc[order] % spec.P, corpus.doc[order], order], 1)
        assert (np.diff(key[:, 0]) >= 0).all()
        assert all(tuple(key[i]) < tuple(key[i + 1]) for i in range(len(order) - 1))
    sizes = [len(o.export(oracle.LDA_BLOCK_ORDER, b)) for b in range(spec.B)]
    assert min(sizes) > 0.25 * corpus.ntok


def test_stale_runs_still_raise_the_likelihood():
    spec = _tiny()
    corpus = lc.generate(spec)
    for policy in POLICIES:
        o = _run(spec, corpus, policy, 0)
        ll0 = o.loglik()
        o.clock(10)
        assert o.loglik() > ll0 + 0.1 * abs(ll0)


def test_argument_errors():
    with pytest.raises(oracle.OracleError):
        oracle.LdaOracle(0, 5, 2, 1, 0, 0.1, 0.1)
    with pytest.raises(oracle.OracleError):
        oracle.LdaOracle(2, 5, 2, 1, 0, -0.1, 0.1)
    with pytest.raises(oracle.OracleError):
        oracle.LdaOracle(2, 5, 2, 1, 0, 0.1, 0.1, policy=3)
    o = oracle.LdaOracle(2, 5, 2, 1, 0, 0.1, 0.1)
    with pytest.raises(oracle.OracleError):
        o.clock(1)  # nothing loaded
    with pytest.raises(oracle.OracleError):
        o.load([0, 2], [0, 1], [0, 0])  # document out of range
    with pytest.raises(oracle.OracleError):
        o.load([0, 1], [0, 5], [0, 0])  # word out of range
    with pytest.raises(oracle.OracleError):
        o.load([0, 1], [0, 1], [0, 2])  # topic out of range
    o.load([], [], [])
    o.clock(2)
    assert o.loglik() == pytest.approx(0.0, abs=0)


def test_policy_identities():
    # ESSP reads one clock back whatever s >= 1 is; at s = 0 every policy is BSP
    spec = _tiny(P=5)
    corpus = lc.generate(spec)

    def state(policy, s):
        o = oracle.LdaOracle(spec.D, spec.V, spec.K, spec.P, s, spec.alpha, spec.beta, policy, spec.B, spec.seed)
        o.load(corpus.doc, corpus.word, corpus.z0)
        o.clock(6)
        return o.z(), o.nwk()

    a, b = state(oracle.ESSP, 1), state(oracle.ESSP, 7)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])
    bsp = state(oracle.ESSP, 0)
    for pol in (oracle.SSP_LAZY, oracle.SSP_WORST):
        x = state(pol, 0)
        np.testing.assert_array_equal(x[0], bsp[0])
        np.testing.assert_array_equal(x[1], bsp[1])
    assert not np.array_equal(a[0], bsp[0])
    # SSP_WORST at s = 1 is ESSP at s = 1 (both read exactly one clock back)
    w = state(oracle.SSP_WORST, 1)
    np.testing.assert_array_equal(w[0], a[0])
