"""HIP collapsed-Gibbs LDA under SSP / ESSP vs the CPU oracle, through the C ABI (MI355X).

The sampler's state is integer (assignments, doc-topic counts, versioned word-topic counts)
and its draw is exact integer arithmetic over fp64 weights evaluated in the same IEEE
operations on both sides, so the bar is bit-exact: every assignment and count after every
checked clock.  The log-likelihood (fp64 sums of lgamma terms in different orders, the
library's lgamma against the C library's) within a relative 1e-9.
"""
import hashlib
import json
import os
import sys

import numpy as np
import pytest

import oracle
from paper_1410_8043_amd.synth import lda_corpus as lc

pytestmark = pytest.mark.gpu

LL_RTOL = 1e-9
POLICIES = [oracle.SSP_LAZY, oracle.SSP_WORST, oracle.ESSP]


@pytest.fixture(scope="module")
def lda():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_1410_8043_amd import ps_lda

    return ps_lda


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def both(lda, spec, corpus, policy, clocks, check_every=None, **opts):
    say(f"lda case {spec.name} D={spec.D} V={spec.V} K={spec.K} P={spec.P} s={spec.s} B={spec.B} "
        f"alpha={spec.alpha} policy={policy} tokens={corpus.ntok} clocks={clocks}")
    g = lda.PsLda(spec.D, spec.V, spec.K, spec.P, spec.s, spec.alpha, spec.beta, policy=policy, B=spec.B,
                  seed=spec.seed, **opts)
    g.load(corpus.doc, corpus.word, corpus.z0)
    o = oracle.LdaOracle(spec.D, spec.V, spec.K, spec.P, spec.s, spec.alpha, spec.beta, policy, spec.B, spec.seed)
    o.load(corpus.doc, corpus.word, corpus.z0)
    step = check_every or clocks
    done = 0
    while done < clocks:
        n = min(step, clocks - done)
        g.clock(n)
        o.clock(n)
        done += n
        np.testing.assert_array_equal(g.z(), o.z(), err_msg=f"assignments after {done} clocks")
        np.testing.assert_array_equal(g.ndk(), o.ndk(), err_msg=f"doc-topic counts after {done} clocks")
        np.testing.assert_array_equal(g.nwk(), o.nwk(), err_msg=f"word-topic counts after {done} clocks")
    np.testing.assert_array_equal(g.export(lda.X_VERSION_LOG), o.export(oracle.LDA_VERSION_LOG))
    assert g.get_clock() == clocks
    assert g.loglik() == pytest.approx(o.loglik(), rel=LL_RTOL)
    return g, o


@pytest.mark.parametrize("policy", POLICIES)
@pytest.mark.parametrize("P,s,B", [(4, 2, 2), (3, 0, 1), (7, 3, 3), (1, 1, 2)])
def test_tiny_corpus_bit_exact(lda, policy, P, s, B):
    spec = lc.scaled(lc.CORPORA["tiny"], 1.0, P=P, s=s, B=B)
    both(lda, spec, lc.generate(spec), policy, 10, check_every=3)


@pytest.mark.parametrize("K", [1, 2, 63, 64, 65, 100, 130, 200, 320, 512])
def test_every_topic_count_layout(lda, K):
    # one to eight topics per lane, ragged last lane group
    spec = lc.scaled(lc.CORPORA["tiny"], 0.3, K=K, V=80, P=3, s=1)
    both(lda, spec, lc.generate(spec), oracle.ESSP, 5)


@pytest.mark.parametrize("alpha", [1e-6, 1e-9])
def test_extreme_weight_ratios(lda, alpha):
    # one- and two-token documents with a tiny alpha: a token's weights span six to nine
    # decades, and the scale is set by its own topic
    spec = lc.scaled(lc.CORPORA["tiny"], 1.0, D=300, V=10, K=6, P=3, s=1, mean_len=1, alpha=alpha, beta=0.5)
    both(lda, spec, lc.generate(spec), oracle.ESSP, 6, check_every=2)


@pytest.mark.parametrize("K", [2, 100, 256, 512])
@pytest.mark.parametrize("policy", POLICIES)
def test_flat_addressing_bit_exact(lda, policy, K):
    # the 64-bit form of the sampling kernel (used for tables over 2 GiB), forced on small ones
    spec = lc.scaled(lc.CORPORA["tiny"], 1.0, K=K, P=5, s=2, B=2)
    both(lda, spec, lc.generate(spec), policy, 6, check_every=3, flat=True)


def test_more_workers_than_documents(lda):
    spec = lc.scaled(lc.CORPORA["tiny"], 1.0, D=40, P=300, s=2)
    both(lda, spec, lc.generate(spec), oracle.SSP_LAZY, 6)


def test_repeated_words_in_a_document(lda):
    # tiny vocabulary: a worker's consecutive tokens share a word, its delta row is read back at once
    spec = lc.scaled(lc.CORPORA["tiny"], 1.0, D=50, V=3, K=5, P=2, s=2, mean_len=40, beta=0.1)
    both(lda, spec, lc.generate(spec), oracle.SSP_WORST, 8, check_every=2)


def test_empty_corpus(lda):
    g = lda.PsLda(5, 7, 3, 2, 1, 0.1, 0.1)
    g.load([], [], [])
    g.clock(3)
    assert g.z().size == 0
    assert (g.ndk() == 0).all() and (g.nwk() == 0).all()
    assert g.loglik() == 0.0
    assert g.export(lda.X_VERSION_LOG).size == 6


def test_on_a_caller_stream_with_timing(lda):
    import torch

    spec = lc.scaled(lc.CORPORA["tiny"], 1.0)
    corpus = lc.generate(spec)
    st = torch.cuda.Stream()
    g, _ = both(lda, spec, corpus, oracle.ESSP, 4, stream=st, timing=True)
    ms, n = g.kernel_time()
    assert n == 4 and ms > 0


@pytest.mark.parametrize("policy", POLICIES)
def test_full_corpus_bit_exact(lda, policy):
    # 4.0M tokens, 20k words, K = 100, P = 64, s = 3, half the tokens per clock
    spec = lc.CORPORA["small"]
    both(lda, spec, lc.generate(spec), policy, 3 if policy == oracle.ESSP else 5, check_every=1)


def test_full_corpus_bit_exact_256_workers(lda):
    # the same corpus in the launch shape bench.py --workload lda --workers 256 times
    spec = lc.scaled(lc.CORPORA["small"], 1.0, P=256)
    both(lda, spec, lc.generate(spec), oracle.ESSP, 2, check_every=1)


def test_full_corpus_bit_exact_256_topics(lda):
    # four topics per lane at full size: the small corpus with K = 256
    spec = lc.scaled(lc.CORPORA["small"], 1.0, K=256)
    both(lda, spec, lc.generate(spec), oracle.SSP_LAZY, 2, check_every=1)


def test_full_corpus_counts_stay_tallies(lda):
    spec = lc.CORPORA["small"]
    corpus = lc.generate(spec)
    say(f"lda full-size tallies: tokens={corpus.ntok}")
    g = lda.PsLda(spec.D, spec.V, spec.K, spec.P, spec.s, spec.alpha, spec.beta, policy=lda.SSP_LAZY, B=spec.B,
                  seed=spec.seed)
    g.load(corpus.doc, corpus.word, corpus.z0)
    ll0 = g.loglik()
    g.clock(8)
    z = g.z()
    ndk = np.zeros((spec.D, spec.K), np.int64)
    np.add.at(ndk, (corpus.doc, z), 1)
    n = np.zeros((spec.V + 1, spec.K), np.int64)
    np.add.at(n, (corpus.word, z), 1)
    n[spec.V] = np.bincount(z, minlength=spec.K)
    np.testing.assert_array_equal(g.ndk(), ndk)
    np.testing.assert_array_equal(g.nwk(), n)
    assert g.loglik() > ll0


def _digest(a):
    """SHA-256 of an integer array as little-endian int32 in C order."""
    a = np.ascontiguousarray(a)
    return hashlib.sha256(a.astype("<i4").tobytes()).hexdigest()


def test_paper_scale_corpus_against_the_oracle(lda):
    # the paper's topic-model shape as bench.py --workload lda --corpus nyt runs it: 100M
    # tokens, 100k words, K = 100, P = 512 (eight ballot rounds of 64 workers in the
    # commit), half of the tokens per clock, ESSP.  The oracle's state after each of two
    # clocks is stored as SHA-256 digests (tests/golden/make_lda_nyt_golden.py, a few CPU
    # minutes); the GPU's assignments and counts must hash the same, i.e. be equal bit for
    # bit, and the counts must be the tallies of the assignments.
    with open(os.path.join(os.path.dirname(__file__), "golden", "lda_nyt_oracle.json")) as f:
        gold = json.load(f)
    spec = lc.CORPORA["nyt"]
    assert gold["corpus"]["name"] == spec.name and gold["policy"] == "ESSP"
    say("lda paper-scale corpus: generating")
    corpus = lc.generate(spec)
    assert corpus.ntok == gold["corpus"]["ntok"]
    for key in ("doc", "word", "z0"):
        assert _digest(getattr(corpus, key)) == gold["corpus"][key], f"the generator's {key} changed"
    say(f"lda paper-scale corpus: {corpus.ntok} tokens, loading")
    g = lda.PsLda(spec.D, spec.V, spec.K, spec.P, spec.s, spec.alpha, spec.beta, policy=lda.ESSP, B=spec.B,
                  seed=spec.seed)
    g.load(corpus.doc, corpus.word, corpus.z0)
    ll0 = g.loglik()
    K = spec.K
    for entry in gold["clocks"]:
        g.clock(1)
        z, ndk, nwk = g.z(), g.ndk(), g.nwk()
        say(f"lda paper-scale corpus: clock {entry['clock']}, {float((z != corpus.z0).mean()):.3f} moved")
        assert _digest(z) == entry["z"], f"assignments after clock {entry['clock']}"
        assert _digest(ndk) == entry["ndk"], f"doc-topic counts after clock {entry['clock']}"
        assert _digest(nwk) == entry["nwk"], f"word-topic counts after clock {entry['clock']}"
        assert g.loglik() == pytest.approx(entry["loglik"], rel=LL_RTOL)
    np.testing.assert_array_equal(ndk, np.bincount(corpus.doc.astype(np.int64) * K + z,
                                                   minlength=spec.D * K).reshape(spec.D, K))
    np.testing.assert_array_equal(nwk[:spec.V], np.bincount(corpus.word.astype(np.int64) * K + z,
                                                            minlength=spec.V * K).reshape(spec.V, K))
    np.testing.assert_array_equal(nwk[spec.V], np.bincount(z, minlength=K))
    assert g.loglik() > ll0
    g.close()


def test_policy_identities_at_full_size(lda):
    # properties that hold at any size: ESSP reads one clock back whatever s >= 1 is, and at
    # s = 0 every policy is BSP; each pair must agree bit for bit on the full small corpus
    spec = lc.CORPORA["small"]
    corpus = lc.generate(spec)

    def run(policy, s, clocks=4):
        g = lda.PsLda(spec.D, spec.V, spec.K, spec.P, s, spec.alpha, spec.beta, policy=policy, B=spec.B,
                      seed=spec.seed)
        g.load(corpus.doc, corpus.word, corpus.z0)
        g.clock(clocks)
        out = (g.z(), g.nwk(), g.export(lda.X_VERSION_LOG))
        g.close()
        return out

    say("lda policy identities: ESSP s=1 vs s=7, and the three policies at s=0")
    a, b = run(lda.ESSP, 1), run(lda.ESSP, 7)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])
    np.testing.assert_array_equal(a[2], b[2])
    bsp = run(lda.ESSP, 0)
    for pol in (lda.SSP_LAZY, lda.SSP_WORST):
        x = run(pol, 0)
        np.testing.assert_array_equal(x[0], bsp[0])
        np.testing.assert_array_equal(x[1], bsp[1])
    assert not np.array_equal(a[0], bsp[0])  # stale and fresh views do differ
