"""Seeded synthetic corpora shaped like the paper's topic-model experiment.

Section 5 of arXiv 1410.8043 runs LDA by collapsed Gibbs sampling on the New York Times
corpus (100M tokens, 100k words, K = 100 topics).  That corpus is not available, so these
generators stand in for it: documents drawn from the LDA generative process itself, with
Poisson document lengths, Dirichlet topic mixtures, and topics that favour Zipf-ranked
words.  This module produces inputs only (tokens and the initial topic of every token) and
holds none of the sampler's arithmetic.
"""
from __future__ import annotations

import dataclasses

import numpy as np

BASE_SEED = 0x14108043


@dataclasses.dataclass(frozen=True)
class CorpusSpec:
    name: str
    D: int            # documents
    V: int            # vocabulary
    K: int            # topics
    mean_len: float   # Poisson mean of the document length
    P: int            # workers (document d on worker d mod P)
    s: int            # staleness
    alpha: float      # doc-topic prior of the sampler
    beta: float       # topic-word prior of the sampler
    B: int            # token minibatch blocks (2: half the tokens per clock)
    clocks: int
    seed: int
    gen_alpha: float = 0.1   # generator: document topic mixtures ~ Dirichlet(gen_alpha)
    zipf: float = 1.05       # generator: word weights within a topic ~ rank^-zipf


CORPORA = {
    "tiny": CorpusSpec("tiny", D=200, V=300, K=8, mean_len=50, P=4, s=2, alpha=0.1, beta=0.01, B=2, clocks=10,
                       seed=BASE_SEED + 101),
    # 4M tokens, 100 topics: the paper's K, a vocabulary and corpus one GPU's sequential
    # workers sweep in well under a second per clock
    "small": CorpusSpec("small", D=20_000, V=20_000, K=100, mean_len=200, P=64, s=3, alpha=0.1, beta=0.01, B=2,
                        clocks=10, seed=BASE_SEED + 102),
    # the paper's topic-model workload shape: 100M tokens, 100k words, K = 100, half of the
    # tokens per clock, 512 workers (its 8 nodes x 64 cores)
    "nyt": CorpusSpec("nyt", D=300_000, V=100_000, K=100, mean_len=333, P=512, s=3, alpha=0.1, beta=0.01, B=2,
                      clocks=10, seed=BASE_SEED + 103),
}


@dataclasses.dataclass
class Corpus:
    doc: np.ndarray    # int32 [tokens], documents in order, tokens of a document contiguous
    word: np.ndarray   # int32 [tokens]
    z0: np.ndarray     # int32 [tokens] initial topics, uniform
    ntok: int


def scaled(spec: CorpusSpec, frac: float, **over) -> CorpusSpec:
    """The same laws with frac of the documents (at least 8)."""
    d = dict(dataclasses.asdict(spec))
    d["D"] = max(8, int(round(spec.D * frac)))
    d["name"] = f"{spec.name}@{frac:g}"
    d.update(over)
    return CorpusSpec(**d)


def generate(spec: CorpusSpec) -> Corpus:
    rng = np.random.default_rng(spec.seed)
    lens = np.maximum(1, rng.poisson(spec.mean_len, size=spec.D)).astype(np.int64)
    n = int(lens.sum())
    doc = np.repeat(np.arange(spec.D, dtype=np.int32), lens)
    theta = rng.dirichlet(np.full(spec.K, spec.gen_alpha), size=spec.D)
    # each topic ranks the vocabulary by its own permutation and weights rank r by r^-zipf
    base = 1.0 / np.arange(1, spec.V + 1) ** spec.zipf
    base /= base.sum()
    perms = np.stack([rng.permutation(spec.V) for _ in range(spec.K)])
    # a token's topic from its document's mixture, its word from that topic
    u = rng.random(n)
    cum_theta = np.cumsum(theta, axis=1)
    topic = np.empty(n, dtype=np.int64)
    start = 0
    for d in range(spec.D):
        end = start + int(lens[d])
        topic[start:end] = np.searchsorted(cum_theta[d], u[start:end] * cum_theta[d, -1], side="right")
        start = end
    topic = topic.clip(0, spec.K - 1)
    cum_base = np.cumsum(base)
    rank = np.searchsorted(cum_base, rng.random(n) * cum_base[-1]).clip(0, spec.V - 1)
    word = perms[topic, rank].astype(np.int32)
    z0 = rng.integers(0, spec.K, size=n).astype(np.int32)
    return Corpus(doc=doc, word=word, z0=z0, ntok=n)
