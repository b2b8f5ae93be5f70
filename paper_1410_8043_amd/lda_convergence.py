"""LDA convergence per clock under BSP, SSP and ESSP, measured on the GPU (arXiv 1410.8043, §5).

The paper trains LDA by collapsed Gibbs sampling with 50% of the tokens per Clock() and
compares the consistency models by the log-likelihood reached per iteration and per
second (its convergence figure).  This script runs the library on a seeded synthetic
corpus for each policy and staleness and prints, as a markdown table, the collapsed
log-likelihood after selected clocks and the kernel time per clock.  BSP is s = 0 (every
worker reads the previous clock's version).

    python -m paper_1410_8043_amd.lda_convergence [--corpus small] [--workers 256] [--clocks 40]
        [--s 3 7] [--at 2 4 10 20 40]
"""
from __future__ import annotations

import argparse

POLICIES = {"lazy": 0, "worst": 1, "essp": 2}


def trace(spec, corpus, P: int, s: int, policy: int, at):
    """Log-likelihood after each clock count in `at`, and the mean sampling-kernel ms per clock."""
    import torch

    from paper_1410_8043_amd import ps_lda

    g = ps_lda.PsLda(spec.D, spec.V, spec.K, P, s, spec.alpha, spec.beta, policy=policy, B=spec.B, seed=spec.seed,
                     timing=True, stream=torch.cuda.current_stream())
    g.load(corpus.doc, corpus.word, corpus.z0)
    out = [g.loglik()]
    done = 0
    for c in at:
        g.clock(c - done)
        done = c
        out.append(g.loglik())
    ms, n = g.kernel_time()
    g.close()
    return out, ms / max(n, 1)


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--corpus", default="small")
    ap.add_argument("--workers", type=int, default=None, help="P (default: the corpus's)")
    ap.add_argument("--s", type=int, nargs="+", default=[3, 7])
    ap.add_argument("--at", type=int, nargs="+", default=[2, 4, 10, 20, 40], help="clock counts to report")
    args = ap.parse_args(argv)
    import torch

    from paper_1410_8043_amd.synth import lda_corpus as lc

    torch.cuda.set_device(0)
    spec = lc.CORPORA[args.corpus]
    P = args.workers or spec.P
    corpus = lc.generate(spec)
    at = sorted(set(args.at))
    runs = [("BSP (s=0)", 0, POLICIES["essp"])]
    for s in args.s:
        runs += [(f"SSP lazy s={s}", s, POLICIES["lazy"]), (f"SSP worst s={s}", s, POLICIES["worst"]),
                 (f"ESSP s={s}", s, POLICIES["essp"])]
    print(f"corpus {args.corpus}: {spec.D} documents, {spec.V} words, {corpus.ntok} tokens, K={spec.K}, P={P}, "
          f"B={spec.B} (one clock = 1/{spec.B} of the tokens); collapsed log-likelihood / 1e6")
    print()
    print("| policy | ms / clock | clock 0 | " + " | ".join(f"clock {c}" for c in at) + " |")
    print("|---|---|---|" + "---|" * len(at))
    for name, s, pol in runs:
        ll, ms = trace(spec, corpus, P, s, pol, at)
        print(f"| {name} | {ms:.2f} | " + " | ".join(f"{x / 1e6:.4f}" for x in ll) + " |", flush=True)


if __name__ == "__main__":
    main()
