"""Brute-force clocked SSP / ESSP collapsed Gibbs sampling for LDA (test helper).

A different code shape from the oracle: every committed version of the shared counts is
kept (a list of dense [V+1, K] arrays, row V the topic totals) and the view of worker p at
clock c is read from that history directly; each worker works on a private copy of its
view that it updates in place, and the clock's new version is the latest version plus
the sum over workers of (copy - view).  Same reading of the draw: with
p_k = ((n_dk + alpha)(n_wk + beta)) / (n_k + V beta) over counts that exclude the token
(floored at zero), e the binary exponent of the largest p_k and c_K = ceil(log2 K), the
weights are floor(p_k 2^(62 - c_K - e)); the new topic is the first whose prefix sum of
weights exceeds floor(r W / 2^64).
"""
import numpy as np

from tests.dense_ref import delay, splitmix64

M64 = (1 << 64) - 1
DRAW_SALT = 0x5851F42D4C957F2D


def token_block(t, seed, B):
    return 0 if B == 1 else splitmix64((seed ^ t) & M64) % B


def draw(nd, nw, nk, k0, alpha, beta, Vb, r):
    K = nd.shape[0]
    self_ = np.zeros(K, np.int64)
    self_[k0] = 1
    a = (nd.astype(np.int64) - self_).astype(np.float64) + alpha
    b = np.maximum(nw.astype(np.int64) - self_, 0).astype(np.float64) + beta
    c = np.maximum(nk.astype(np.int64) - self_, 0).astype(np.float64) + Vb
    p = (a * b) / c
    # frexp: p = m 2^x with m in [0.5, 1), so the binary exponent is x - 1
    e = int(np.frexp(p)[1].max()) - 1
    shift = 62 - (K - 1).bit_length() - e
    w = [int(x) for x in np.floor(np.ldexp(p, shift))]
    total = sum(w)
    target = (r * total) >> 64
    cum = 0
    for k in range(K):
        cum += w[k]
        if cum > target:
            return k
    raise AssertionError("prefix sums end at the total")


def run_lda_dense(doc, word, z0, *, D, V, K, P, s, alpha, beta, policy, B, seed, clocks):
    """Returns (z, ndk [D, K], n [V+1, K] latest version, version log [clocks, P])."""
    doc = np.asarray(doc, np.int64)
    word = np.asarray(word, np.int64)
    z = np.asarray(z0, np.int64).copy()
    n_tok = doc.shape[0]
    ndk = np.zeros((D, K), np.int64)
    n0 = np.zeros((V + 1, K), np.int64)
    for t in range(n_tok):
        ndk[doc[t], z[t]] += 1
        n0[word[t], z[t]] += 1
        n0[V, z[t]] += 1
    hist = [n0]
    blocks = [token_block(t, seed, B) for t in range(n_tok)]
    Vb = V * beta
    vlog = []
    for c in range(clocks):
        b = c % B
        new = hist[c].copy()
        row = []
        for p in range(P):
            v = max(0, c - delay(policy, p, c, s))
            row.append(v)
            view = hist[v]
            mine = view.copy()
            toks = sorted((int(doc[t]), t) for t in range(n_tok) if blocks[t] == b and doc[t] % P == p)
            for d, t in toks:
                w, k0 = word[t], int(z[t])
                r = splitmix64((seed ^ DRAW_SALT ^ (c << 40) ^ t) & M64)
                k1 = draw(ndk[d], mine[w], mine[V], k0, alpha, beta, Vb, r)
                if k1 != k0:
                    ndk[d, k0] -= 1
                    ndk[d, k1] += 1
                    mine[w, k0] -= 1
                    mine[w, k1] += 1
                    mine[V, k0] -= 1
                    mine[V, k1] += 1
                    z[t] = k1
            new += mine - view
        hist.append(new)
        vlog.append(row)
    return z, ndk, hist[-1], np.array(vlog, np.int64).reshape(clocks, P)
