"""Dense brute force of clocked SSP matrix-factorization gradient descent (test helper).

A different code shape from the sparse oracle: the ratings become dense N x M matrices
(W = number of ratings of each cell, D = their mean value), and each clock is matrix
algebra on the objective F_w(L, R) = 1/2 sum_Omega [(D_ij - L_i.R_j)^2 + lambda(|L_i|^2 + |R_j|^2)]:
    E = W * (D - L R^T),  grad_L = -E R + lambda diag(n_u) L,  grad_R = -E^T L + lambda diag(n_i) R,
    x_{c+1} = fp32(x_c - eta S grad(x_view)),   S = I (SUM) or diag(1/n) (ROWMEAN).
With several workers each user's rows of E use that user's owner's view, and the item
gradient sums each worker's part at its own view.
"""
import numpy as np


def splitmix64(x):
    M = (1 << 64) - 1
    z = (x + 0x9E3779B97F4A7C15) & M
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M
    return z ^ (z >> 31)


def block_of(i, j, seed, B):
    if B == 1:
        return 0
    return splitmix64((seed ^ ((int(i) << 32) | int(j))) & ((1 << 64) - 1)) % B


def dense_mats(user, item, val, N, M, blocks=None, b=None):
    W = np.zeros((N, M))
    S = np.zeros((N, M))
    for t in range(len(user)):
        if blocks is not None and blocks[t] != b:
            continue
        W[user[t], item[t]] += 1
        S[user[t], item[t]] += float(val[t])
    D = np.divide(S, W, out=np.zeros_like(S), where=W > 0)
    return W, D


def delay(policy, p, c, s):
    if policy == 0:
        return (c + p % (s + 1)) % (s + 1)
    if policy == 1:
        return s
    return min(s, 1)


def vap_delay(hist, c, s, v0):
    """The value-bounded view: the largest d <= min(c, s) with max |x_c - x_{c-d}| (fp32
    differences of the stored versions) <= v0 / sqrt(c + 1)."""
    bound = v0 / np.sqrt(c + 1.0)
    d = 0
    for k in range(0, min(c, s) + 1):
        diff = max(np.abs(hist[c][0] - hist[c - k][0]).max(initial=0), np.abs(hist[c][1] - hist[c - k][1]).max(initial=0))
        if float(diff) <= bound:
            d = k
    return d


def run_dense(user, item, val, L0, R0, *, N, M, K, P, s, eta, lam, clocks, policy=0, step=0, B=1, seed=0,
              owner=None, vap_v0=None, eta_decay=False):
    """policy 0/1/2: SSP_LAZY / SSP_WORST / ESSP delays; vap_v0: the value-bounded view
    instead; eta_decay: step eta / sqrt(c + 1) at clock c."""
    owner = np.arange(N) % P if owner is None else np.asarray(owner)
    blocks = np.array([block_of(i, j, seed, B) for i, j in zip(user, item)]) if B > 1 else None
    mats = [dense_mats(user, item, val, N, M, blocks, b) for b in range(B)]
    hist = [(np.asarray(L0, np.float32).reshape(N, K).copy(), np.asarray(R0, np.float32).reshape(M, K).copy())]
    for c in range(clocks):
        W, D = mats[c % B]
        nu, ni = W.sum(1), W.sum(0)
        dL = np.zeros((N, K))
        dR = np.zeros((M, K))
        d_vap = vap_delay(hist, c, s, vap_v0) if vap_v0 is not None else None
        for p in range(P):
            rows = owner == p
            if not rows.any():
                continue
            v = max(0, c - (d_vap if d_vap is not None else delay(policy, p, c, s)))
            Lv, Rv = (x.astype(np.float64) for x in hist[v])
            Wp = W * rows[:, None]
            E = Wp * (D - Lv @ Rv.T)
            gL = -(E @ Rv) + lam * Wp.sum(1)[:, None] * Lv
            gR = -(E.T @ Lv) + lam * Wp.sum(0)[:, None] * Rv
            dL[rows] -= gL[rows]
            dR -= gR
        if step == 0:
            dL /= np.where(nu > 0, nu, 1)[:, None]
            dR /= np.where(ni > 0, ni, 1)[:, None]
        Lc, Rc = hist[c]
        eta_c = eta / np.sqrt(c + 1.0) if eta_decay else eta
        hist.append(((Lc.astype(np.float64) + eta_c * dL).astype(np.float32),
                     (Rc.astype(np.float64) + eta_c * dR).astype(np.float32)))
    return hist


def loss_dense(user, item, val, L, R):
    L = L.astype(np.float64)
    R = R.astype(np.float64)
    e = val.astype(np.float64) - np.einsum("tk,tk->t", L[user], R[item])
    return float(np.dot(e, e))


def run_dense_rowviews(user, item, val, L0, R0, *, N, M, K, P, C, eta, lam, views, step=0, B=1, seed=0,
                       owner=None):
    """The same matrix algebra with a version per row: views[c] = (vL, vR) with vL[i] the
    version of user row i read at clock c (by its owner's client) and vR[m][j] the version
    of item row j that client m reads (entries of rows not read are ignored).  Users of
    client m form E_m = W_m * (D - Lv Rv_m^T) with Lv, Rv_m gathered from those versions."""
    owner = np.arange(N) % P if owner is None else np.asarray(owner)
    client = owner % C
    blocks = np.array([block_of(i, j, seed, B) for i, j in zip(user, item)]) if B > 1 else None
    mats = [dense_mats(user, item, val, N, M, blocks, b) for b in range(B)]
    hist = [(np.asarray(L0, np.float32).reshape(N, K).copy(), np.asarray(R0, np.float32).reshape(M, K).copy())]
    for c, (vL, vR) in enumerate(views):
        W, D = mats[c % B]
        nu, ni = W.sum(1), W.sum(0)
        Lv = np.stack([hist[max(int(vL[i]), 0)][0][i] for i in range(N)]).astype(np.float64)
        dL = np.zeros((N, K))
        dR = np.zeros((M, K))
        for m in range(C):
            rows = client == m
            if not rows.any():
                continue
            Rv = np.stack([hist[max(int(vR[m][j]), 0)][1][j] for j in range(M)]).astype(np.float64)
            Wm = W * rows[:, None]
            E = Wm * (D - Lv @ Rv.T)
            gL = -(E @ Rv) + lam * Wm.sum(1)[:, None] * Lv
            gR = -(E.T @ Lv) + lam * Wm.sum(0)[:, None] * Rv
            dL[rows] -= gL[rows]
            dR -= gR
        if step == 0:
            dL /= np.where(nu > 0, nu, 1)[:, None]
            dR /= np.where(ni > 0, ni, 1)[:, None]
        Lc, Rc = hist[c]
        hist.append(((Lc.astype(np.float64) + eta * dL).astype(np.float32),
                     (Rc.astype(np.float64) + eta * dR).astype(np.float32)))
    return hist
