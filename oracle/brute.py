"""Dense fp64 NumPy formulations used to pin the oracle (test infrastructure).

TEST INFRASTRUCTURE ONLY.  These restate the paper's definitions in a form
that never builds the recurrent state, so that a mistake in the state path of
``oracle.c`` (a transposed S, a dropped term in the update, a wrong slot or
head index) shows up as a disagreement:

* ``hybrid_block_brute``: the linear branch as the explicit prefix sum
  sum_t phi(q).phi(k_t) v_t (Eq. 1 with the state unrolled, Section 2.2).
* ``block_causal_brute``: the Figure 2 pattern as one dense T x T weight
  matrix -- w*exp(q.k/sqrt(d)) on diagonal blocks, phi(q).phi(k) below them,
  zero above -- normalised row by row (Section 3.1's shared normaliser).
* ``state_brute``: S = phi(K)^T V and z = sum_t phi(k_t) as one matrix
  product (Section 3.1 state definition).

Only the feature map is shared between these three, and it is pinned on its
own by closed-form fixtures.
"""
from __future__ import annotations

import numpy as np


def phi(X, Wt):
    """Hedgehog feature map of Section 3.1 for rows of X [..., d]; Wt [F][d]."""
    U = np.asarray(X, np.float64) @ np.asarray(Wt, np.float64).T
    pos = np.exp(U - U.max(axis=-1, keepdims=True))
    neg = np.exp(-U - (-U).max(axis=-1, keepdims=True))
    pos /= pos.sum(axis=-1, keepdims=True)
    neg /= neg.sum(axis=-1, keepdims=True)
    return np.concatenate([pos, neg], axis=-1)


def sigmoid(a):
    return 1.0 / (1.0 + np.exp(-np.asarray(a, np.float64)))


def _kv_head(h, Hq, Hkv):
    return h // (Hq // Hkv)


def hybrid_block_brute(q, k, v, kp, vp, plen, Wt, alpha):
    """Hybrid output with the prefix kept as explicit tokens.

    q [B][L][Hq][d]; k, v [B][L][Hkv][d]; kp, vp [B][Pmax][Hkv][d]; plen [B].
    Returns out [B][L][Hq][d].
    """
    q = np.asarray(q, np.float64)
    B, L, Hq, d = q.shape
    Hkv = k.shape[2]
    out = np.zeros_like(q)
    for b in range(B):
        P = int(plen[b])
        for h in range(Hq):
            g = _kv_head(h, Hq, Hkv)
            w = sigmoid(alpha[h])
            Q = q[b, :, h, :]
            Kb, Vb = np.asarray(k[b, :, g, :], np.float64), np.asarray(v[b, :, g, :], np.float64)
            A_blk = np.exp(Q @ Kb.T / np.sqrt(d))              # a_j, [L][L]
            Kp, Vp = np.asarray(kp[b, :P, g, :], np.float64), np.asarray(vp[b, :P, g, :], np.float64)
            A_lin = phi(Q, Wt[h]) @ phi(Kp, Wt[h]).T           # phi(q).phi(k_t), [L][P]
            num = w * A_blk @ Vb + A_lin @ Vp
            den = w * A_blk.sum(1) + A_lin.sum(1)
            out[b, :, h, :] = num / den[:, None]
    return out


def block_causal_weights(Q, K, Wt_h, w, L):
    """Dense Figure 2 weight matrix for one head over a T-token sequence."""
    T, d = Q.shape
    blk = np.arange(T) // L
    same = blk[:, None] == blk[None, :]
    before = blk[None, :] < blk[:, None]
    A_sm = w * np.exp(Q @ K.T / np.sqrt(d))
    A_lin = phi(Q, Wt_h) @ phi(K, Wt_h).T
    return np.where(same, A_sm, 0.0) + np.where(before, A_lin, 0.0)


def block_causal_brute(q, k, v, Wt, alpha, L):
    """Prefill outputs from the dense Figure 2 pattern; q [B][T][Hq][d]."""
    q = np.asarray(q, np.float64)
    B, T, Hq, d = q.shape
    Hkv = k.shape[2]
    out = np.zeros_like(q)
    for b in range(B):
        for h in range(Hq):
            g = _kv_head(h, Hq, Hkv)
            A = block_causal_weights(q[b, :, h, :], np.asarray(k[b, :, g, :], np.float64),
                                     Wt[h], sigmoid(alpha[h]), L)
            out[b, :, h, :] = (A @ np.asarray(v[b, :, g, :], np.float64)) / A.sum(1)[:, None]
    return out


def state_brute(k, v, Wt, Hq):
    """S [B][Hq][2F][d] = phi(K)^T V and z [B][Hq][2F] = sum_t phi(k_t)."""
    B, T, Hkv, d = k.shape
    F = Wt.shape[1]
    S = np.zeros((B, Hq, 2 * F, d))
    z = np.zeros((B, Hq, 2 * F))
    for b in range(B):
        for h in range(Hq):
            g = _kv_head(h, Hq, Hkv)
            P = phi(np.asarray(k[b, :, g, :], np.float64), Wt[h])
            S[b, h] = P.T @ np.asarray(v[b, :, g, :], np.float64)
            z[b, h] = P.sum(0)
    return S, z
