"""Oracle attention: masked GQA softmax attention, forward and backward.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Each segment is an independent attention unit whose keys are limited by the
dense visibility mask of the segment (Sec. 3.3: only the W most recent
screenshots stay visible, all text stays visible; causal order).  Grouped
query attention: query head h reads key/value head h // (hq // hkv).

Forward (per segment, per query head, float64):
    S = scale * Q K^T, invisible pairs set to -inf
    P = softmax(S) over keys,  O = P V,  LSE = log(sum_k exp(S))
Backward, from the definition of the softmax Jacobian:
    dV = P^T dO,  dP = dO V^T
    dS = P * (dP - rowsum(P * dP))
    dQ = scale * dS K,  dK = scale * dS^T Q
dK and dV of a key/value head sum the contributions of all its query heads.
"""
from __future__ import annotations

import numpy as np


def _kv_head(h, hq, hkv):
    return h // (hq // hkv)


def forward(q, k, v, mask, scale):
    """q [n, hq, d], k/v [n, hkv, d], mask [n, n] bool -> O [n, hq, d], LSE [hq, n]."""
    n, hq, d = q.shape
    hkv = k.shape[1]
    o = np.zeros((n, hq, d), np.float64)
    lse = np.zeros((hq, n), np.float64)
    for h in range(hq):
        g = _kv_head(h, hq, hkv)
        s = scale * (q[:, h, :] @ k[:, g, :].T)
        s = np.where(mask, s, -np.inf)
        m = s.max(axis=1, keepdims=True)
        p = np.exp(s - m)
        tot = p.sum(axis=1, keepdims=True)
        p = p / tot
        o[:, h, :] = p @ v[:, g, :]
        lse[h] = (m + np.log(tot))[:, 0]
    return o, lse


def backward(q, k, v, mask, scale, dout):
    """Gradients of sum(O * dout) w.r.t. q, k, v (same shapes as q, k, v)."""
    n, hq, d = q.shape
    hkv = k.shape[1]
    dq = np.zeros_like(q, dtype=np.float64)
    dk = np.zeros_like(k, dtype=np.float64)
    dv = np.zeros_like(v, dtype=np.float64)
    for h in range(hq):
        g = _kv_head(h, hq, hkv)
        s = scale * (q[:, h, :] @ k[:, g, :].T)
        s = np.where(mask, s, -np.inf)
        p = np.exp(s - s.max(axis=1, keepdims=True))
        p = p / p.sum(axis=1, keepdims=True)
        dv[:, g, :] += p.T @ dout[:, h, :]
        dp = dout[:, h, :] @ v[:, g, :].T
        ds = p * (dp - (p * dp).sum(axis=1, keepdims=True))
        dq[:, h, :] = scale * (ds @ k[:, g, :])
        dk[:, g, :] += scale * (ds.T @ q[:, h, :])
    return dq, dk, dv


def forward_rows(q_rows, k, v, mask_rows, scale):
    """Forward for a subset of query rows: q_rows [r, hq, d], mask_rows [r, n]."""
    return forward_generic(q_rows, k, v, mask_rows, scale)


def forward_generic(q, k, v, mask, scale):
    """Like :func:`forward` but with a rectangular mask [rows, keys]."""
    r, hq, d = q.shape
    hkv = k.shape[1]
    o = np.zeros((r, hq, d), np.float64)
    lse = np.zeros((hq, r), np.float64)
    for h in range(hq):
        g = _kv_head(h, hq, hkv)
        s = scale * (q[:, h, :] @ k[:, g, :].T)
        s = np.where(mask, s, -np.inf)
        m = s.max(axis=1, keepdims=True)
        p = np.exp(s - m)
        tot = p.sum(axis=1, keepdims=True)
        o[:, h, :] = (p / tot) @ v[:, g, :]
        lse[h] = (m + np.log(tot))[:, 0]
    return o, lse


def key_grads(q, k, v, mask, scale, dout, keys):
    """dK and dV of the keys ``keys`` only, from query rows ``q`` [r, hq, d]
    with their mask rows [r, n] over all n keys k, v [n, hkv, d] and their
    dout [r, hq, d].  Each row's softmax (its max, sum and so its LSE) and
    Delta = dout . O are taken over every key the row sees; a key's gradient
    is the sum over the given rows, so rows that do not see the keys may be
    left out, and disjoint row sets add up (the backward definitions above,
    restricted to a few columns of P and dS)."""
    r, hq, d = q.shape
    hkv = k.shape[1]
    keys = np.asarray(keys)
    dk = np.zeros((len(keys), hkv, d), np.float64)
    dv = np.zeros((len(keys), hkv, d), np.float64)
    for h in range(hq):
        g = _kv_head(h, hq, hkv)
        s = scale * (q[:, h, :] @ k[:, g, :].T)
        s = np.where(mask, s, -np.inf)
        p = np.exp(s - s.max(axis=1, keepdims=True))
        p = p / p.sum(axis=1, keepdims=True)
        delta = (dout[:, h, :] * (p @ v[:, g, :])).sum(axis=1)
        pk = p[:, keys]
        dpk = dout[:, h, :] @ v[keys, g, :].T
        dsk = pk * (dpk - delta[:, None])
        dv[:, g, :] += pk.T @ dout[:, h, :]
        dk[:, g, :] += scale * (dsk.T @ q[:, h, :])
    return dk, dv
