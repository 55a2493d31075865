"""Oracle decoder layer around the segmented attention, forward and backward.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper trains the language model of a vision-language agent on VCS
segments and keeps the vision encoder fixed during RL (App. E, RL stage), so
the screenshot tokens enter the language model as given hidden states.  It does
not spell out the layer, so this follows a generic Qwen-family decoder layer
(pre-norm RMSNorm, grouped-query attention with rotary position embedding,
SwiGLU MLP; no biases, no per-head q/k norm), float64 throughout:

    a  = rms(x) * g1                    rms(x) = x / sqrt(mean(x^2) + eps)
    q, k, v = a Wq^T, a Wk^T, a Wv^T    (heads of d columns)
    q', k' = rope(q, pos), rope(k, pos)
    o  = segmented attention(q', k', v) (oracle.attention, per segment mask)
    y1 = x + o Wo^T
    b  = rms(y1) * g2
    g, u = b Wg^T, b Wu^T
    y  = y1 + (silu(g) * u) Wd^T

Rotary embedding (rotate-half pairing): for i < d/2 with angle
theta_i = pos * base^(-2i/d), the pair (x_i, x_{i + d/2}) is rotated by
theta_i.  Readings: pos is the token's row inside its segment (a segment is
a re-tokenised stream that starts at position 0); base, eps are arguments.

The backward is derived by hand from these definitions (chain rule); the
tests pin it with central finite differences, not with an autodiff library.
"""
from __future__ import annotations

import numpy as np

from . import attention as OA


def rms_forward(x, g, eps):
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return x * r * g, r[..., 0]


def rms_backward(x, g, r, dy):
    """dx, dg of y = x * r * g with r = (mean(x^2) + eps)^(-1/2)."""
    n = x.shape[-1]
    r = r[..., None]
    gy = dy * g
    dx = r * gy - (r ** 3) * x * np.sum(gy * x, axis=-1, keepdims=True) / n
    dg = np.sum(dy * x * r, axis=tuple(range(x.ndim - 1)))
    return dx, dg


def rope_angles(pos, d, base):
    i = np.arange(d // 2, dtype=np.float64)
    inv = base ** (-2.0 * i / d)
    return np.asarray(pos, np.float64)[:, None] * inv[None, :]  # [n, d/2]


def rope(x, pos, base, inverse=False):
    """x [n, heads, d] -> rotated copy; inverse rotates by -theta (the transpose)."""
    d = x.shape[-1]
    t = rope_angles(pos, d, base)
    c, s = np.cos(t)[:, None, :], np.sin(t)[:, None, :]
    if inverse:
        s = -s
    x1, x2 = x[..., : d // 2], x[..., d // 2:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(g):
    return g / (1.0 + np.exp(-g))


def silu_grad(g):
    sg = 1.0 / (1.0 + np.exp(-g))
    return sg * (1.0 + g * (1.0 - sg))


def segment_positions(segments, packed):
    """Row index inside its segment for every packed row (-1 for padding)."""
    pos = np.full(packed, -1, np.int64)
    for sg in segments:
        pos[sg.start:sg.start + sg.length] = np.arange(sg.length)
    return pos


class Weights:
    """Layer weights (float64 arrays): g1, wq, wk, wv, wo, g2, wg, wu, wd."""

    def __init__(self, **kw):
        self.__dict__.update(kw)


def forward(x, w, segments, masks, hq, hkv, d, eps, base):
    """x [P, H] (padding rows are carried through unchanged apart from the
    residual path), masks: one visibility mask per segment.  Returns y and
    the saved intermediates."""
    P = x.shape[0]
    pos = segment_positions(segments, P)
    a, r1 = rms_forward(x, w.g1, eps)
    q = (a @ w.wq.T).reshape(P, hq, d)
    k = (a @ w.wk.T).reshape(P, hkv, d)
    v = (a @ w.wv.T).reshape(P, hkv, d)
    pz = np.maximum(pos, 0)
    qr, kr = rope(q, pz, base), rope(k, pz, base)
    o = np.zeros((P, hq, d))
    lse = np.zeros((hq, P))
    scale = 1.0 / np.sqrt(d)
    for sg, m in zip(segments, masks):
        rows = slice(sg.start, sg.start + sg.length)
        o[rows], lse[:, rows] = OA.forward(qr[rows], kr[rows], v[rows], m, scale)
    y1 = x + o.reshape(P, hq * d) @ w.wo.T
    b, r2 = rms_forward(y1, w.g2, eps)
    gt, ut = b @ w.wg.T, b @ w.wu.T
    mm = silu(gt) * ut
    y = y1 + mm @ w.wd.T
    saved = dict(pos=pos, a=a, r1=r1, qr=qr, kr=kr, v=v, o=o, lse=lse, y1=y1, b=b, r2=r2,
                 gt=gt, ut=ut, mm=mm)
    return y, saved


def backward(x, w, segments, masks, hq, hkv, d, eps, base, saved, dy):
    """Gradients of sum(y * dy) over the segment rows: dx and the weight
    gradients (a dict).  Padding rows carry no gradient (their dy counts as 0)."""
    P = x.shape[0]
    s = saved
    dy = dy * (s["pos"] >= 0)[:, None]
    scale = 1.0 / np.sqrt(d)
    grads = {}
    # MLP
    grads["wd"] = dy.T @ s["mm"]
    dmm = dy @ w.wd
    dgt = dmm * s["ut"] * silu_grad(s["gt"])
    dut = dmm * silu(s["gt"])
    grads["wg"] = dgt.T @ s["b"]
    grads["wu"] = dut.T @ s["b"]
    db = dgt @ w.wg + dut @ w.wu
    dy1_n, grads["g2"] = rms_backward(s["y1"], w.g2, s["r2"], db)
    dy1 = dy + dy1_n
    # attention output projection
    grads["wo"] = dy1.T @ s["o"].reshape(P, hq * d)
    do = (dy1 @ w.wo).reshape(P, hq, d)
    dq = np.zeros((P, hq, d))
    dk = np.zeros((P, hkv, d))
    dv = np.zeros((P, hkv, d))
    for sg, m in zip(segments, masks):
        rows = slice(sg.start, sg.start + sg.length)
        dq[rows], dk[rows], dv[rows] = OA.backward(s["qr"][rows], s["kr"][rows], s["v"][rows],
                                                    m, scale, do[rows])
    pz = np.maximum(s["pos"], 0)
    dq = rope(dq, pz, base, inverse=True).reshape(P, hq * d)
    dk = rope(dk, pz, base, inverse=True).reshape(P, hkv * d)
    dv = dv.reshape(P, hkv * d)
    grads["wq"] = dq.T @ s["a"]
    grads["wk"] = dk.T @ s["a"]
    grads["wv"] = dv.T @ s["a"]
    da = dq @ w.wq + dk @ w.wk + dv @ w.wv
    dx_n, grads["g1"] = rms_backward(x, w.g1, s["r1"], da)
    return dy1 + dx_n, grads


def forward_rows(x_seg, w, mask, rows, hq, hkv, d, eps, base):
    """Layer output y for some rows of ONE segment, from that segment's hidden
    states x_seg [L, H] (row i at position i) and its visibility mask [L, L]:
    keys and values come from every row of the segment, queries and the rest
    of the layer only from `rows`.  Same definitions as :func:`forward`."""
    L = x_seg.shape[0]
    rows = np.asarray(rows)
    a, _ = rms_forward(x_seg, w.g1, eps)
    pos = np.arange(L)
    k = rope((a @ w.wk.T).reshape(L, hkv, d), pos, base)
    v = (a @ w.wv.T).reshape(L, hkv, d)
    q = rope((a[rows] @ w.wq.T).reshape(len(rows), hq, d), pos[rows], base)
    o, _ = OA.forward_rows(q, k, v, mask[rows], 1.0 / np.sqrt(d))
    y1 = x_seg[rows] + o.reshape(len(rows), hq * d) @ w.wo.T
    b, _ = rms_forward(y1, w.g2, eps)
    return y1 + (silu(b @ w.wg.T) * (b @ w.wu.T)) @ w.wd.T
