"""Pins of the oracle decoder layer (oracle/layer.py) against closed forms,
invariants and central finite differences, on the CPU."""
import numpy as np
import pytest

from oracle import layer as OLY
from oracle import layout as OL
from paper_2607_11185_amd import workload as WL


def test_rope_is_a_rotation_with_relative_positions():
    rng = np.random.default_rng(0)
    n, h, d = 7, 3, 16
    q = rng.standard_normal((n, h, d))
    k = rng.standard_normal((n, h, d))
    pos = rng.integers(0, 50, size=n)
    base = 100.0
    qr = OLY.rope(q, pos, base)
    # each (i, i + d/2) pair keeps its length
    np.testing.assert_allclose(qr[..., :8] ** 2 + qr[..., 8:] ** 2, q[..., :8] ** 2 + q[..., 8:] ** 2,
                               rtol=1e-12)
    # position 0 is the identity; the inverse undoes the rotation
    np.testing.assert_allclose(OLY.rope(q, np.zeros(n, int), base), q, rtol=0, atol=0)
    np.testing.assert_allclose(OLY.rope(qr, pos, base, inverse=True), q, rtol=1e-12, atol=1e-12)
    # scores depend only on the position difference
    pq, pk = pos, rng.integers(0, 50, size=n)
    s1 = np.einsum("nhd,nhd->nh", OLY.rope(q, pq, base), OLY.rope(k, pk, base))
    s2 = np.einsum("nhd,nhd->nh", OLY.rope(q, pq + 13, base), OLY.rope(k, pk + 13, base))
    np.testing.assert_allclose(s1, s2, rtol=1e-10, atol=1e-10)


def test_rope_closed_form_first_pair():
    """For i = 0 the angle is the position itself (base^0 = 1)."""
    x = np.zeros((3, 1, 4))
    x[:, 0, 0] = 1.0
    pos = np.array([0, 1, 2])
    y = OLY.rope(x, pos, 10000.0)
    np.testing.assert_allclose(y[:, 0, 0], np.cos(pos), atol=1e-15)
    np.testing.assert_allclose(y[:, 0, 2], np.sin(pos), atol=1e-15)
    # the second pair (i = 1) turns by pos * base^(-1/2)
    x = np.zeros((1, 1, 4))
    x[0, 0, 1] = 1.0
    y = OLY.rope(x, np.array([3]), 100.0)
    np.testing.assert_allclose([y[0, 0, 1], y[0, 0, 3]], [np.cos(0.3), np.sin(0.3)], atol=1e-15)


def test_rmsnorm_closed_forms():
    g = np.array([1.0, 2.0, 3.0, 4.0])
    x = np.full((2, 4), -5.0)
    y, r = OLY.rms_forward(x, g, 0.0)
    np.testing.assert_allclose(y, -g[None, :].repeat(2, 0), rtol=1e-15)
    np.testing.assert_allclose(r, [0.2, 0.2], rtol=1e-15)
    # invariant to a positive rescaling of the row (eps = 0)
    rng = np.random.default_rng(1)
    x = rng.standard_normal((3, 10))
    np.testing.assert_allclose(OLY.rms_forward(7.5 * x, np.ones(10), 0.0)[0],
                               OLY.rms_forward(x, np.ones(10), 0.0)[0], rtol=1e-13)


def test_silu_closed_forms():
    assert OLY.silu(np.array(0.0)) == 0.0
    assert abs(OLY.silu_grad(np.array(0.0)) - 0.5) < 1e-15
    g = np.linspace(-6, 6, 25)
    h = 1e-6
    fd = (OLY.silu(g + h) - OLY.silu(g - h)) / (2 * h)
    np.testing.assert_allclose(OLY.silu_grad(g), fd, rtol=1e-7, atol=1e-9)


def test_rmsnorm_backward_finite_differences():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((3, 6))
    g = rng.standard_normal(6)
    dy = rng.standard_normal((3, 6))
    eps = 1e-3
    y, r = OLY.rms_forward(x, g, eps)
    dx, dg = OLY.rms_backward(x, g, r, dy)
    h = 1e-6
    for i in range(3):
        for j in range(6):
            e = np.zeros_like(x)
            e[i, j] = h
            fd = (np.sum(OLY.rms_forward(x + e, g, eps)[0] * dy) -
                  np.sum(OLY.rms_forward(x - e, g, eps)[0] * dy)) / (2 * h)
            assert abs(dx[i, j] - fd) < 1e-7 * max(1, abs(fd))
    for j in range(6):
        e = np.zeros_like(g)
        e[j] = h
        fd = (np.sum(OLY.rms_forward(x, g + e, eps)[0] * dy) -
              np.sum(OLY.rms_forward(x, g - e, eps)[0] * dy)) / (2 * h)
        assert abs(dg[j] - fd) < 1e-7 * max(1, abs(fd))


def _tiny(seed=0, hq=4, hkv=2, d=8, H=12, I=10, buffers=0):
    """A two-trajectory batch of a few turns and random float64 weights."""
    sp = WL.explicit_spans([3, 2], [3, 2], [4, 3, 2, 4, 3], [3, 4, 2, 3, 2], [1, 2, 1, 1, 2])
    lay = OL.build(sp, 2, 2, 4, buffer_tokens=buffers, with_tiles=False)
    rng = np.random.default_rng(seed)
    P = lay.packed_tokens
    x = rng.standard_normal((P, H))
    w = OLY.Weights(g1=1 + 0.1 * rng.standard_normal(H), wq=0.3 * rng.standard_normal((hq * d, H)),
                    wk=0.3 * rng.standard_normal((hkv * d, H)),
                    wv=0.3 * rng.standard_normal((hkv * d, H)),
                    wo=0.3 * rng.standard_normal((H, hq * d)),
                    g2=1 + 0.1 * rng.standard_normal(H), wg=0.3 * rng.standard_normal((I, H)),
                    wu=0.3 * rng.standard_normal((I, H)), wd=0.3 * rng.standard_normal((H, I)))
    masks = [OL.visibility(sg, 2) for sg in lay.segments]
    return lay, x, w, masks, dict(hq=hq, hkv=hkv, d=d, eps=1e-5, base=50.0)


@pytest.mark.parametrize("buffers", [0, 32])
def test_layer_backward_finite_differences(buffers):
    """dx and every weight gradient against central differences of
    sum(y * dy) over the segment rows, in random directions."""
    lay, x, w, masks, a = _tiny(buffers=buffers)
    rng = np.random.default_rng(3)
    seg_rows = OLY.segment_positions(lay.segments, x.shape[0]) >= 0
    dy = rng.standard_normal(x.shape)
    y, saved = OLY.forward(x, w, lay.segments, masks, **a)
    dx, grads = OLY.backward(x, w, lay.segments, masks, **a, saved=saved, dy=dy)

    def f(xx, ww):
        yy, _ = OLY.forward(xx, ww, lay.segments, masks, **a)
        return float(np.sum((yy * dy)[seg_rows]))

    h = 1e-5
    for trial in range(3):
        e = rng.standard_normal(x.shape)
        fd = (f(x + h * e, w) - f(x - h * e, w)) / (2 * h)
        assert abs(np.sum(dx * e) - fd) < 1e-6 * max(1.0, abs(fd))
    for name in ("g1", "wq", "wk", "wv", "wo", "g2", "wg", "wu", "wd"):
        base = getattr(w, name)
        e = rng.standard_normal(base.shape)
        wp = OLY.Weights(**{**w.__dict__, name: base + h * e})
        wm = OLY.Weights(**{**w.__dict__, name: base - h * e})
        fd = (f(x, wp) - f(x, wm)) / (2 * h)
        assert abs(np.sum(grads[name] * e) - fd) < 1e-6 * max(1.0, abs(fd)), name
    # padding rows get no gradient
    assert np.all(dx[~seg_rows] == 0)


def test_layer_with_zero_projections_is_the_identity():
    lay, x, w, masks, a = _tiny(seed=4)
    w.wo[:] = 0
    w.wd[:] = 0
    y, saved = OLY.forward(x, w, lay.segments, masks, **a)
    np.testing.assert_array_equal(y, x)
    dy = np.random.default_rng(5).standard_normal(x.shape)
    dx, grads = OLY.backward(x, w, lay.segments, masks, **a, saved=saved, dy=dy)
    np.testing.assert_allclose(dx, dy, rtol=0, atol=0)
    for name in ("wq", "wk", "wv", "g1", "wg", "wu", "g2"):
        assert np.all(grads[name] == 0), name


def test_layer_attention_part_uses_segment_positions():
    """Two identical segments get identical attention outputs: positions
    restart at 0 in every segment, and segments do not see each other."""
    sp = WL.explicit_spans([2, 2], [3, 3], [2, 2, 2, 2], [3, 3, 3, 3], [1, 1, 1, 1])
    lay = OL.build(sp, 2, 2, 4, with_tiles=False)
    assert len(lay.segments) == 2 and lay.segments[0].length == lay.segments[1].length
    n = lay.segments[0].length
    rng = np.random.default_rng(6)
    H, hq, hkv, d = 8, 2, 1, 4
    x0 = rng.standard_normal((n, H))
    x = np.concatenate([x0, x0])
    w = OLY.Weights(g1=np.ones(H), wq=rng.standard_normal((hq * d, H)),
                    wk=rng.standard_normal((hkv * d, H)), wv=rng.standard_normal((hkv * d, H)),
                    wo=rng.standard_normal((H, hq * d)), g2=np.ones(H),
                    wg=rng.standard_normal((6, H)), wu=rng.standard_normal((6, H)),
                    wd=rng.standard_normal((H, 6)))
    masks = [OL.visibility(sg, 2) for sg in lay.segments]
    y, _ = OLY.forward(x, w, lay.segments, masks, hq, hkv, d, 1e-6, 1e4)
    np.testing.assert_allclose(y[:n], y[n:], rtol=1e-13, atol=1e-13)


def test_forward_rows_matches_forward():
    """The row-sampled forward (keys of the whole segment, queries of some
    rows) equals the full forward on those rows."""
    lay, x, w, masks, a = _tiny(seed=7, buffers=32)
    y, _ = OLY.forward(x, w, lay.segments, masks, **a)
    for sg, m in zip(lay.segments, masks):
        rows = np.array([0, sg.length // 2, sg.length - 1])
        ys = OLY.forward_rows(x[sg.start:sg.start + sg.length], w, m, rows, **a)
        np.testing.assert_allclose(ys, y[sg.start + rows], rtol=1e-12, atol=1e-12)


def test_layer_forward_matches_torch_composition():
    """The whole forward against the same layer composed from library
    primitives on the CPU in float64: torch's RMS normalisation formula,
    rotary embedding as a complex multiplication of (x_i + i x_{i+d/2}) by
    e^{i theta}, scaled_dot_product_attention with the boolean visibility
    mask and kv heads repeated per group, and F.silu for the MLP."""
    import torch
    import torch.nn.functional as F
    lay, x, w, masks, a = _tiny(seed=7, hq=6, hkv=2, d=8)
    y_o, _ = OLY.forward(x, w, lay.segments, masks, **a)
    hq, hkv, d, eps, base = a["hq"], a["hkv"], a["d"], a["eps"], a["base"]
    T = {n: torch.from_numpy(np.asarray(v)) for n, v in w.__dict__.items()}
    for sg, m in zip(lay.segments, masks):
        xs = torch.from_numpy(x[sg.start:sg.start + sg.length])
        n = xs.shape[0]
        an = xs * torch.rsqrt(xs.pow(2).mean(-1, keepdim=True) + eps) * T["g1"]
        q = (an @ T["wq"].T).view(n, hq, d)
        k = (an @ T["wk"].T).view(n, hkv, d)
        v = (an @ T["wv"].T).view(n, hkv, d)
        inv = base ** (-torch.arange(0, d, 2, dtype=torch.float64) / d)
        rot = torch.polar(torch.ones(n, d // 2, dtype=torch.float64),
                          torch.arange(n, dtype=torch.float64)[:, None] * inv[None, :])

        def rope(t):
            z = torch.complex(t[..., : d // 2], t[..., d // 2:]) * rot[:, None, :]
            return torch.cat([z.real, z.imag], dim=-1)

        qh = rope(q).transpose(0, 1)
        kh = rope(k).transpose(0, 1).repeat_interleave(hq // hkv, dim=0)
        vh = v.transpose(0, 1).repeat_interleave(hq // hkv, dim=0)
        o = F.scaled_dot_product_attention(qh, kh, vh, attn_mask=torch.from_numpy(m))
        y1 = xs + o.transpose(0, 1).reshape(n, hq * d) @ T["wo"].T
        b = y1 * torch.rsqrt(y1.pow(2).mean(-1, keepdim=True) + eps) * T["g2"]
        y = y1 + (F.silu(b @ T["wg"].T) * (b @ T["wu"].T)) @ T["wd"].T
        np.testing.assert_allclose(y_o[sg.start:sg.start + sg.length], y.numpy(),
                                   rtol=1e-10, atol=1e-10)
