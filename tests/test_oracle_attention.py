"""Pins of the oracle's masked GQA attention (forward and backward).

Checks against library routines (torch's scaled_dot_product_attention and
autograd on the CPU in float64), a per-row pure-Python brute force, central
finite differences, the trajectory-level special case (plain causal
attention) and the segment == step-wise invariant for action rows (Sec. 3.3).
"""
import math

import numpy as np
import pytest
import torch

from oracle import attention as OA
from oracle import layout as OL
from paper_2607_11185_amd import workload as WL


def _seg_inputs(rng, n, hq, hkv, d):
    q = rng.standard_normal((n, hq, d))
    k = rng.standard_normal((n, hkv, d))
    v = rng.standard_normal((n, hkv, d))
    return q, k, v


def _sdpa(q, k, v, mask, scale):
    """torch SDPA (float64, CPU) with the kv heads repeated for GQA."""
    n, hq, d = q.shape
    rep = hq // k.shape[1]
    tq = torch.tensor(q).permute(1, 0, 2)
    tk = torch.tensor(k).repeat_interleave(rep, dim=1).permute(1, 0, 2)
    tv = torch.tensor(v).repeat_interleave(rep, dim=1).permute(1, 0, 2)
    o = torch.nn.functional.scaled_dot_product_attention(
        tq, tk, tv, attn_mask=torch.tensor(mask), scale=scale)
    return o.permute(1, 0, 2).numpy()


def _segment(W=2, L=3, seed=0):
    rng = np.random.default_rng(seed)
    sp = WL.explicit_spans([5], [3], rng.integers(1, 6, 5), rng.integers(2, 6, 5), [1] * 5)
    lay = OL.build(sp, W, L, 4)
    return lay.segments[0], OL.visibility(lay.segments[0], W)


@pytest.mark.parametrize("hq,hkv", [(4, 1), (4, 2), (6, 3)])
def test_forward_matches_sdpa(hq, hkv):
    sg, mask = _segment()
    rng = np.random.default_rng(1)
    q, k, v = _seg_inputs(rng, sg.length, hq, hkv, 8)
    scale = 1 / math.sqrt(8)
    o, lse = OA.forward(q, k, v, mask, scale)
    assert np.allclose(o, _sdpa(q, k, v, mask, scale), atol=1e-12, rtol=1e-12)


def test_lse_brute_force():
    sg, mask = _segment(W=1, L=2, seed=3)
    rng = np.random.default_rng(2)
    q, k, v = _seg_inputs(rng, sg.length, 2, 1, 4)
    scale = 0.5
    o, lse = OA.forward(q, k, v, mask, scale)
    for h in range(2):
        for i in range(sg.length):
            terms = [math.exp(scale * sum(q[i, h, t] * k[j, 0, t] for t in range(4)))
                     for j in range(sg.length) if mask[i, j]]
            assert abs(math.log(sum(terms)) - lse[h, i]) < 1e-12
            # output row is the probability-weighted mean of the visible values
            num = np.zeros(4)
            for j in range(sg.length):
                if mask[i, j]:
                    num += math.exp(scale * float(q[i, h] @ k[j, 0])) * v[j, 0]
            assert np.allclose(num / sum(terms), o[i, h], atol=1e-12)


def test_trajectory_level_is_causal_sdpa():
    sp = WL.explicit_spans([4], [3], [3] * 4, [2] * 4, [1] * 4)
    lay = OL.build(sp, 8, 8, 4)
    sg = lay.segments[0]
    rng = np.random.default_rng(5)
    q, k, v = _seg_inputs(rng, sg.length, 2, 2, 8)
    o, _ = OA.forward(q, k, v, OL.visibility(sg, 8), 0.3)
    want = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(q).permute(1, 0, 2), torch.tensor(k).permute(1, 0, 2),
        torch.tensor(v).permute(1, 0, 2), is_causal=True, scale=0.3).permute(1, 0, 2).numpy()
    assert np.allclose(o, want, atol=1e-12)


def test_backward_matches_autograd():
    sg, mask = _segment(W=2, L=4, seed=7)
    rng = np.random.default_rng(3)
    hq, hkv, d = 4, 2, 8
    q, k, v = _seg_inputs(rng, sg.length, hq, hkv, d)
    dout = rng.standard_normal((sg.length, hq, d))
    scale = 1 / math.sqrt(d)
    dq, dk, dv = OA.backward(q, k, v, mask, scale, dout)
    tq = torch.tensor(q, requires_grad=True)
    tk = torch.tensor(k, requires_grad=True)
    tv = torch.tensor(v, requires_grad=True)
    rep = hq // hkv
    o = torch.nn.functional.scaled_dot_product_attention(
        tq.permute(1, 0, 2), tk.repeat_interleave(rep, 1).permute(1, 0, 2),
        tv.repeat_interleave(rep, 1).permute(1, 0, 2), attn_mask=torch.tensor(mask),
        scale=scale).permute(1, 0, 2)
    (o * torch.tensor(dout)).sum().backward()
    assert np.allclose(dq, tq.grad.numpy(), atol=1e-10)
    assert np.allclose(dk, tk.grad.numpy(), atol=1e-10)
    assert np.allclose(dv, tv.grad.numpy(), atol=1e-10)


def test_key_grads_match_autograd_on_row_subsets():
    """dK/dV of a few keys from only the rows that see them, split into two
    disjoint row sets and summed, equal torch autograd's full gradients at
    those keys (and the screenshot keys' rows exclude expired turns)."""
    sg, mask = _segment(W=1, L=4, seed=11)
    rng = np.random.default_rng(4)
    hq, hkv, d = 6, 2, 8
    q, k, v = _seg_inputs(rng, sg.length, hq, hkv, d)
    dout = rng.standard_normal((sg.length, hq, d))
    scale = 1 / math.sqrt(d)
    tq = torch.tensor(q, requires_grad=True)
    tk = torch.tensor(k, requires_grad=True)
    tv = torch.tensor(v, requires_grad=True)
    rep = hq // hkv
    o = torch.nn.functional.scaled_dot_product_attention(
        tq.permute(1, 0, 2), tk.repeat_interleave(rep, 1).permute(1, 0, 2),
        tv.repeat_interleave(rep, 1).permute(1, 0, 2), attn_mask=torch.tensor(mask),
        scale=scale).permute(1, 0, 2)
    (o * torch.tensor(dout)).sum().backward()
    keys = np.nonzero(sg.kind == OL.KIND_IMAGE)[0][:3]
    rows = np.nonzero(mask[:, keys].any(1))[0]
    assert 0 < len(rows) < sg.length - keys.min()    # the window hides them from later turns
    half = len(rows) // 2
    parts = [OA.key_grads(q[r], k, v, mask[r], scale, dout[r], keys)
             for r in (rows[:half], rows[half:])]
    dk = parts[0][0] + parts[1][0]
    dv = parts[0][1] + parts[1][1]
    assert np.allclose(dk, tk.grad.numpy()[keys], atol=1e-10)
    assert np.allclose(dv, tv.grad.numpy()[keys], atol=1e-10)


def test_backward_finite_differences():
    sg, mask = _segment(W=1, L=3, seed=9)
    rng = np.random.default_rng(4)
    hq, hkv, d = 2, 1, 4
    q, k, v = _seg_inputs(rng, sg.length, hq, hkv, d)
    dout = rng.standard_normal((sg.length, hq, d))
    scale = 0.7
    grads = OA.backward(q, k, v, mask, scale, dout)

    def f(q_, k_, v_):
        return float((OA.forward(q_, k_, v_, mask, scale)[0] * dout).sum())

    eps = 1e-6
    for which in range(3):
        base = [q, k, v]
        direction = rng.standard_normal(base[which].shape)
        plus = list(base)
        minus = list(base)
        plus[which] = base[which] + eps * direction
        minus[which] = base[which] - eps * direction
        fd = (f(*plus) - f(*minus)) / (2 * eps)
        an = float((grads[which] * direction).sum())
        assert abs(fd - an) < 1e-6 * max(1.0, abs(an)), (which, fd, an)


def test_action_rows_segment_equals_stepwise():
    """Attention output of every action-predicting row is the same in the
    segmented layout and in the step-wise decomposition (Sec. 3.3)."""
    sp = WL.explicit_spans([7, 5], [4, 3], [3, 2, 4, 1, 3, 2, 2, 3, 1, 2, 4, 3],
                           [3, 4, 2, 5, 3, 4, 2, 3, 4, 2, 3, 5], [1, 2, 1, 2, 1, 1, 2, 1, 1, 2, 1, 2])
    W, L = 2, 3
    rng = np.random.default_rng(8)
    n = int(sp.canon_offsets()[-1])
    q, k, v = _seg_inputs(rng, n, 4, 2, 8)
    out = {}
    for LL in (L, 1):
        lay = OL.build(sp, W, LL, 4)
        res = {}
        for sg in lay.segments:
            o, lse = OA.forward(q[sg.canon], k[sg.canon], v[sg.canon], OL.visibility(sg, W), 0.35)
            for p, t in zip(lay.loss_pred_row, lay.loss_tgt_src):
                if sg.start <= p < sg.start + sg.length:
                    res[int(t)] = (o[p - sg.start], lse[:, p - sg.start])
        out[LL] = res
    assert out[L].keys() == out[1].keys()
    for t in out[1]:
        assert np.allclose(out[L][t][0], out[1][t][0], atol=1e-13)
        assert np.allclose(out[L][t][1], out[1][t][1], atol=1e-13)
