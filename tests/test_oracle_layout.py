"""Pins of the oracle's layout (segmentation, packing, visibility, tiles, loss rows).

Every check here is independent of the oracle's own code path: hand-worked
fixtures, closed-form counts, special cases that reduce to plain causal
attention or to the step-wise decomposition, and invariants the paper states
(Sec. 3.3; App. D; Eq. loss).
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import layout as OL
from paper_2607_11185_amd import workload as WL

GOLD = os.path.join(os.path.dirname(__file__), "golden")
TILE_CH = {"S": 0, "P": OL.CLS_PARTIAL, "F": OL.CLS_FULL}


def _fixture(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def _spans(d):
    s = d["spans"]
    return WL.explicit_spans(s["steps"], s["prompt"], s["img"], s["text"], s["action"])


def _tile_grid(lay, si):
    """Dense class grid of segment si rebuilt from the CSR."""
    info = lay.seg_info[si]
    base, n = int(info[5]), int(info[4])
    nt = -(-n // lay.tile)
    grid = np.zeros((nt, nt), np.int64)
    for i in range(nt):
        g = base + i
        for e in range(lay.qt_ptr[g], lay.qt_ptr[g + 1]):
            grid[i, lay.qt_col[e] - base] = lay.qt_cls[e]
    return grid


@pytest.mark.parametrize("name", ["appA_example_a.json", "appA_example_b.json"])
def test_hand_worked_examples(name):
    d = _fixture(name)
    sp = _spans(d)
    lay = OL.build(sp, d["window"], d["seg_steps"], d["tile"])
    assert [list(map(int, r[:5])) for r in lay.seg_info] == d["segments"]
    assert lay.tok_src.tolist() == d["tok_src"]
    got_rows = [[int(p), int(t)] for p, t in zip(lay.loss_pred_row, lay.loss_tgt_src)]
    assert got_rows == d["loss_rows"]
    for si, sg in enumerate(lay.segments):
        m = OL.visibility(sg, d["window"])
        want = np.array([[c == "1" for c in r] for r in d["masks"][si]])
        assert (m == want).all(), f"mask of segment {si}"
        grid = _tile_grid(lay, si)
        want_t = np.array([[TILE_CH[c] for c in r] for r in d["tiles"][si]])
        assert (grid == want_t).all(), f"tiles of segment {si}"
    sw = OL.build(sp, d["window"], 1, d["tile"])
    assert [int(r[4]) for r in sw.seg_info] == d["stepwise_lengths"]


def _random_spans(rng, ntraj, tmax, p=(1, 9), m=(0, 7), x=(1, 9)):
    T = rng.integers(0, tmax + 1, size=ntraj)
    n = int(T.sum())
    text = rng.integers(x[0], x[1] + 1, size=n)
    act = np.array([rng.integers(0, t + 1) for t in text], np.int64)
    return WL.explicit_spans(T, rng.integers(p[0], p[1] + 1, size=ntraj),
                             rng.integers(m[0], m[1] + 1, size=n), text, act)


@pytest.mark.parametrize("seed", range(6))
def test_invariants_random(seed):
    rng = np.random.default_rng(seed)
    sp = _random_spans(rng, 3, 9)
    W = int(rng.integers(1, 5))
    L = int(rng.integers(1, 5))
    tile = int(rng.choice([1, 3, 4, 8]))
    lay = OL.build(sp, W, L, tile)
    kind, step, traj = WL.canonical_tokens(sp)
    # O(nT/K) items: ceil(T/L) segments per trajectory with no cap (Sec. 3.3)
    T = np.diff(sp.step_offsets)
    assert len(lay.segments) == sum(math.ceil(t / L) for t in T)
    # every action token is trained exactly once (Eq. loss)
    act = []
    off = sp.canon_offsets()
    for t in range(sp.num_traj):
        c = off[t] + sp.prompt_len[t]
        for s in range(sp.step_offsets[t], sp.step_offsets[t + 1]):
            c += sp.img_len[s]
            act.extend(range(c + sp.text_len[s] - sp.action_len[s], c + sp.text_len[s]))
            c += sp.text_len[s]
    assert sorted(lay.loss_tgt_src.tolist()) == sorted(act)
    # the advantage is shared per rollout: each row carries its token's trajectory
    assert (lay.loss_traj == traj[lay.loss_tgt_src]).all()
    # the predicting row is the packed token right before the target
    assert (lay.tok_src[lay.loss_pred_row + 1] == lay.loss_tgt_src).all()
    for sg in lay.segments:
        m = OL.visibility(sg, W)
        assert m.diagonal().all()                      # every row sees itself
        # a query of a trained turn s sees exactly min(s, W) screenshots
        for i in range(sg.length):
            s = int(sg.step[i])
            if s >= sg.a:
                vis_img = set(sg.step[(sg.kind == OL.KIND_IMAGE) & m[i]].tolist())
                present = set(range(max(1, s - W + 1), s + 1))
                if sg.kind[i] == OL.KIND_IMAGE:
                    # an image token only sees its own block up to itself
                    assert vis_img <= present
                else:
                    imgs_present = {j for j in present if sp.img_len[sp.step_offsets[sg.traj] + j - 1] > 0}
                    assert vis_img == imgs_present
    # tile map: t = 1 equals the mask itself; CSR and transposed CSR agree
    entries_q = {(g, int(c), int(k)) for g in range(len(lay.tile_seg))
                 for c, k in zip(lay.qt_col[lay.qt_ptr[g]:lay.qt_ptr[g + 1]],
                                 lay.qt_cls[lay.qt_ptr[g]:lay.qt_ptr[g + 1]])}
    entries_k = {(int(r), g, int(k)) for g in range(len(lay.tile_seg))
                 for r, k in zip(lay.kt_row[lay.kt_ptr[g]:lay.kt_ptr[g + 1]],
                                 lay.kt_cls[lay.kt_ptr[g]:lay.kt_ptr[g + 1]])}
    assert entries_q == entries_k
    assert lay.seg_pairs.sum() == sum(int(OL.visibility(sg, W).sum()) for sg in lay.segments)


def test_visibility_rows_are_rows_of_the_mask():
    rng = np.random.default_rng(5)
    sp = _random_spans(rng, 2, 6)
    lay = OL.build(sp, 2, 3, 4)
    for sg in lay.segments:
        rows = np.arange(sg.length)[::2]
        assert (OL.visibility_rows(sg, 2, rows) == OL.visibility(sg, 2)[rows]).all()


def test_tile_one_is_the_mask():
    rng = np.random.default_rng(11)
    sp = _random_spans(rng, 2, 5)
    lay = OL.build(sp, 2, 3, 1)
    for si, sg in enumerate(lay.segments):
        grid = _tile_grid(lay, si)
        m = OL.visibility(sg, 2)
        assert ((grid == OL.CLS_FULL) == m).all()
        assert not (grid == OL.CLS_PARTIAL).any()


def test_trajectory_level_is_plain_causal():
    """W >= T and L >= T: one segment per trajectory with plain causal
    visibility (the trajectory-level mode, Sec. 1)."""
    sp = WL.explicit_spans([5, 4], [3, 2], [4] * 9, [3] * 9, [1] * 9)
    lay = OL.build(sp, 10, 10, 4)
    assert len(lay.segments) == 2
    off = sp.canon_offsets()
    for t, sg in enumerate(lay.segments):
        assert (sg.canon == np.arange(off[t], off[t + 1])).all()
        m = OL.visibility(sg, 10)
        assert (m == np.tril(np.ones((sg.length, sg.length), bool))).all()


def test_stepwise_keeps_only_final_screenshot():
    """L = 1 and W = 1: each turn is a sample holding the prompt, all earlier
    text and only the current screenshot (step-wise decomposition, Sec. 1)."""
    sp = WL.explicit_spans([4], [3], [5, 6, 7, 8], [2, 3, 4, 5], [1, 1, 2, 2])
    lay = OL.build(sp, 1, 1, 4)
    assert len(lay.segments) == 4
    for j, sg in enumerate(lay.segments, start=1):
        assert set(sg.step[sg.kind == OL.KIND_IMAGE].tolist()) == {j}
        assert sg.length == 3 + sum([2, 3, 4, 5][:j]) + [5, 6, 7, 8][j - 1]


@pytest.mark.parametrize("W,L", [(1, 2), (2, 3), (3, 5), (2, 1)])
def test_segment_equals_stepwise_context(W, L):
    """An action token sees the same canonical keys inside its segment as in
    its step-wise sample (both keep all text and the last W screenshots).

    This holds whenever the row predicting a turn's first action token
    belongs to that turn, i.e. every turn has a screenshot (m >= 1); the
    workloads always do.
    """
    rng = np.random.default_rng(W * 10 + L)
    sp = _random_spans(rng, 2, 7, m=(1, 7))
    seg = OL.build(sp, W, L, 4)
    sw = OL.build(sp, W, 1, 4)

    def visible_sets(lay):
        out = {}
        for sg in lay.segments:
            m = OL.visibility(sg, W)
            for p, t in zip(lay.loss_pred_row, lay.loss_tgt_src):
                if sg.start <= p < sg.start + sg.length:
                    i = p - sg.start
                    out[int(t)] = frozenset(sg.canon[m[i]].tolist())
        return out

    assert visible_sets(seg) == visible_sets(sw)


def test_capacity_cap_and_error():
    sp = WL.explicit_spans([6], [4], [10] * 6, [3] * 6, [1] * 6)
    cap = 45
    lay = OL.build(sp, 2, 6, 4, cap=cap)
    for sg in lay.segments:
        assert sg.length <= cap
    # each segment closes because L is reached or the next turn would overflow
    for sg in lay.segments[:-1]:
        p, img, text, _ = 4, np.full(6, 10), np.full(6, 3), None
        assert OL.segment_length(p, img, text, 2, sg.a, sg.b + 1) > cap or sg.b - sg.a == 6
    with pytest.raises(OL.CapacityError):
        OL.build(sp, 2, 6, 4, cap=10)


def test_buffers_next_fit():
    sp = WL.explicit_spans([3, 3], [2, 2], [3] * 6, [2] * 6, [1] * 6)
    lay = OL.build(sp, 1, 1, 4, buffer_tokens=16)
    B = 16
    assert lay.packed_tokens == lay.num_buffers * B
    prev_buf, fill = -1, 0
    for sg in lay.segments:
        buf = sg.start // B
        assert (sg.start + sg.length - 1) // B == buf      # never straddles
        if buf != prev_buf:
            assert sg.start == buf * B
            if prev_buf >= 0:
                assert fill + sg.length > B                 # opened only when needed
            prev_buf, fill = buf, 0
        fill += sg.length
    pads = lay.tok_src < 0
    assert (lay.tok_meta[pads] == OL.KIND_PAD).all()
    assert pads.sum() == lay.packed_tokens - sum(sg.length for sg in lay.segments)


def test_empty_and_zero_turn_trajectories():
    sp = WL.explicit_spans([0, 2, 0], [3, 3, 3], [2, 2], [2, 2], [1, 1])
    lay = OL.build(sp, 1, 1, 4)
    assert len(lay.segments) == 2 and all(sg.traj == 1 for sg in lay.segments)
    sp0 = WL.explicit_spans([], [], [], [], [])
    lay0 = OL.build(sp0, 1, 1, 4)
    assert lay0.packed_tokens == 0 and len(lay0.segments) == 0


# ---- anchored mode (the algorithm as printed)

def test_anchored_hand_worked_example():
    with open(os.path.join(GOLD, "alg2_anchored_example.json")) as f:
        d = json.load(f)
    s = d["spans"]
    sp = WL.explicit_spans(s["steps"], s["prompt"], s["img"], s["text"], s["action"])
    lay = OL.build(sp, d["K"], d["delta"], 4, mode="anchored")
    got = [[sg.traj, sg.a, sg.b, sg.start, sg.length] for sg in lay.segments]
    assert got == d["segments"]
    imgs = [sorted(set(sg.step[sg.kind == OL.KIND_IMAGE].tolist())) for sg in lay.segments]
    assert imgs == d["images"]
    assert lay.tok_src.tolist() == d["tok_src"]
    assert list(zip(lay.loss_pred_row.tolist(), lay.loss_tgt_src.tolist())) == \
        [tuple(r) for r in d["loss_rows"]]
    assert lay.seg_pairs.tolist() == d["pairs"]
    assert OL.anchored_turns(7, 2, 2) == [(1, 5, (1, 2, 3, 4)), (5, 7, (3, 4, 5, 6)),
                                         (7, 8, (5, 6, 7))]


def test_anchored_no_turns_no_segment():
    assert OL.anchored_turns(0, 3, 5) == []


@pytest.mark.parametrize("T,K,D", [(1, 1, 1), (5, 1, 1), (30, 3, 5), (30, 5, 5), (50, 8, 5),
                                   (12, 3, 40), (9, 2, 1)])
def test_anchored_counts_and_invariants(T, K, D):
    """First segment K + Delta turns, then Delta turns each; every stream
    holds at most K + Delta screenshots and a new stream starts with K + 1;
    Delta >= T gives the whole trajectory as one item."""
    segs = OL.anchored_turns(T, K, D)
    lens = [b - a for a, b, _ in segs]
    if T <= K + D:
        assert segs == [(1, T + 1, tuple(range(1, T + 1)))]
    else:
        assert lens[0] == K + D and all(n == D for n in lens[1:-1]) and 1 <= lens[-1] <= D
        assert len(segs) == 1 + -(-(T - K - D) // D)
    assert segs[0][0] == 1 and segs[-1][1] == T + 1
    assert all(segs[i][1] == segs[i + 1][0] for i in range(len(segs) - 1))
    for i, (a, b, imgs) in enumerate(segs):
        assert len(imgs) <= K + D
        assert list(imgs) == list(range(max(1, a - K) if i else 1, b))
        if i:
            assert sum(1 for j in imgs if j <= a) == K + 1


def test_anchored_tokens_equal_window_k_plus_one():
    """The screenshots the algorithm keeps are those a window of K + 1
    turns before each segment start would keep (two constructions)."""
    rng = np.random.default_rng(5)
    for _ in range(20):
        T = int(rng.integers(1, 25))
        K, D = int(rng.integers(1, 6)), int(rng.integers(1, 6))
        p = int(rng.integers(1, 9))
        img = rng.integers(0, 5, size=T)
        text = rng.integers(0, 5, size=T)
        for a, b, imgs in OL.anchored_turns(T, K, D):
            c1 = OL.segment_tokens_with(p, img, text, imgs, b, 0)
            c2 = OL.segment_tokens(p, img, text, K + 1, a, b, 0)
            for x, y in zip(c1, c2):
                assert np.array_equal(x, y)


def test_anchored_visibility_is_causal_and_trains_every_action_once():
    rng = np.random.default_rng(6)
    T = 11
    sp = WL.explicit_spans([T], [5], rng.integers(1, 4, size=T), rng.integers(2, 6, size=T),
                           [1] * T)
    lay = OL.build(sp, 3, 2, 4, mode="anchored")
    for sg in lay.segments:
        n = sg.length
        assert np.array_equal(OL.visibility(sg, None), np.tril(np.ones((n, n), bool)))
    assert len(lay.loss_tgt_src) == T
    assert len(set(lay.loss_tgt_src.tolist())) == T
    with pytest.raises(ValueError):
        OL.build(sp, 3, 2, 4, cap=100, mode="anchored")


def test_empty_prompt():
    """A trajectory without a prompt opens its first segment with turn 1's
    screenshot; later turns stop seeing it once it leaves the window.  A
    segment without tokens, and a trained token opening its segment (no row
    before it predicts it, Eq. loss), are argument errors."""
    sp = WL.explicit_spans([3], [0], [2, 2, 2], [2, 2, 2], [1, 1, 1])
    lay = OL.build(sp, 1, 3, 4)
    sg = lay.segments[0]
    assert sg.length == 12 and sg.kind[0] == OL.KIND_IMAGE and sg.canon[0] == 0
    m = OL.visibility(sg, 1)
    later = np.nonzero(sg.step >= 2)[0]
    assert not m[later][:, :2].any()          # turn 1's screenshot has expired
    assert m[later][:, 2:4].all()             # turn 1's text has not
    assert lay.loss_pred_row.tolist() == [2, 6, 10]
    with pytest.raises(ValueError):           # turn 1 is all trained text
        OL.build(WL.explicit_spans([2], [0], [0, 1], [2, 2], [2, 1]), 1, 1, 4)
    with pytest.raises(ValueError):           # turn 1 has no token at all
        OL.build(WL.explicit_spans([2], [0], [0, 1], [0, 2], [0, 1]), 1, 1, 4)
