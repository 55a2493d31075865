"""GPU layout (seg_build_layout through the C ABI) bit-exact against the oracle:
tokens, loss rows, segment records, tile map (CSR and transposed CSR, and the
attention kernels' FULL-first walking orders of both) and the exact
visible-pair counts."""
import json
import os

import numpy as np
import pytest

from oracle import layout as OL
from paper_2607_11185_amd import seg as S
from paper_2607_11185_amd import workload as WL
from tests.gpu_helpers import say

pytestmark = pytest.mark.gpu
GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gpu(sp, W, L, tile, cap=0, buf=0, mode="sliding"):
    say(f"  layout W={W} L={L} tile={tile} cap={cap} buf={buf} traj={sp.num_traj} {mode}")
    pr = S.Problem.from_spans(sp, W, L, cap, buf, tile, mode)
    return S.seg_build_layout(pr, device="cuda").host()


def _balance8(work):
    """Boundaries of eight consecutive ranges of about equal total work: the
    first index whose prefix reaches ceil(total * x / 8)."""
    pre = np.concatenate([[0], np.cumsum(work)]).astype(np.int64)
    b = [0]
    for x in range(1, 8):
        b.append(max(int(np.searchsorted(pre, (pre[-1] * x + 7) // 8, "left")), b[-1]))
    return b + [len(work)]


def _check_schedule(got):
    """The attention launch schedule, recomputed from the layout's own CSR
    lengths (listed k-tiles per q-tile, listed q-tiles per k-tile): the
    host's balanced tile ranges must be what the GPU's tile map gives."""
    rows, cols = np.diff(got["qt_ptr"]), np.diff(got["kt_ptr"])
    assert got["xcd_rows"].tolist() == _balance8(rows)
    assert got["xcd_cols"].tolist() == _balance8(cols)


def _want_order(cols, cls):
    """One q-tile's walking order of the q-tile-stationary kernels: its listed
    k-tiles with every FULL one first and the PARTIAL ones after, each in
    ascending order, bit 31 marking PARTIAL (as int32)."""
    cols = np.asarray(cols, np.int64)
    cls = np.asarray(cls)
    full, part = cols[cls == OL.CLS_FULL], cols[cls == OL.CLS_PARTIAL]
    assert len(full) + len(part) == len(cols)
    return np.concatenate([full, part | (1 << 31)]).astype(np.uint32).view(np.int32)


def _check_order(got, g, e0, e1):
    want = _want_order(got["qt_col"][e0:e1], got["qt_cls"][e0:e1])
    assert np.array_equal(got["qt_ord"][e0:e1], want), ("qt_ord", g)


def _check_col_order(got, g, e0, e1):
    """One k-tile's walking order of the dK/dV kernel: FULL q-tiles first,
    then PARTIAL ones, each descending, bit 31 marking PARTIAL."""
    rows = np.asarray(got["kt_row"][e0:e1], np.int64)
    cls = np.asarray(got["kt_cls"][e0:e1])
    full, part = rows[cls == OL.CLS_FULL], rows[cls == OL.CLS_PARTIAL]
    assert len(full) + len(part) == len(rows)
    want = np.concatenate([full[::-1], part[::-1] | (1 << 31)]).astype(np.uint32).view(np.int32)
    assert np.array_equal(got["kt_ord"][e0:e1], want), ("kt_ord", g)


def _check_all(got, ref):
    for f in ("tok_src", "tok_meta", "loss_pred_row", "loss_tgt_src", "loss_traj", "tile_seg",
              "qt_ptr", "qt_col", "qt_cls", "kt_ptr", "kt_row", "kt_cls", "seg_pairs"):
        assert np.array_equal(got[f].astype(np.int64), getattr(ref, f).astype(np.int64)), f
    assert np.array_equal(got["seg_info"].astype(np.int64), ref.seg_info), "seg_info"
    assert int(got["tile_nnz"][0]) == len(ref.qt_col)
    ptr, kptr = got["qt_ptr"], got["kt_ptr"]
    for g in range(len(ptr) - 1):
        _check_order(got, g, ptr[g], ptr[g + 1])
        _check_col_order(got, g, kptr[g], kptr[g + 1])
    if len(got["qt_ptr"]) > 1:
        _check_schedule(got)


@pytest.mark.parametrize("name", ["appA_example_a.json", "appA_example_b.json"])
def test_hand_worked(name):
    with open(os.path.join(GOLD, name)) as f:
        d = json.load(f)
    s = d["spans"]
    sp = WL.explicit_spans(s["steps"], s["prompt"], s["img"], s["text"], s["action"])
    got = _gpu(sp, d["window"], d["seg_steps"], d["tile"])
    _check_all(got, OL.build(sp, d["window"], d["seg_steps"], d["tile"]))


@pytest.mark.parametrize("seed", range(12))
def test_random_spans(seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(1, 5))
    T = rng.integers(0, 9, size=n)
    ns = int(T.sum())
    text = rng.integers(0, 40, size=ns)
    sp = WL.explicit_spans(T, rng.integers(1, 50, size=n), rng.integers(0, 60, size=ns), text,
                           [int(rng.integers(0, t + 1)) for t in text])
    W, L = int(rng.integers(1, 5)), int(rng.integers(1, 5))
    tile = int(rng.choice([1, 3, 4, 16, 128]))
    buf = int(rng.choice([0, 0, 400]))
    try:
        ref = OL.build(sp, W, L, tile, buffer_tokens=buf)
    except OL.CapacityError:
        ref = OL.build(sp, W, L, tile)
        buf = 0
    _check_all(_gpu(sp, W, L, tile, buf=buf), ref)


@pytest.mark.parametrize("seed", range(6))
def test_random_spans_empty_prompts(seed):
    """Prompts of 0-2 tokens: layouts bit-exact where the oracle accepts the
    batch; where it rejects it (a segment without tokens, or a trained token
    opening its segment) the library returns an argument error."""
    from paper_2607_11185_amd import _lib
    rng = np.random.default_rng(300 + seed)
    n = int(rng.integers(1, 4))
    T = rng.integers(1, 7, size=n)
    ns = int(T.sum())
    text = rng.integers(0, 30, size=ns)
    sp = WL.explicit_spans(T, rng.integers(0, 3, size=n), rng.integers(0, 50, size=ns), text,
                           [int(rng.integers(0, t + 1)) for t in text])
    W, L = int(rng.integers(1, 4)), int(rng.integers(1, 4))
    tile = int(rng.choice([1, 4, 16, 128]))
    try:
        ref = OL.build(sp, W, L, tile)
    except ValueError:
        with pytest.raises(_lib.SegError) as ei:
            _gpu(sp, W, L, tile)
        assert ei.value.status == _lib.SEG_ERR_ARG
        return
    _check_all(_gpu(sp, W, L, tile), ref)


@pytest.mark.parametrize("cfg", [WL.TINY, WL.SMALL], ids=lambda c: c.name)
def test_configs_full(cfg):
    sp = WL.make_spans(cfg)
    got = _gpu(sp, cfg.window, cfg.seg_steps, 128, cfg.max_seg_tokens, cfg.buffer_tokens)
    _check_all(got, OL.build(sp, cfg.window, cfg.seg_steps, 128, cfg.max_seg_tokens,
                             cfg.buffer_tokens))


@pytest.mark.parametrize("cfg", [WL.SEVEN_B, WL.STEPWISE_7B, WL.LONG], ids=lambda c: c.name)
def test_configs_large_sampled(cfg):
    """Full-size layouts: every token, loss row and segment record exact; the
    tile map and pair counts of sampled segments exact."""
    sp = WL.make_spans(cfg)
    got = _gpu(sp, cfg.window, cfg.seg_steps, 128, cfg.max_seg_tokens, cfg.buffer_tokens)
    ref = OL.build(sp, cfg.window, cfg.seg_steps, 128, cfg.max_seg_tokens, cfg.buffer_tokens,
                   with_tiles=False)
    for f in ("tok_src", "tok_meta", "loss_pred_row", "loss_tgt_src", "loss_traj"):
        assert np.array_equal(got[f].astype(np.int64), getattr(ref, f).astype(np.int64)), f
    assert np.array_equal(got["seg_info"].astype(np.int64), ref.seg_info)
    _check_schedule(got)
    S_ = len(ref.segments)
    lens = [sg.length for sg in ref.segments]
    picks = sorted({0, S_ // 2, S_ - 1, int(np.argmax(lens))})
    for si in picks:
        sg = ref.segments[si]
        say(f"  tiles of segment {si} ({sg.length} tokens)")
        cls, pairs = OL.segment_tiles(sg, cfg.window, 128)
        assert int(got["seg_pairs"][si]) == pairs
        base = int(ref.seg_info[si][5])
        nt = cls.shape[0]
        for i in range(nt):
            g = base + i
            e0, e1 = got["qt_ptr"][g], got["qt_ptr"][g + 1]
            cols = got["qt_col"][e0:e1] - base
            want = np.nonzero(cls[i])[0]
            assert np.array_equal(cols, want), (si, i)
            assert np.array_equal(got["qt_cls"][e0:e1], cls[i][want]), (si, i)
            _check_order(got, g, e0, e1)
        for j in range(nt):
            g = base + j
            e0, e1 = got["kt_ptr"][g], got["kt_ptr"][g + 1]
            rows = got["kt_row"][e0:e1] - base
            want = np.nonzero(cls[:, j])[0]
            assert np.array_equal(rows, want), (si, j)
            assert np.array_equal(got["kt_cls"][e0:e1], cls[want, j]), (si, j)
            _check_col_order(got, g, e0, e1)
    # with multi-turn segments, expired screenshots make skipped tiles; a
    # step-wise sample already holds only its last W screenshots
    total_lower = sum((n := -(-l // 128)) * (n + 1) // 2 for l in lens)
    if cfg.seg_steps > 1:
        assert int(got["tile_nnz"][0]) < total_lower
    else:
        assert int(got["tile_nnz"][0]) <= total_lower


def test_empty_batch():
    sp = WL.explicit_spans([0, 0], [3, 3], [], [], [])
    got = _gpu(sp, 2, 2, 128)
    assert got["tok_src"].size == 0 and int(got["qt_ptr"][0]) == 0


@pytest.mark.parametrize("mode", ["sliding", "anchored"])
def test_tile_one(mode):
    """Single-token tiles: every visible pair is its own tile, the diagonal
    ones full."""
    rng = np.random.default_rng(7)
    T = [4, 0, 6]
    ns = sum(T)
    text = rng.integers(0, 9, size=ns)
    sp = WL.explicit_spans(T, [3, 2, 5], rng.integers(0, 7, size=ns), text,
                           [int(rng.integers(0, t + 1)) for t in text])
    ref = OL.build(sp, 2, 2, 1, mode=mode)
    assert (ref.qt_cls == OL.CLS_FULL).all()
    _check_all(_gpu(sp, 2, 2, 1, mode=mode), ref)


# ---- anchored mode (the App. D algorithm as printed)

def test_anchored_hand_worked():
    with open(os.path.join(GOLD, "alg2_anchored_example.json")) as f:
        d = json.load(f)
    s = d["spans"]
    sp = WL.explicit_spans(s["steps"], s["prompt"], s["img"], s["text"], s["action"])
    got = _gpu(sp, d["K"], d["delta"], 4, mode="anchored")
    assert got["tok_src"].tolist() == d["tok_src"]
    assert got["seg_info"][:, [0, 1, 2, 3, 4]].tolist() == d["segments"]
    assert list(zip(got["loss_pred_row"].tolist(), got["loss_tgt_src"].tolist())) == \
        [tuple(r) for r in d["loss_rows"]]
    assert got["seg_pairs"].tolist() == d["pairs"]
    _check_all(got, OL.build(sp, d["K"], d["delta"], 4, mode="anchored"))


@pytest.mark.parametrize("seed", range(10))
def test_anchored_random_spans(seed):
    rng = np.random.default_rng(300 + seed)
    n = int(rng.integers(1, 5))
    T = rng.integers(0, 14, size=n)
    ns = int(T.sum())
    text = rng.integers(0, 40, size=ns)
    sp = WL.explicit_spans(T, rng.integers(1, 50, size=n), rng.integers(0, 60, size=ns), text,
                           [int(rng.integers(0, t + 1)) for t in text])
    K, D = int(rng.integers(1, 5)), int(rng.integers(1, 5))
    tile = int(rng.choice([1, 3, 16, 128]))
    buf = int(rng.choice([0, 0, 900]))
    try:
        ref = OL.build(sp, K, D, tile, buffer_tokens=buf, mode="anchored")
    except OL.CapacityError:
        ref = OL.build(sp, K, D, tile, mode="anchored")
        buf = 0
    _check_all(_gpu(sp, K, D, tile, buf=buf, mode="anchored"), ref)
