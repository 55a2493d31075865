"""Host-side checks of libseg's C ABI (no GPU): the library loads and exports
every symbol of include/seg.h; seg_layout_query agrees with the oracle's
segmentation; argument validation rejects bad input before any HIP call."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import layout as OL
from paper_2607_11185_amd import _lib
from paper_2607_11185_amd import seg as S
from paper_2607_11185_amd import workload as WL

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _lib_or_skip():
    if not os.path.exists(_lib.LIB_PATH):
        pytest.skip("libseg.so not built")
    return _lib.lib()


def test_exports_every_declared_symbol():
    L = _lib_or_skip()
    with open(os.path.join(ROOT, "include", "seg.h")) as f:
        hdr = f.read()
    declared = set(re.findall(r"^\s*(?:seg_status|size_t|void|const char \*)\s*(seg_\w+)\s*\(", hdr, re.M))
    assert declared == set(_lib.EXPORTS)
    for name in declared:
        assert hasattr(L, name), name


def _sizes_oracle(sp, W, L, tile, cap=0, buf=0, mode="sliding"):
    lay = OL.build(sp, W, L, tile, cap=cap, buffer_tokens=buf, with_tiles=False, mode=mode)
    G = sum(-(-sg.length // tile) for sg in lay.segments)
    Z = sum((n := -(-sg.length // tile)) * (n + 1) // 2 for sg in lay.segments)
    return dict(num_segments=len(lay.segments), num_buffers=lay.num_buffers,
                loss_rows=len(lay.loss_pred_row), num_qtiles=G,
                packed_tokens=lay.packed_tokens,
                traj_tokens=int(sp.canon_offsets()[-1]), tile_nnz_max=Z,
                max_seg_len=max((sg.length for sg in lay.segments), default=0))


@pytest.mark.parametrize("cfg", [WL.TINY, WL.SMALL, WL.SEVEN_B, WL.STEPWISE_7B, WL.LONG],
                         ids=lambda c: c.name)
def test_query_matches_oracle(cfg):
    _lib_or_skip()
    sp = WL.make_spans(cfg)
    pr = S.Problem.from_spans(sp, cfg.window, cfg.seg_steps, cfg.max_seg_tokens, cfg.buffer_tokens)
    got = S.seg_layout_query(pr).as_dict()
    want = _sizes_oracle(sp, cfg.window, cfg.seg_steps, 128, cfg.max_seg_tokens, cfg.buffer_tokens)
    for k, v in want.items():
        assert got[k] == v, (k, got[k], v)
    assert got["workspace_bytes"] > 0


def test_query_random_and_edge():
    _lib_or_skip()
    rng = np.random.default_rng(0)
    for it in range(30):
        n = int(rng.integers(0, 4))
        T = rng.integers(0, 7, size=n)
        ns = int(T.sum())
        text = rng.integers(0, 9, size=ns)
        # prompts may be empty: a segment without tokens, or one opened by a
        # trained token, is an argument error on both sides
        sp = WL.explicit_spans(T, rng.integers(0, 9, size=n), rng.integers(0, 9, size=ns), text,
                               [int(rng.integers(0, t + 1)) for t in text])
        W, L, tile = int(rng.integers(1, 4)), int(rng.integers(1, 4)), int(rng.choice([1, 4, 128]))
        pr = S.Problem.from_spans(sp, W, L, 0, 0, tile)
        try:
            want = _sizes_oracle(sp, W, L, tile)
        except ValueError:
            with pytest.raises(_lib.SegError) as ei:
                S.seg_layout_query(pr)
            assert ei.value.status == _lib.SEG_ERR_ARG
            continue
        got = S.seg_layout_query(pr).as_dict()
        for k, v in want.items():
            assert got[k] == v, (it, k, got[k], v)


def _prob(**kw):
    sp = WL.explicit_spans([3], [4], [5, 5, 5], [3, 3, 3], [1, 1, 1])
    d = dict(window=2, seg_steps=2, max_seg_tokens=0, buffer_tokens=0, tile=128)
    d.update(kw)
    return S.Problem.from_spans(sp, **d)


@pytest.mark.parametrize("kw,status,text", [
    (dict(window=0), _lib.SEG_ERR_ARG, "window"),
    (dict(seg_steps=0), _lib.SEG_ERR_ARG, "seg_steps"),
    (dict(tile=0), _lib.SEG_ERR_ARG, "tile"),
    (dict(max_seg_tokens=10), _lib.SEG_ERR_CAPACITY, "max_seg_tokens"),
    (dict(buffer_tokens=12), _lib.SEG_ERR_CAPACITY, "buffer_tokens"),
    (dict(mode=7), _lib.SEG_ERR_ARG, "mode"),
    (dict(mode=1, max_seg_tokens=100), _lib.SEG_ERR_UNSUPPORTED, "anchored"),
])
def test_query_errors(kw, status, text):
    _lib_or_skip()
    with pytest.raises(_lib.SegError) as ei:
        S.seg_layout_query(_prob(**kw))
    assert ei.value.status == status and text in str(ei.value)


def test_bad_spans():
    _lib_or_skip()
    bad = [
        WL.explicit_spans([2], [-1], [1, 1], [2, 2], [1, 1]),       # negative prompt
        WL.explicit_spans([2], [0], [0, 1], [2, 2], [2, 1]),        # trained token opens a segment
        WL.explicit_spans([2], [0], [0, 1], [0, 2], [0, 1]),        # segment without tokens
        WL.explicit_spans([2], [3], [1, -1], [2, 2], [1, 1]),       # negative screenshot
        WL.explicit_spans([2], [3], [1, 1], [2, 2], [3, 1]),        # action longer than text
    ]
    for sp in bad:
        with pytest.raises(_lib.SegError) as ei:
            S.seg_layout_query(S.Problem.from_spans(sp, 1, 1))
        assert ei.value.status == _lib.SEG_ERR_ARG
    pr = _prob()
    pr.step_offsets = np.array([1, 3], np.int32)
    with pytest.raises(_lib.SegError):
        S.seg_layout_query(pr)


def test_null_problem_and_last_error():
    L = _lib_or_skip()
    sz = _lib.SegSizes()
    assert L.seg_layout_query(None, ctypes.byref(sz)) == _lib.SEG_ERR_ARG
    assert b"NULL" in L.seg_last_error()
    assert L.seg_layout_query(ctypes.byref(_prob().c()), ctypes.byref(sz)) == _lib.SEG_OK
    assert L.seg_last_error() == b""


def test_build_and_compute_reject_bad_args_before_any_launch():
    L = _lib_or_skip()
    pr = _prob()
    sz = S.seg_layout_query(pr)
    lay = _lib.SegLayout()
    # workspace too small
    st = L.seg_build_layout(ctypes.byref(pr.c()), ctypes.byref(sz), ctypes.byref(lay), None, 0, None)
    assert st == _lib.SEG_ERR_WORKSPACE
    # sizes that do not belong to the problem
    sz2 = _lib.SegSizes.from_buffer_copy(sz)
    sz2.loss_rows += 1
    st = L.seg_build_layout(ctypes.byref(pr.c()), ctypes.byref(sz2), ctypes.byref(lay), None,
                            1 << 30, None)
    assert st == _lib.SEG_ERR_ARG
    # attention: unsupported head_dim / ratio / tile
    lay.tile, lay.window = 128, 2
    for hq, hkv, d, want in ((4, 1, 96, _lib.SEG_ERR_UNSUPPORTED), (4, 3, 64, _lib.SEG_ERR_UNSUPPORTED)):
        st = L.seg_attn_fwd(ctypes.byref(lay), ctypes.byref(sz), 0, hq, hkv, d, 0.1, None, None,
                            None, None, None, None, 1 << 40, None)
        assert st == want, (hq, hkv, d, st)
    lay.tile = 64
    st = L.seg_attn_fwd(ctypes.byref(lay), ctypes.byref(sz), 0, 4, 1, 64, 0.1, None, None, None,
                        None, None, None, 1 << 40, None)
    assert st == _lib.SEG_ERR_UNSUPPORTED
    lay.tile = 128
    # a layout whose launch schedule was not set by seg_build_layout
    st = L.seg_attn_bwd(ctypes.byref(lay), ctypes.byref(sz), 0, 4, 1, 64, 0.1, None, None, None,
                        None, None, None, None, None, None, None, 0, None)
    assert st == _lib.SEG_ERR_ARG and b"schedule" in L.seg_last_error()
    G = sz.num_qtiles
    for x in range(9):
        lay.xcd_rows[x] = lay.xcd_cols[x] = G * x // 8
    lay.xcd_cols[3], lay.xcd_cols[4] = lay.xcd_cols[4], lay.xcd_cols[3]   # not monotonic
    st = L.seg_attn_bwd(ctypes.byref(lay), ctypes.byref(sz), 0, 4, 1, 64, 0.1, None, None, None,
                        None, None, None, None, None, None, None, 0, None)
    assert st == _lib.SEG_ERR_ARG
    lay.xcd_cols[3], lay.xcd_cols[4] = lay.xcd_cols[4], lay.xcd_cols[3]
    st = L.seg_attn_bwd(ctypes.byref(lay), ctypes.byref(sz), 0, 4, 1, 64, 0.1, None, None, None,
                        None, None, None, None, None, None, None, 0, None)
    assert st == _lib.SEG_ERR_WORKSPACE
    # log-prob: hidden not a multiple of 8, workspace, null tensors
    cfg = S.LossCfg().c()
    args = [None] * 8   # h, row_index, w, target, old_logp, ref_logp, adv, row_traj
    outs = [None] * 7   # logp, loss_tok, clipped, kl_tok, loss_sum, dh, dw
    st = L.seg_logprob_loss(4, 12, 10, 0, *args, 1, ctypes.byref(cfg), *outs, None, 0, None)
    assert st == _lib.SEG_ERR_UNSUPPORTED
    st = L.seg_logprob_loss(4, 16, 10, 0, *args, 1, ctypes.byref(cfg), *outs, None, 0, None)
    assert st == _lib.SEG_ERR_WORKSPACE
    need = L.seg_logprob_workspace_bytes(4, 16, 10, 0)
    st = L.seg_logprob_loss(4, 16, 10, 0, *args, 1, ctypes.byref(cfg), *outs, None, need, None)
    assert st == _lib.SEG_ERR_ARG
    # a KL penalty needs the reference log-probs; a negative one is rejected
    for kl in (0.1, -1.0):
        kcfg = S.LossCfg(kl_coef=kl).c()
        st = L.seg_logprob_loss(4, 16, 10, 0, *args, 1, ctypes.byref(kcfg), *outs, None, need,
                                None)
        assert st == _lib.SEG_ERR_ARG
        assert b"kl" in L.seg_last_error()


def test_noalloc_backward_rejects_before_any_launch():
    """The fixed-scratch backward checks its size limit and the shapes on the
    host: no device is touched for a rejected call."""
    L = _lib_or_skip()
    sz = S.seg_layout_query(_prob())
    lay = _lib.SegLayout()
    lay.tile, lay.window = 128, 2
    for x in range(9):
        lay.xcd_rows[x] = lay.xcd_cols[x] = sz.num_qtiles * x // 8
    big = _lib.SegSizes.from_buffer_copy(sz)
    hq, hkv, d = 28, 4, 128
    big.packed_tokens = _lib.SEG_ATTN_BWD_SCRATCH_BYTES // (8 * hq) + 256
    assert L.seg_attn_workspace_bytes(ctypes.byref(big), 0, hq, hkv, d, 1) > \
        _lib.SEG_ATTN_BWD_SCRATCH_BYTES
    nul = [None] * 10
    st = L.seg_attn_bwd_noalloc(ctypes.byref(lay), ctypes.byref(big), 0, hq, hkv, d, 0.1, *nul, None)
    assert st == _lib.SEG_ERR_WORKSPACE
    assert b"seg_attn_bwd_noalloc" in L.seg_last_error()
    st = L.seg_attn_bwd_noalloc(ctypes.byref(lay), ctypes.byref(sz), 0, 4, 1, 96, 0.1, *nul, None)
    assert st == _lib.SEG_ERR_UNSUPPORTED


def test_query_anchored_matches_oracle():
    """Sizes of the anchored mode (the App. D algorithm) against the oracle,
    on the workloads and on random span lists."""
    _lib_or_skip()
    for cfg in (WL.SMALL, WL.SEVEN_B):
        sp = WL.make_spans(cfg)
        pr = S.Problem.from_spans(sp, cfg.window, cfg.seg_steps, 0, 0, 128, "anchored")
        got = S.seg_layout_query(pr).as_dict()
        want = _sizes_oracle(sp, cfg.window, cfg.seg_steps, 128, mode="anchored")
        for k, v in want.items():
            assert got[k] == v, (cfg.name, k, got[k], v)
    rng = np.random.default_rng(1)
    for it in range(30):
        n = int(rng.integers(0, 4))
        T = rng.integers(0, 12, size=n)
        ns = int(T.sum())
        text = rng.integers(0, 9, size=ns)
        sp = WL.explicit_spans(T, rng.integers(1, 9, size=n), rng.integers(0, 9, size=ns), text,
                               [int(rng.integers(0, t + 1)) for t in text])
        K, D, tile = int(rng.integers(1, 5)), int(rng.integers(1, 5)), int(rng.choice([1, 4, 128]))
        got = S.seg_layout_query(S.Problem.from_spans(sp, K, D, 0, 0, tile, "anchored")).as_dict()
        want = _sizes_oracle(sp, K, D, tile, mode="anchored")
        for k, v in want.items():
            assert got[k] == v, (it, k, got[k], v)


def test_layer_sizing_and_argument_checks():
    """Layer workspace sizing and argument rejection, before any launch."""
    L = _lib_or_skip()
    pr = _prob()
    sz = S.seg_layout_query(pr)
    lay = _lib.SegLayout()
    lay.tile, lay.window = 128, 2
    cfg = S.LayerCfg(256, 512, 4, 2, 64)
    f = L.seg_layer_workspace_bytes(ctypes.byref(sz), ctypes.byref(cfg.c()), 0)
    b = L.seg_layer_workspace_bytes(ctypes.byref(sz), ctypes.byref(cfg.c()), 1)
    assert 0 < f < b
    # smaller row chunks need less workspace
    assert sz.packed_tokens >= 8
    c2 = S.LayerCfg(256, 512, 4, 2, 64, chunk_rows=sz.packed_tokens // 4)
    assert L.seg_layer_workspace_bytes(ctypes.byref(sz), ctypes.byref(c2.c()), 1) < b
    assert L.seg_layer_workspace_bytes(ctypes.byref(sz), ctypes.byref(S.LayerCfg(0, 8, 1, 1, 64).c()),
                                       0) == 0
    w = _lib.SegLayerWeights(*([1] * 9))
    sv = _lib.SegLayerSaved(*([1] * 8))
    g = _lib.SegLayerGrads(*([1] * 9))
    bad = [(S.LayerCfg(250, 512, 4, 2, 64), _lib.SEG_ERR_UNSUPPORTED),     # hidden % 8
           (S.LayerCfg(256, 500, 4, 2, 64), _lib.SEG_ERR_UNSUPPORTED),     # inter % 8
           (S.LayerCfg(16384, 512, 4, 2, 64), _lib.SEG_ERR_UNSUPPORTED),   # hidden too wide
           (S.LayerCfg(256, 512, 4, 3, 64), _lib.SEG_ERR_UNSUPPORTED),     # hq % hkv
           (S.LayerCfg(256, 512, 4, 2, 96), _lib.SEG_ERR_UNSUPPORTED),     # head_dim
           (S.LayerCfg(256, 512, 4, 2, 64, rms_eps=0.0), _lib.SEG_ERR_ARG),
           (S.LayerCfg(256, 512, 4, 2, 64, rope_base=1.0), _lib.SEG_ERR_ARG),
           (S.LayerCfg(256, 512, 4, 2, 64, chunk_rows=-1), _lib.SEG_ERR_ARG)]
    for c, want in bad:
        st = L.seg_layer_fwd(ctypes.byref(lay), ctypes.byref(sz), ctypes.byref(c.c()), ctypes.byref(w),
                             1, 1, ctypes.byref(sv), 1, 1 << 40, None)
        assert st == want, (c, st)
        st = L.seg_layer_bwd(ctypes.byref(lay), ctypes.byref(sz), ctypes.byref(c.c()), ctypes.byref(w),
                             1, ctypes.byref(sv), 1, 1, ctypes.byref(g), 1, 1 << 40, None)
        assert st == want, (c, st)
    # workspace too small, then a NULL weight
    st = L.seg_layer_fwd(ctypes.byref(lay), ctypes.byref(sz), ctypes.byref(cfg.c()), ctypes.byref(w),
                         1, 1, ctypes.byref(sv), 1, f - 1, None)
    assert st == _lib.SEG_ERR_WORKSPACE
    st = L.seg_layer_bwd(ctypes.byref(lay), ctypes.byref(sz), ctypes.byref(cfg.c()), ctypes.byref(w),
                         1, ctypes.byref(sv), 1, 1, ctypes.byref(g), 1, b - 1, None)
    assert st == _lib.SEG_ERR_WORKSPACE
    w.wd = None
    st = L.seg_layer_fwd(ctypes.byref(lay), ctypes.byref(sz), ctypes.byref(cfg.c()), ctypes.byref(w),
                         1, 1, ctypes.byref(sv), 1, f, None)
    assert st == _lib.SEG_ERR_ARG and b"NULL" in L.seg_last_error()
