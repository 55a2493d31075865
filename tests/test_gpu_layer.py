"""GPU decoder layer around the segmented attention (seg_layer_fwd /
seg_layer_bwd through the C ABI) against the float64 oracle layer.

Full parity of the outputs, the saved activations, dx and every weight
gradient on workloads the oracle finishes in seconds: several segments of
several 128-row tiles with ragged tails, hidden and MLP widths that are not
multiples of the GEMM tile, head_dim 64 and 128, buffer padding, row chunking
smaller than the batch; six seeded random problems (widths, head shape,
window, segment length, buffers, chunking, mode).  Plus: chunking leaves the
row-wise results bitwise
unchanged, padding rows get no gradient, and an empty batch gives zero
weight gradients.  At the 7B-class layer width (hidden 3584, MLP 18944,
28q/4kv): sampled output rows against the oracle's row-sampled forward, and
the chunking / padding properties with buffers."""
import numpy as np
import pytest

from oracle import layer as OLY
from oracle import layout as OL
from paper_2607_11185_amd import seg as S
from paper_2607_11185_amd import workload as WL
from tests.gpu_helpers import TOL, GpuRun, rel, say, vis_window

pytestmark = pytest.mark.gpu

MED = WL.Config("med", 2, (4, 7), 48, 150, (30, 90), 6, 2, 3, 4, 2, 64, 128, 1000)
# (workload, hidden, inter, chunk_rows)
CASES = {
    "d64_gqa2_ragged": (MED, 328, 200, 0),
    "d128_chunked": (MED.with_(head_dim=128, seed=1), 256, 688, 300),
    "d64_gqa4_buffers": (MED.with_(hq=8, hkv=2, buffer_tokens=1400, seed=2, steps=(3, 5)), 384, 520,
                         512),
    "mha_w1_l2": (MED.with_(hq=2, hkv=2, window=1, seg_steps=2, seed=3), 136, 72, 97),
    "anchored_k2_d3": (MED.with_(mode="anchored", window=2, seg_steps=3, seed=4, steps=(8, 9)), 264,
                       320, 0),
}
EPS, BASE = 1e-6, 10000.0


class LayerRun:
    def __init__(self, cfg, H, I, chunk_rows, seed=None):
        import torch
        self.cfg, self.H, self.I = cfg, H, I
        self.seed = cfg.seed if seed is None else seed
        self.run = GpuRun(cfg)
        self.lay, self.P, self.dev = self.run.lay, self.run.P, self.run.dev
        self.lc = S.LayerCfg(H, I, cfg.hq, cfg.hkv, cfg.head_dim, EPS, BASE, chunk_rows)
        self.w = WL.layer_weights_torch(self.seed, H, I, cfg.hq, cfg.hkv, cfg.head_dim, self.dev)
        # packed rows carry the hidden state of their canonical token (a
        # padding row, tok_src = -1, takes the last canonical row)
        src = self.run.host["tok_src"].astype(np.int64)
        n_canon = self.run.inp.n_canon
        self.src = np.where(src >= 0, src, n_canon - 1)
        xc = WL.layer_rows_torch(self.seed, "x", n_canon, H, self.dev)
        self.x = xc[torch.from_numpy(self.src).to(self.dev)].contiguous()
        self.dy = WL.layer_rows_torch(self.seed, "dy", self.P, H, self.dev)

    def gpu(self):
        import torch
        y, saved = S.seg_layer_fwd(self.lay, self.lc, self.w, self.x)
        dx, grads = S.seg_layer_bwd(self.lay, self.lc, self.w, self.x, saved, self.dy)
        torch.cuda.synchronize()
        return y, saved, dx, grads

    def oracle(self):
        c = self.cfg
        ref = OL.build(self.run.spans, c.window, c.seg_steps, 128, c.max_seg_tokens,
                       c.buffer_tokens, with_tiles=False, mode=c.mode)
        assert np.array_equal(self.run.host["tok_src"], ref.tok_src)
        x = WL.layer_rows_np(self.seed, "x", self.src, self.H)
        dy = WL.layer_rows_np(self.seed, "dy", np.arange(self.P), self.H)
        w = OLY.Weights(**WL.layer_weights_np(self.seed, self.H, self.I, c.hq, c.hkv, c.head_dim))
        masks = [OL.visibility(sg, vis_window(c)) for sg in ref.segments]
        a = dict(hq=c.hq, hkv=c.hkv, d=c.head_dim, eps=EPS, base=BASE)
        y, saved = OLY.forward(x, w, ref.segments, masks, **a)
        dx, grads = OLY.backward(x, w, ref.segments, masks, **a, saved=saved, dy=dy)
        return ref, y, saved, dx, grads


def _np(t):
    return t.float().cpu().numpy().astype(np.float64)


def _big_tiles(M, N):
    """256x256 tiles of an M x N product: the data-gradient and projection
    GEMMs take the 256-wide kernel from 192 tiles on."""
    return -(-M // 256) * -(-N // 256)


# GEMMs on the 256-wide kernel: ~4.9k packed rows at the 7B-class widths
# (hidden 3584, 28q/4kv, d = 128) with an MLP width of 3072, so dm, db, dO and
# the dq/dk/dv data gradients (and the forward projections) pass 192 tiles
WIDE = (MED.with_(hq=28, hkv=4, head_dim=128, steps=(4, 5), img_len=300, text_len=(60, 120),
                  seed=33), 3584, 3072)


@pytest.mark.parametrize("name", list(CASES))
def test_layer_full_parity(name):
    cfg, H, I, chunk = CASES[name]
    _full_parity(name, cfg, H, I, chunk)


def test_layer_wide_gemm_parity():
    """Full parity where the layer's GEMMs run the 256x256 kernels with the
    accumulate / fp32-store epilogues of the backward (dx and all nine weight
    gradients against the oracle)."""
    cfg, H, I = WIDE
    lr = _full_parity("wide", cfg, H, I, 0)
    assert _big_tiles(lr.P, H) >= 192 and _big_tiles(lr.P, I) >= 192
    assert _big_tiles(lr.P, cfg.hq * cfg.head_dim) >= 192


def _random_layer_case(i):
    """Seeded random layer problem: widths (multiples of 8 only), head shape,
    segment window and length, buffers, row chunking and mode drawn from one
    generator per case."""
    rng = np.random.default_rng(5000 + i)
    hq, hkv, d = [(2, 1, 64), (4, 2, 128), (6, 6, 64), (7, 1, 128), (8, 2, 64)][rng.integers(5)]
    cfg = MED.with_(num_traj=int(rng.integers(1, 3)), steps=(2, 2 + int(rng.integers(0, 3))),
                    prompt_len=int(rng.integers(0, 120)), img_len=int(rng.integers(1, 200)),
                    text_len=(20, 20 + int(rng.integers(0, 100))), action_len=4,
                    window=int(rng.integers(1, 4)), seg_steps=int(rng.integers(1, 4)),
                    hq=hq, hkv=hkv, head_dim=d, seed=6000 + i,
                    mode="anchored" if rng.random() < 0.2 else "sliding")
    if cfg.mode == "sliding" and rng.random() < 0.4:
        ref = OL.build(WL.Inputs(cfg).spans, cfg.window, cfg.seg_steps, 128, with_tiles=False)
        cfg = cfg.with_(buffer_tokens=max(sg.length for sg in ref.segments) + int(rng.integers(0, 500)))
    H = 8 * int(rng.integers(1, 81))
    I = 8 * int(rng.integers(1, 151))
    chunk = int(rng.choice([0, int(rng.integers(1, 900))]))
    return cfg, H, I, chunk


@pytest.mark.parametrize("i", range(6))
def test_layer_random_shapes_parity(i):
    cfg, H, I, chunk = _random_layer_case(i)
    say(f"layer random case {i}: {cfg}")
    _full_parity(f"random{i}", cfg, H, I, chunk)


def _full_parity(name, cfg, H, I, chunk):
    say(f"case {name}: H={H} I={I} chunk_rows={chunk}")
    lr = LayerRun(cfg, H, I, chunk)
    y, saved, dx, grads = lr.gpu()
    ref, y_r, s_r, dx_r, g_r = lr.oracle()
    seg = s_r["pos"] >= 0
    say(f"  P={lr.P} segment rows={int(seg.sum())} segments={len(ref.segments)}")
    checks = [("y", _np(y)[seg], y_r[seg]), ("y1", _np(saved["y1"])[seg], s_r["y1"][seg]),
              ("q", _np(saved["q"])[seg], s_r["qr"][seg]), ("k", _np(saved["k"])[seg], s_r["kr"][seg]),
              ("v", _np(saved["v"])[seg], s_r["v"][seg]), ("o", _np(saved["o"])[seg], s_r["o"][seg]),
              ("lse", _np(saved["lse"])[:, seg], s_r["lse"][:, seg]),
              ("rstd1", _np(saved["rstd1"])[seg], s_r["r1"][seg]),
              ("rstd2", _np(saved["rstd2"])[seg], s_r["r2"][seg]),
              ("dx", _np(dx), dx_r)]
    checks += [("d" + n, _np(grads[n]), g_r[n]) for n in WL.LAYER_WEIGHTS]
    bad = []
    for n, g, r in checks:
        e = rel(g, r)
        say(f"  {n}: rel err {e:.2e}")
        if not e < TOL:
            bad.append((n, e))
    assert not bad, (name, bad)
    # padding rows carry no gradient
    assert np.all(_np(dx)[~seg] == 0)
    return lr


def test_layer_chunking_keeps_rowwise_results_bitwise():
    """Row chunking only changes the order of the weight-gradient sums."""
    cfg, H, I, _ = CASES["d64_gqa2_ragged"]
    lr = LayerRun(cfg.with_(seed=21), H, I, 0)
    y0, s0, dx0, g0 = lr.gpu()
    y0, dx0 = y0.clone(), dx0.clone()
    s0 = {n: t.clone() for n, t in s0.items()}
    g0 = {n: t.clone() for n, t in g0.items()}
    lr.lc.chunk_rows = 131
    y1, s1, dx1, g1 = lr.gpu()
    import torch
    assert torch.equal(y0, y1)
    assert torch.equal(dx0, dx1)
    for n in s0:
        assert torch.equal(s0[n], s1[n]), n
    for n in g0:
        e = rel(_np(g1[n]), _np(g0[n]))
        assert e < 1e-4, (n, e)


def test_layer_determinism_bitwise():
    cfg, H, I, chunk = CASES["d128_chunked"]
    lr = LayerRun(cfg.with_(seed=22), H, I, chunk)
    a = lr.gpu()
    a = (a[0].clone(), a[2].clone(), {n: t.clone() for n, t in a[3].items()})
    b = lr.gpu()
    import torch
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[2])
    for n in a[2]:
        assert torch.equal(a[2][n], b[3][n]), n


def test_layer_empty_batch_zero_grads():
    import torch
    sp = WL.explicit_spans([], [], [], [], [])
    prob = S.Problem.from_spans(sp, 2, 3)
    lay = S.seg_build_layout(prob, device="cuda")
    assert lay.sizes.packed_tokens == 0
    H, I = 64, 40
    lc = S.LayerCfg(H, I, 2, 1, 64, EPS, BASE)
    w = WL.layer_weights_torch(0, H, I, 2, 1, 64, "cuda")
    x = torch.empty((0, H), dtype=torch.bfloat16, device="cuda")
    y, saved = S.seg_layer_fwd(lay, lc, w, x)
    grads = {n: torch.full(w[n].shape, 7.0, device="cuda") for n in WL.LAYER_WEIGHTS}
    dx, grads = S.seg_layer_bwd(lay, lc, w, x, saved, torch.empty_like(x), grads=grads)
    torch.cuda.synchronize()
    assert y.shape == (0, H) and dx.shape == (0, H)
    for n in grads:
        assert torch.count_nonzero(grads[n]).item() == 0, n


# the 7B-class layer width (hidden 3584, MLP 18944, 28q/4kv, d = 128) on one
# trajectory of the 7b workload's turn shapes
FULL = WL.SEVEN_B.with_(num_traj=1, steps=(12, 12), seed=31)
FULL_I = 18944


def test_layer_full_width_sampled_rows():
    """Outputs of sampled rows (first, last and random rows of every segment)
    against the oracle's row-sampled forward, which takes keys and values
    from the whole segment."""
    c = FULL
    lr = LayerRun(c, c.hidden, FULL_I, 0)
    say(f"full width: P={lr.P}")
    y, _, _, _ = lr.gpu()
    yg = y.float().cpu().numpy()
    ref = OL.build(lr.run.spans, c.window, c.seg_steps, 128, with_tiles=False, mode=c.mode)
    w = OLY.Weights(**WL.layer_weights_np(lr.seed, c.hidden, FULL_I, c.hq, c.hkv, c.head_dim))
    rng = np.random.default_rng(5)
    for sg in ref.segments:
        rows = np.unique(np.concatenate([[0, sg.length - 1],
                                         rng.choice(sg.length, 6, replace=False)]))
        x_seg = WL.layer_rows_np(lr.seed, "x", lr.src[sg.start:sg.start + sg.length], c.hidden)
        mask = OL.visibility(sg, vis_window(c))
        yr = OLY.forward_rows(x_seg, w, mask, rows, c.hq, c.hkv, c.head_dim, EPS, BASE)
        e = rel(yg[sg.start + rows], yr)
        say(f"  segment at {sg.start} ({sg.length} rows): rel err {e:.2e}")
        assert e < TOL, (sg.start, e)


def test_layer_full_width_chunking_and_padding():
    """At the full width with buffer padding: row chunking leaves y and dx
    bitwise unchanged and the weight gradients equal up to summation order;
    padding rows get dx = 0."""
    import torch
    c = FULL.with_(buffer_tokens=40000, seed=32)
    lr = LayerRun(c, c.hidden, FULL_I, 0)
    pad = lr.run.host["tok_src"] < 0
    say(f"full width with buffers: P={lr.P}, padding rows {int(pad.sum())}")
    assert pad.any()
    y0, _, dx0, g0 = lr.gpu()
    y0, dx0 = y0.clone(), dx0.clone()
    g0 = {n: t.clone() for n, t in g0.items()}
    lr.lc.chunk_rows = 10000
    y1, _, dx1, g1 = lr.gpu()
    assert torch.equal(y0, y1)
    assert torch.equal(dx0, dx1)
    for n in g0:
        e = rel(_np(g1[n]), _np(g0[n]))
        assert e < 1e-4, (n, e)
    assert np.all(_np(dx0)[pad] == 0)
