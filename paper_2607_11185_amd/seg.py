"""Python binding of the libseg entry points, on PyTorch device tensors.

Functions carry the C names (seg_layout_query, seg_build_layout, seg_attn_fwd,
seg_attn_bwd, seg_logprob_loss, seg_layer_fwd, seg_layer_bwd) and only marshal
arguments: they allocate
outputs and workspace with torch on the tensors' device and pass raw
pointers plus torch's current stream to the library.
"""
from __future__ import annotations

import ctypes
import dataclasses
from typing import Optional

import numpy as np

from . import _lib
from ._lib import SegLayout, SegLossCfg, SegProblem, SegSizes, check


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


@dataclasses.dataclass
class Problem:
    """Host-side problem (keeps the int32 span arrays alive for ctypes)."""
    step_offsets: np.ndarray
    prompt_len: np.ndarray
    img_len: np.ndarray
    text_len: np.ndarray
    action_len: np.ndarray
    window: int
    seg_steps: int
    max_seg_tokens: int = 0
    buffer_tokens: int = 0
    tile: int = 128
    mode: int = 0   # _lib.SEG_MODE_SLIDING or _lib.SEG_MODE_ANCHORED

    @classmethod
    def from_spans(cls, spans, window, seg_steps, max_seg_tokens=0, buffer_tokens=0, tile=128,
                   mode=0):
        if isinstance(mode, str):
            mode = {"sliding": _lib.SEG_MODE_SLIDING, "anchored": _lib.SEG_MODE_ANCHORED}[mode]
        return cls(_i32(spans.step_offsets), _i32(spans.prompt_len), _i32(spans.img_len),
                   _i32(spans.text_len), _i32(spans.action_len), int(window), int(seg_steps),
                   int(max_seg_tokens), int(buffer_tokens), int(tile), int(mode))

    def c(self) -> SegProblem:
        def ptr(a):
            return a.ctypes.data_as(_lib.P32) if a.size else ctypes.cast(None, _lib.P32)
        return SegProblem(len(self.prompt_len), ptr(self.step_offsets), ptr(self.prompt_len),
                          ptr(self.img_len), ptr(self.text_len), ptr(self.action_len),
                          self.window, self.seg_steps, self.max_seg_tokens, self.buffer_tokens,
                          self.tile, self.mode)


def seg_layout_query(problem: Problem) -> SegSizes:
    """Sizes of the layout (host only)."""
    sz = SegSizes()
    check(_lib.lib().seg_layout_query(ctypes.byref(problem.c()), ctypes.byref(sz)))
    return sz


def _stream(device) -> ctypes.c_void_p:
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


class Layout:
    """Device arrays of one layout (torch tensors) and the C struct over them."""

    FIELDS = ["seg_info", "tok_src", "tok_meta", "loss_pred_row", "loss_tgt_src", "loss_traj",
              "tile_seg", "qt_ptr", "qt_col", "qt_cls", "qt_ord", "kt_ptr", "kt_row", "kt_cls",
              "kt_ord", "seg_pairs", "tile_nnz"]

    def __init__(self, sizes: SegSizes, device):
        import torch
        S, P, R, G = (sizes.num_segments, sizes.packed_tokens, sizes.loss_rows, sizes.num_qtiles)
        Z = sizes.tile_nnz_max
        i32, u8, i64 = torch.int32, torch.uint8, torch.int64

        def e(n, dt):
            return torch.empty(max(int(n), 1), dtype=dt, device=device)

        self.sizes = sizes
        self.device = device
        self.seg_info = e(S * 8, i32)
        self.tok_src = e(P, i32)
        self.tok_meta = e(P, i32)
        self.loss_pred_row = e(R, i32)
        self.loss_tgt_src = e(R, i32)
        self.loss_traj = e(R, i32)
        self.tile_seg = e(G, i32)
        self.qt_ptr = e(G + 1, i32)
        self.qt_col = e(Z, i32)
        self.qt_cls = e(Z, u8)
        self.qt_ord = e(Z, i32)
        self.kt_ptr = e(G + 1, i32)
        self.kt_row = e(Z, i32)
        self.kt_cls = e(Z, u8)
        self.kt_ord = e(Z, i32)
        self.seg_pairs = e(S, i64)
        self.tile_nnz = e(1, i64)
        self.ws = e(sizes.workspace_bytes, u8)
        self.c = SegLayout(*[getattr(self, f).data_ptr() for f in self.FIELDS], 0, 0)

    def host(self) -> dict:
        """All arrays copied to host numpy, trimmed to their logical sizes."""
        s = self.sizes
        nnz = int(self.tile_nnz.cpu()[0]) if s.num_segments else 0
        lens = {"seg_info": s.num_segments * 8, "tok_src": s.packed_tokens,
                "tok_meta": s.packed_tokens, "loss_pred_row": s.loss_rows,
                "loss_tgt_src": s.loss_rows, "loss_traj": s.loss_rows,
                "tile_seg": s.num_qtiles, "qt_ptr": s.num_qtiles + 1, "qt_col": nnz,
                "qt_cls": nnz, "qt_ord": nnz, "kt_ptr": s.num_qtiles + 1, "kt_row": nnz,
                "kt_cls": nnz, "kt_ord": nnz, "seg_pairs": s.num_segments, "tile_nnz": 1}
        out = {f: getattr(self, f)[:lens[f]].cpu().numpy() for f in self.FIELDS}
        out["seg_info"] = out["seg_info"].reshape(-1, 8)
        out["xcd_rows"] = np.array(self.c.xcd_rows[:], np.int64)
        out["xcd_cols"] = np.array(self.c.xcd_cols[:], np.int64)
        return out


def seg_build_layout(problem: Problem, sizes: Optional[SegSizes] = None, device="cuda",
                     out: Optional[Layout] = None) -> Layout:
    """Build every layout array on the device (token, loss-row and tile kernels).

    ``out`` reuses the arrays of an earlier layout of the same sizes.
    """
    import torch
    device = torch.device(device)
    if sizes is None:
        sizes = seg_layout_query(problem)
    if out is not None:
        if bytes(out.sizes) != bytes(sizes):
            raise ValueError("out was built for different sizes")
        lay = out
    else:
        lay = Layout(sizes, device)
    check(_lib.lib().seg_build_layout(ctypes.byref(problem.c()), ctypes.byref(sizes),
                                      ctypes.byref(lay.c), lay.ws.data_ptr(), lay.ws.numel(),
                                      _stream(device)))
    lay.window = problem.window
    return lay


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return _lib.SEG_BF16
    if t.dtype == torch.float32:
        return _lib.SEG_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def attn_workspace(lay: Layout, dt: int, hq: int, hkv: int, d: int, bwd: bool):
    import torch
    n = _lib.lib().seg_attn_workspace_bytes(ctypes.byref(lay.sizes), dt, hq, hkv, d, int(bwd))
    return torch.empty(max(n, 1), dtype=torch.uint8, device=lay.device)


def seg_attn_fwd(lay: Layout, q, k, v, softmax_scale: float, o=None, lse=None, ws=None):
    """Masked GQA attention forward; q [P, hq, d], k/v [P, hkv, d]."""
    import torch
    P, hq, d = q.shape
    hkv = k.shape[1]
    dt = _dtype_code(q)
    assert q.is_contiguous() and k.is_contiguous() and v.is_contiguous()
    assert k.dtype == q.dtype == v.dtype
    if o is None:
        o = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((hq, P), dtype=torch.float32, device=q.device)
    if ws is None:
        ws = attn_workspace(lay, dt, hq, hkv, d, False)
    check(_lib.lib().seg_attn_fwd(ctypes.byref(lay.c), ctypes.byref(lay.sizes), dt, hq, hkv, d,
                                  float(softmax_scale), q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                  o.data_ptr(), lse.data_ptr(), ws.data_ptr(), ws.numel(),
                                  _stream(q.device)))
    return o, lse


def seg_attn_bwd(lay: Layout, q, k, v, o, lse, dout, softmax_scale: float, dq=None, dk=None,
                 dv=None, ws=None):
    """Gradients of sum(O * dout) w.r.t. q, k, v."""
    import torch
    P, hq, d = q.shape
    hkv = k.shape[1]
    dt = _dtype_code(q)
    for t in (q, k, v, o, dout):
        assert t.is_contiguous() and t.dtype == q.dtype
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    if ws is None:
        ws = attn_workspace(lay, dt, hq, hkv, d, True)
    check(_lib.lib().seg_attn_bwd(ctypes.byref(lay.c), ctypes.byref(lay.sizes), dt, hq, hkv, d,
                                  float(softmax_scale), q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                  o.data_ptr(), lse.data_ptr(), dout.data_ptr(), dq.data_ptr(),
                                  dk.data_ptr(), dv.data_ptr(), ws.data_ptr(), ws.numel(),
                                  _stream(q.device)))
    return dq, dk, dv


def seg_attn_bwd_noalloc(lay: Layout, q, k, v, o, lse, dout, softmax_scale: float, dq, dk, dv):
    """seg_attn_bwd on the library's fixed device scratch: the caller passes
    every output, nothing is allocated (calls on one GPU must not overlap)."""
    dt = _dtype_code(q)
    P, hq, d = q.shape
    hkv = k.shape[1]
    for t in (q, k, v, o, dout, dq):
        assert t.is_contiguous() and t.dtype == q.dtype
    for t in (dk, dv):
        assert t.is_contiguous() and t.dtype == q.dtype
    check(_lib.lib().seg_attn_bwd_noalloc(ctypes.byref(lay.c), ctypes.byref(lay.sizes), dt, hq,
                                          hkv, d, float(softmax_scale), q.data_ptr(),
                                          k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                          lse.data_ptr(), dout.data_ptr(), dq.data_ptr(),
                                          dk.data_ptr(), dv.data_ptr(), _stream(q.device)))
    return dq, dk, dv


@dataclasses.dataclass
class LossCfg:
    eps_low: float = 0.2
    eps_high: float = 0.2
    dual_clip_c: float = 0.0
    loss_scale: float = 1.0
    logit_scale: float = 1.0
    want_grad: bool = True
    kl_coef: float = 0.0

    def c(self) -> SegLossCfg:
        return SegLossCfg(self.eps_low, self.eps_high, self.dual_clip_c, self.loss_scale,
                          self.logit_scale, int(self.want_grad), self.kl_coef)


def logprob_workspace(rows, hidden, vocab, dt, device):
    import torch
    n = _lib.lib().seg_logprob_workspace_bytes(rows, hidden, vocab, dt)
    return torch.empty(max(n, 1), dtype=torch.uint8, device=device)


def seg_logprob_loss(h, row_index, w, target, old_logp, adv, row_traj, cfg: LossCfg, out=None,
                     ws=None, ref_logp=None):
    """Fused log-prob + clipped-ratio loss with KL penalty (+ gradients when
    cfg.want_grad).

    h [n_h, H]; row_index [R] int32 device or None; w [V, H]; target [R] int32;
    old_logp [R] fp32; adv [num_traj] fp32; row_traj [R] int32; ref_logp [R]
    fp32 or None (needed when cfg.kl_coef > 0).
    Returns dict(logp, loss_tok, clipped, kl_tok, loss_sum, dh, dw).
    """
    import torch
    dev = h.device
    R = int(target.numel())
    V, H = w.shape
    dt = _dtype_code(h)
    assert w.dtype == h.dtype and h.is_contiguous() and w.is_contiguous()
    if out is None:
        out = {
            "logp": torch.empty(max(R, 1), dtype=torch.float32, device=dev),
            "loss_tok": torch.empty(max(R, 1), dtype=torch.float32, device=dev),
            "clipped": torch.empty(max(R, 1), dtype=torch.uint8, device=dev),
            "kl_tok": torch.empty(max(R, 1), dtype=torch.float32, device=dev),
            "loss_sum": torch.empty(1, dtype=torch.float32, device=dev),
            "dh": torch.empty((max(R, 1), H), dtype=h.dtype, device=dev) if cfg.want_grad else None,
            "dw": torch.empty((V, H), dtype=torch.float32, device=dev) if cfg.want_grad else None,
        }
    if ws is None:
        ws = logprob_workspace(R, H, V, dt, dev)
    check(_lib.lib().seg_logprob_loss(
        R, H, V, dt, h.data_ptr(), _ptr(row_index), w.data_ptr(), target.data_ptr(),
        old_logp.data_ptr(), _ptr(ref_logp), adv.data_ptr(), row_traj.data_ptr(),
        int(adv.numel()), ctypes.byref(cfg.c()), out["logp"].data_ptr(),
        out["loss_tok"].data_ptr(), out["clipped"].data_ptr(), _ptr(out.get("kl_tok")),
        out["loss_sum"].data_ptr(), _ptr(out["dh"]), _ptr(out["dw"]), ws.data_ptr(), ws.numel(),
        _stream(dev)))
    return out


@dataclasses.dataclass
class LayerCfg:
    """Shape and settings of the decoder layer (seg_layer_cfg)."""
    hidden: int
    inter: int
    hq: int
    hkv: int
    d: int
    rms_eps: float = 1e-6
    rope_base: float = 1e6
    chunk_rows: int = 0

    def c(self) -> "_lib.SegLayerCfg":
        return _lib.SegLayerCfg(self.hidden, self.inter, self.hq, self.hkv, self.d, self.rms_eps,
                                self.rope_base, self.chunk_rows)


def layer_workspace(lay: Layout, cfg: LayerCfg, bwd: bool):
    import torch
    n = _lib.lib().seg_layer_workspace_bytes(ctypes.byref(lay.sizes), ctypes.byref(cfg.c()),
                                             int(bwd))
    return torch.empty(max(n, 1), dtype=torch.uint8, device=lay.device)


def _layer_weights(w: dict):
    return _lib.SegLayerWeights(*[w[n].data_ptr() for n in _lib.LAYER_WEIGHTS])


def seg_layer_fwd(lay: Layout, cfg: LayerCfg, w: dict, x, y=None, saved=None, ws=None):
    """Decoder-layer forward over the packed rows; x [P, H] bf16, w: the bf16
    weights by name (g1, wq, wk, wv, wo, g2, wg, wu, wd).  Returns (y, saved)."""
    import torch
    P, H = x.shape
    dev = x.device
    assert x.dtype == torch.bfloat16 and x.is_contiguous()
    for n in _lib.LAYER_WEIGHTS:
        assert w[n].dtype == torch.bfloat16 and w[n].is_contiguous(), n
    if y is None:
        y = torch.empty_like(x)
    if saved is None:
        bf = dict(dtype=torch.bfloat16, device=dev)
        saved = {"q": torch.empty((P, cfg.hq, cfg.d), **bf), "k": torch.empty((P, cfg.hkv, cfg.d), **bf),
                 "v": torch.empty((P, cfg.hkv, cfg.d), **bf), "o": torch.empty((P, cfg.hq, cfg.d), **bf),
                 "lse": torch.empty((cfg.hq, P), dtype=torch.float32, device=dev),
                 "y1": torch.empty((P, H), **bf),
                 "rstd1": torch.empty(P, dtype=torch.float32, device=dev),
                 "rstd2": torch.empty(P, dtype=torch.float32, device=dev)}
    sv = _lib.SegLayerSaved(*[saved[n].data_ptr() for n in ("q", "k", "v", "o", "lse", "y1", "rstd1",
                                                             "rstd2")])
    if ws is None:
        ws = layer_workspace(lay, cfg, False)
    check(_lib.lib().seg_layer_fwd(ctypes.byref(lay.c), ctypes.byref(lay.sizes), ctypes.byref(cfg.c()),
                                   ctypes.byref(_layer_weights(w)), x.data_ptr(), y.data_ptr(),
                                   ctypes.byref(sv), ws.data_ptr(), ws.numel(), _stream(dev)))
    return y, saved


def seg_layer_bwd(lay: Layout, cfg: LayerCfg, w: dict, x, saved: dict, dy, dx=None, grads=None,
                  ws=None):
    """Decoder-layer backward: returns (dx, grads) with fp32 weight gradients by name."""
    import torch
    dev = x.device
    assert dy.dtype == torch.bfloat16 and dy.is_contiguous() and dy.shape == x.shape
    if dx is None:
        dx = torch.empty_like(x)
    if grads is None:
        grads = {n: torch.empty(w[n].shape, dtype=torch.float32, device=dev) for n in _lib.LAYER_WEIGHTS}
    sv = _lib.SegLayerSaved(*[saved[n].data_ptr() for n in ("q", "k", "v", "o", "lse", "y1", "rstd1",
                                                             "rstd2")])
    g = _lib.SegLayerGrads(*[grads[n].data_ptr() for n in _lib.LAYER_WEIGHTS])
    if ws is None:
        ws = layer_workspace(lay, cfg, True)
    check(_lib.lib().seg_layer_bwd(ctypes.byref(lay.c), ctypes.byref(lay.sizes), ctypes.byref(cfg.c()),
                                   ctypes.byref(_layer_weights(w)), x.data_ptr(), ctypes.byref(sv),
                                   dy.data_ptr(), dx.data_ptr(), ctypes.byref(g), ws.data_ptr(),
                                   ws.numel(), _stream(dev)))
    return dx, grads
