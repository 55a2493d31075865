"""ctypes binding of libseg (the C ABI declared in include/seg.h).

Argument marshalling only: every step of the path runs in the HIP library.
PyTorch tensors provide device memory and the stream.  The library is loaded
from this package directory; if it is missing the binding raises instead of
falling back to anything else.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
# SEG_LIB_PATH selects another build of the same library (the host-sanitizer
# build of build.py); by default the in-tree libseg.so
LIB_PATH = os.environ.get("SEG_LIB_PATH") or os.path.join(HERE, "libseg.so")

SEG_OK, SEG_ERR_ARG, SEG_ERR_CAPACITY, SEG_ERR_WORKSPACE, SEG_ERR_UNSUPPORTED, SEG_ERR_HIP = range(6)
STATUS_NAMES = {0: "SEG_OK", 1: "SEG_ERR_ARG", 2: "SEG_ERR_CAPACITY", 3: "SEG_ERR_WORKSPACE",
                4: "SEG_ERR_UNSUPPORTED", 5: "SEG_ERR_HIP"}
SEG_BF16, SEG_F32 = 0, 1
SEG_ATTN_BWD_SCRATCH_BYTES = 64 << 20

# every symbol include/seg.h declares
EXPORTS = ["seg_layout_query", "seg_build_layout", "seg_attn_workspace_bytes", "seg_attn_fwd",
           "seg_attn_bwd", "seg_attn_bwd_noalloc", "seg_logprob_workspace_bytes", "seg_logprob_loss",
           "seg_layer_workspace_bytes", "seg_layer_fwd", "seg_layer_bwd", "seg_profile_enable",
           "seg_profile_reset", "seg_profile_read", "seg_last_error"]

P32 = ctypes.POINTER(ctypes.c_int32)
VP = ctypes.c_void_p


SEG_MODE_SLIDING, SEG_MODE_ANCHORED = 0, 1
SEG_WINDOW_ANCHORED = 1 << 28


class SegProblem(ctypes.Structure):
    _fields_ = [("num_traj", ctypes.c_int32), ("step_offsets", P32), ("prompt_len", P32),
                ("img_len", P32), ("text_len", P32), ("action_len", P32),
                ("window", ctypes.c_int32), ("seg_steps", ctypes.c_int32),
                ("max_seg_tokens", ctypes.c_int32), ("buffer_tokens", ctypes.c_int32),
                ("tile", ctypes.c_int32), ("mode", ctypes.c_int32)]


class SegSizes(ctypes.Structure):
    _fields_ = [("num_segments", ctypes.c_int32), ("num_buffers", ctypes.c_int32),
                ("loss_rows", ctypes.c_int32), ("num_qtiles", ctypes.c_int32),
                ("num_steps", ctypes.c_int32), ("max_seg_len", ctypes.c_int32),
                ("packed_tokens", ctypes.c_int64), ("traj_tokens", ctypes.c_int64),
                ("tile_nnz_max", ctypes.c_int64), ("workspace_bytes", ctypes.c_size_t)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


class SegLayout(ctypes.Structure):
    _fields_ = [("seg_info", VP), ("tok_src", VP), ("tok_meta", VP), ("loss_pred_row", VP),
                ("loss_tgt_src", VP), ("loss_traj", VP), ("tile_seg", VP), ("qt_ptr", VP),
                ("qt_col", VP), ("qt_cls", VP), ("qt_ord", VP), ("kt_ptr", VP), ("kt_row", VP),
                ("kt_cls", VP), ("kt_ord", VP),
                ("seg_pairs", VP), ("tile_nnz", VP),
                ("window", ctypes.c_int32), ("tile", ctypes.c_int32),
                ("xcd_rows", ctypes.c_int32 * 9), ("xcd_cols", ctypes.c_int32 * 9)]


class SegLossCfg(ctypes.Structure):
    _fields_ = [("eps_low", ctypes.c_float), ("eps_high", ctypes.c_float),
                ("dual_clip_c", ctypes.c_float), ("loss_scale", ctypes.c_float),
                ("logit_scale", ctypes.c_float), ("want_grad", ctypes.c_int32),
                ("kl_coef", ctypes.c_float)]


class SegLayerCfg(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("inter", ctypes.c_int32), ("hq", ctypes.c_int32),
                ("hkv", ctypes.c_int32), ("d", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("rope_base", ctypes.c_float), ("chunk_rows", ctypes.c_int32)]


LAYER_WEIGHTS = ("g1", "wq", "wk", "wv", "wo", "g2", "wg", "wu", "wd")


class SegLayerWeights(ctypes.Structure):
    _fields_ = [(n, VP) for n in LAYER_WEIGHTS]


class SegLayerSaved(ctypes.Structure):
    _fields_ = [("q", VP), ("k", VP), ("v", VP), ("o", VP), ("lse", VP), ("y1", VP),
                ("rstd1", VP), ("rstd2", VP)]


class SegLayerGrads(ctypes.Structure):
    _fields_ = [(n, VP) for n in LAYER_WEIGHTS]


class SegError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


_lib: Optional[ctypes.CDLL] = None


def lib() -> ctypes.CDLL:
    """The loaded libseg.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"libseg.so not found at {LIB_PATH}; build it first "
                               "(python -c 'import __graft_entry__; __graft_entry__.build()')")
        L = ctypes.CDLL(LIB_PATH)
        L.seg_last_error.restype = ctypes.c_char_p
        L.seg_last_error.argtypes = []
        L.seg_layout_query.restype = ctypes.c_int
        L.seg_layout_query.argtypes = [ctypes.POINTER(SegProblem), ctypes.POINTER(SegSizes)]
        L.seg_build_layout.restype = ctypes.c_int
        L.seg_build_layout.argtypes = [ctypes.POINTER(SegProblem), ctypes.POINTER(SegSizes),
                                       ctypes.POINTER(SegLayout), VP, ctypes.c_size_t, VP]
        L.seg_attn_workspace_bytes.restype = ctypes.c_size_t
        L.seg_attn_workspace_bytes.argtypes = [ctypes.POINTER(SegSizes), ctypes.c_int,
                                               ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                               ctypes.c_int32]
        L.seg_attn_fwd.restype = ctypes.c_int
        L.seg_attn_fwd.argtypes = [ctypes.POINTER(SegLayout), ctypes.POINTER(SegSizes), ctypes.c_int,
                                   ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_float,
                                   VP, VP, VP, VP, VP, VP, ctypes.c_size_t, VP]
        L.seg_attn_bwd.restype = ctypes.c_int
        L.seg_attn_bwd.argtypes = [ctypes.POINTER(SegLayout), ctypes.POINTER(SegSizes), ctypes.c_int,
                                   ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_float,
                                   VP, VP, VP, VP, VP, VP, VP, VP, VP, VP, ctypes.c_size_t, VP]
        L.seg_attn_bwd_noalloc.restype = ctypes.c_int
        L.seg_attn_bwd_noalloc.argtypes = [ctypes.POINTER(SegLayout), ctypes.POINTER(SegSizes),
                                           ctypes.c_int, ctypes.c_int32, ctypes.c_int32,
                                           ctypes.c_int32, ctypes.c_float,
                                           VP, VP, VP, VP, VP, VP, VP, VP, VP, VP]
        L.seg_logprob_workspace_bytes.restype = ctypes.c_size_t
        L.seg_logprob_workspace_bytes.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                                  ctypes.c_int]
        L.seg_logprob_loss.restype = ctypes.c_int
        # rows, hidden, vocab, dt, h, row_index, w, target, old_logp, ref_logp, adv,
        # row_traj, num_traj, cfg, logp, loss_tok, clipped, kl_tok, loss_sum, dh, dw, ws,
        # ws_bytes, stream
        L.seg_logprob_loss.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int,
                                       VP, VP, VP, VP, VP, VP, VP, VP, ctypes.c_int32,
                                       ctypes.POINTER(SegLossCfg), VP, VP, VP, VP, VP, VP, VP, VP,
                                       ctypes.c_size_t, VP]
        L.seg_layer_workspace_bytes.restype = ctypes.c_size_t
        L.seg_layer_workspace_bytes.argtypes = [ctypes.POINTER(SegSizes), ctypes.POINTER(SegLayerCfg),
                                                ctypes.c_int32]
        L.seg_layer_fwd.restype = ctypes.c_int
        L.seg_layer_fwd.argtypes = [ctypes.POINTER(SegLayout), ctypes.POINTER(SegSizes),
                                    ctypes.POINTER(SegLayerCfg), ctypes.POINTER(SegLayerWeights),
                                    VP, VP, ctypes.POINTER(SegLayerSaved), VP, ctypes.c_size_t, VP]
        L.seg_layer_bwd.restype = ctypes.c_int
        L.seg_layer_bwd.argtypes = [ctypes.POINTER(SegLayout), ctypes.POINTER(SegSizes),
                                    ctypes.POINTER(SegLayerCfg), ctypes.POINTER(SegLayerWeights),
                                    VP, ctypes.POINTER(SegLayerSaved), VP, VP,
                                    ctypes.POINTER(SegLayerGrads), VP, ctypes.c_size_t, VP]
        L.seg_profile_enable.restype = None
        L.seg_profile_enable.argtypes = [ctypes.c_int32]
        L.seg_profile_reset.restype = None
        L.seg_profile_reset.argtypes = []
        L.seg_profile_read.restype = ctypes.c_int
        L.seg_profile_read.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(ctypes.c_int64)]
        _lib = L
    return _lib


def check(status: int) -> None:
    if status != SEG_OK:
        raise SegError(status, lib().seg_last_error().decode(errors="replace"))
