"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
and prepare the oracle's view of the same seeded inputs."""
from __future__ import annotations

import math
import sys

import numpy as np

from paper_2607_11185_amd import seg as S
from paper_2607_11185_amd import workload as WL

TOL = 2e-2  # relative Frobenius error bound for bf16 results


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def rel(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30))


def as_model_dtype(vals: np.ndarray, cfg) -> np.ndarray:
    """The values the kernels compute on: bf16 (f32 inputs are rounded)."""
    if cfg.dtype == "bf16":
        return vals
    return WL.bf16_bits_to_f64(WL.bf16_round_np(vals.astype(np.float32)))


class GpuRun:
    """Layout + packed inputs of one workload on the GPU."""

    def __init__(self, cfg, spans=None, device="cuda", tile=128):
        import torch
        self.cfg = cfg
        self.inp = WL.Inputs(cfg, spans)
        self.spans = self.inp.spans
        self.dev = torch.device(device)
        self.problem = S.Problem.from_spans(self.spans, cfg.window, cfg.seg_steps,
                                            cfg.max_seg_tokens, cfg.buffer_tokens, tile, cfg.mode)
        self.lay = S.seg_build_layout(self.problem, device=self.dev)
        self.host = self.lay.host()
        self.P = self.lay.sizes.packed_tokens
        self.scale = 1.0 / math.sqrt(cfg.head_dim)

    def packed_inputs(self, with_dout=True):
        import torch
        src = torch.from_numpy(self.host["tok_src"].astype(np.int64)).to(self.dev)
        self.q = self.inp.q_torch(self.dev)[src].contiguous()
        self.k = self.inp.k_torch(self.dev)[src].contiguous()
        self.v = self.inp.v_torch(self.dev)[src].contiguous()
        if with_dout:
            self.dout = self.inp.dout_torch(self.P, self.dev)
        return self

    def fwd(self):
        self.o, self.lse = S.seg_attn_fwd(self.lay, self.q, self.k, self.v, self.scale)
        return self.o, self.lse

    def bwd(self):
        self.dq, self.dk, self.dv = S.seg_attn_bwd(self.lay, self.q, self.k, self.v, self.o,
                                                   self.lse, self.dout, self.scale)
        return self.dq, self.dk, self.dv

    # oracle-side values of one segment (from the same generator)
    def seg_np(self, sg):
        c = self.cfg
        q = as_model_dtype(self.inp.q_np(sg.canon), c)
        k = as_model_dtype(self.inp.k_np(sg.canon), c)
        v = as_model_dtype(self.inp.v_np(sg.canon), c)
        dout = as_model_dtype(self.inp.dout_np(np.arange(sg.start, sg.start + sg.length)), c)
        return q, k, v, dout


def vis_window(cfg):
    """Window argument of the oracle's visibility for a workload (None: the
    anchored mode's causal visibility)."""
    return None if cfg.mode == "anchored" else cfg.window
