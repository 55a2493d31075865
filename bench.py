#!/usr/bin/env python3
"""Benchmark of the segmented training hot path on one MI355X.

One step = the whole hot path over one batch: segmentation and packed layout
with its tile map (seg_layout_query + seg_build_layout), masked GQA attention
forward, the fused action-token log-prob / clipped-ratio loss with its KL
penalty (lambda = 1e-4) and gradients, and attention backward.  The reference
/ old-policy forward pass (attention forward + forward-only log-prob) is timed
separately for both decompositions (reference_forward_ms).  Inputs (packed q/k/v/dO, hidden states,
projection, targets, advantages, rollout log-probs) are resident in HBM before
the timed region.  The step-wise decomposition (every turn its own sample,
same kernels) runs the same step for the comparison.

Prints one JSON line.  `value` is the algorithmic attention forward+backward
throughput (12*d FLOP per visible (query, key) pair per query head) over the
device time of the two attention calls (the FlashAttention convention, 14*d
with a 10*d backward that counts the recompute of S, is reported alongside as
attn_tflops_fa_convention); `ms_per_step` and the trajectory token rates cover
the whole step.  roofline.traffic is the counter-measured HBM bytes of one
launch of the dominant kernel (see MEASURED_TRAFFIC).  For the 7B-class
workloads the line also carries `layer`: the training step of one full
decoder layer around the attention (2 timed steps), segmented and step-wise
(`--no-layer` skips it; `--layer` runs it alone with its own options).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "segmented attn fwd+bwd TFLOP/s + trajectory tokens/sec vs step-wise (1 GPU)"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
# algorithmic FLOP per visible pair per query head and per head-dim element
KERNEL_FLOP_PER_PAIR_D = {"attn_fwd": 4, "attn_bwd_dkdv": 6, "attn_bwd_dq": 2}
# HBM bytes per launch of the attention kernels on the 7b workload: rocprofv3
# --pmc FETCH_SIZE and WRITE_SIZE passes over `bench.py --pmc-driver`, each
# scaled by what the same counter reads for the f32->bf16 streaming kernel
# over a known byte count (reads x2.000, writes x1.000).  They describe the
# kernel source they were taken on and are reported only while it is unchanged.
MEASURED_TRAFFIC = {
    "source": "paper_2607_11185_amd/csrc/seg_attn.hip",
    "source_sha256": "9faee5ad671f57e9c720eb8e180fc0dd0f545fc900f2a9e9f8cabf0507596382",
    "config": "7b",
    "bytes_per_launch": {"attn_bwd_dkdv": 315.29e9, "attn_fwd": 72.77e9,
                         "attn_bwd_dq": 99.34e9},
}
KL_COEF = 1e-4  # the paper's KL penalty lambda (hyperparameter table)
KERNELS = ["layout", "attn_prep", "attn_fwd", "attn_delta", "attn_bwd_dkdv", "attn_bwd_dq",
           "lp_prep", "logits", "row_loss", "dz", "dh", "dw"]


def measured_traffic(cfg_name, kernel):
    """Counter-derived HBM bytes of `kernel` for this workload, or None when the
    kernel source has changed since the counters were taken."""
    import hashlib
    m = MEASURED_TRAFFIC
    if cfg_name != m["config"] or kernel not in m["bytes_per_launch"]:
        return None
    try:
        with open(os.path.join(ROOT, m["source"]), "rb") as f:
            digest = hashlib.sha256(f.read()).hexdigest()
    except OSError:
        return None
    return m["bytes_per_launch"][kernel] if digest == m["source_sha256"] else None


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class PathRun:
    """All device buffers of one path (segmented or step-wise) and its step."""

    def __init__(self, cfg, dev, spans=None, quick_inputs=False):
        """quick_inputs: draw q, k, v, dO, hidden states and the projection
        with torch.randn (a handful of large launches; for counter passes,
        which serialise every launch) instead of the workload generator."""
        import numpy as np
        import torch

        from paper_2607_11185_amd import seg as S
        from paper_2607_11185_amd import workload as WL
        self.S, self.cfg, self.dev = S, cfg, dev
        inp = WL.Inputs(cfg, spans)
        self.problem = S.Problem.from_spans(inp.spans, cfg.window, cfg.seg_steps,
                                            cfg.max_seg_tokens, cfg.buffer_tokens, 128, cfg.mode)
        self.sizes = S.seg_layout_query(self.problem)
        self.lay = S.seg_build_layout(self.problem, self.sizes, dev)
        host = self.lay.host()
        self.pairs = int(host["seg_pairs"].sum())
        sz = self.sizes
        P, R = sz.packed_tokens, sz.loss_rows
        log(f"[{cfg.name}] segments={sz.num_segments} packed={P} traj_tokens={sz.traj_tokens} "
            f"loss_rows={R} tiles={sz.num_qtiles} nnz={int(host['tile_nnz'][0])} pairs/head={self.pairs}")
        src = torch.from_numpy(host["tok_src"].astype(np.int64)).to(dev)
        if quick_inputs:
            g = torch.Generator(device=dev)
            g.manual_seed(cfg.seed)

            def rn(*shape, std=1.0):
                return (torch.randn(*shape, generator=g, device=dev, dtype=torch.float32)
                        * std).to(torch.bfloat16)
            hd = cfg.head_dim
            self.q, self.k, self.v = rn(P, cfg.hq, hd), rn(P, cfg.hkv, hd), rn(P, cfg.hkv, hd)
            self.dout, self.h = rn(P, cfg.hq, hd), rn(P, cfg.hidden)
            self.w = rn(cfg.vocab, cfg.hidden, std=cfg.w_std)
        else:
            self.q = inp.q_torch(dev)[src].contiguous()
            self.k = inp.k_torch(dev)[src].contiguous()
            self.v = inp.v_torch(dev)[src].contiguous()
            torch.cuda.empty_cache()
            log(f"  [{cfg.name}] q, k, v ready")
            self.dout = inp.dout_torch(P, dev)
            self.h = inp.h_torch(dev)[src].contiguous()
            torch.cuda.empty_cache()
            self.w = inp.w_torch(dev)
        log(f"  [{cfg.name}] inputs ready")
        self.tgt = torch.from_numpy(inp.tgt_np(host["loss_tgt_src"])).to(dev)
        self.adv = torch.from_numpy(inp.adv_np().astype(np.float32)).to(dev)
        self.scale = 1.0 / math.sqrt(cfg.head_dim)
        dt = 0
        self.ws_fwd = S.attn_workspace(self.lay, dt, cfg.hq, cfg.hkv, cfg.head_dim, False)
        self.ws_bwd = S.attn_workspace(self.lay, dt, cfg.hq, cfg.hkv, cfg.head_dim, True)
        self.ws_lp = S.logprob_workspace(R, cfg.hidden, cfg.vocab, dt, dev)
        self.o = torch.empty_like(self.q)
        self.lse = torch.empty((cfg.hq, P), dtype=torch.float32, device=dev)
        self.dq = torch.empty_like(self.q)
        self.dk = torch.empty_like(self.k)
        self.dv = torch.empty_like(self.v)
        self.lp_out = {
            "logp": torch.empty(R, dtype=torch.float32, device=dev),
            "loss_tok": torch.empty(R, dtype=torch.float32, device=dev),
            "clipped": torch.empty(R, dtype=torch.uint8, device=dev),
            "kl_tok": torch.empty(R, dtype=torch.float32, device=dev),
            "loss_sum": torch.empty(1, dtype=torch.float32, device=dev),
            "dh": torch.empty((R, cfg.hidden), dtype=torch.bfloat16, device=dev),
            "dw": torch.empty((cfg.vocab, cfg.hidden), dtype=torch.float32, device=dev),
        }
        # rollout log-probs: the current policy's log-probs (one forward-only
        # call before timing) plus N(0, 0.1) noise, as the workload specifies
        fwd_only = S.LossCfg(cfg.eps_low, cfg.eps_high, cfg.dual_clip, 1.0 / R, 1.0, False)
        zero = torch.zeros(R, dtype=torch.float32, device=dev)
        S.seg_logprob_loss(self.h, self.lay.loss_pred_row, self.w, self.tgt, zero, self.adv,
                           self.lay.loss_traj, fwd_only,
                           out=dict(self.lp_out, dh=None, dw=None, kl_tok=None), ws=self.ws_lp)
        noise = torch.from_numpy(inp.old_noise_np(host["loss_tgt_src"]).astype(np.float32)).to(dev)
        self.old = (self.lp_out["logp"] + noise).contiguous()
        # reference-policy log-probs: the current ones minus the same noise
        self.ref = (self.lp_out["logp"] - noise).contiguous()
        self.loss_cfg = S.LossCfg(cfg.eps_low, cfg.eps_high, cfg.dual_clip, 1.0 / R, 1.0, True,
                                  KL_COEF)
        self.ref_cfg = fwd_only
        self.ref_out = dict(self.lp_out, dh=None, dw=None, kl_tok=None)
        torch.cuda.synchronize()

    def step(self, ev=None):
        S = self.S
        rec = (lambda name: ev[name].record()) if ev is not None else (lambda name: None)
        rec("t0")
        sz = S.seg_layout_query(self.problem)
        S.seg_build_layout(self.problem, sz, self.dev, out=self.lay)
        rec("t1")
        S.seg_attn_fwd(self.lay, self.q, self.k, self.v, self.scale, o=self.o, lse=self.lse,
                       ws=self.ws_fwd)
        rec("t2")
        S.seg_logprob_loss(self.h, self.lay.loss_pred_row, self.w, self.tgt, self.old, self.adv,
                           self.lay.loss_traj, self.loss_cfg, out=self.lp_out, ws=self.ws_lp,
                           ref_logp=self.ref)
        rec("t3")
        S.seg_attn_bwd(self.lay, self.q, self.k, self.v, self.o, self.lse, self.dout, self.scale,
                       dq=self.dq, dk=self.dk, dv=self.dv, ws=self.ws_bwd)
        rec("t4")

    def ref_forward(self, ev=None):
        """The reference / old-policy pass: attention forward and the
        forward-only log-prob of the action rows (no gradients)."""
        S = self.S
        rec = (lambda name: ev[name].record()) if ev is not None else (lambda name: None)
        rec("r0")
        S.seg_attn_fwd(self.lay, self.q, self.k, self.v, self.scale, o=self.o, lse=self.lse,
                       ws=self.ws_fwd)
        rec("r1")
        S.seg_logprob_loss(self.h, self.lay.loss_pred_row, self.w, self.tgt, self.old, self.adv,
                           self.lay.loss_traj, self.ref_cfg, out=self.ref_out, ws=self.ws_lp)
        rec("r2")

    def attn_flop(self):
        c = self.cfg
        return 12.0 * c.head_dim * self.pairs * c.hq

    def free(self):
        for k in list(self.__dict__):
            if k not in ("cfg", "sizes", "pairs", "S", "dev", "problem"):
                delattr(self, k)


def time_path(run, steps, warmup, profile=True):
    import torch

    from paper_2607_11185_amd import _lib
    L = _lib.lib()
    for _ in range(warmup):
        run.step()
    torch.cuda.synchronize()
    names = ["t0", "t1", "t2", "t3", "t4"]
    evs = [{n: torch.cuda.Event(enable_timing=True) for n in names} for _ in range(steps)]
    L.seg_profile_reset()
    L.seg_profile_enable(1 if profile else 0)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for i in range(steps):
        run.step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    L.seg_profile_enable(0)
    ph = {"layout": 0.0, "attn_fwd": 0.0, "logprob_loss": 0.0, "attn_bwd": 0.0, "step": 0.0}
    for e in evs:
        ph["layout"] += e["t0"].elapsed_time(e["t1"])
        ph["attn_fwd"] += e["t1"].elapsed_time(e["t2"])
        ph["logprob_loss"] += e["t2"].elapsed_time(e["t3"])
        ph["attn_bwd"] += e["t3"].elapsed_time(e["t4"])
        ph["step"] += e["t0"].elapsed_time(e["t4"])
    ph = {k: v / steps for k, v in ph.items()}
    per_step = sorted(e["t0"].elapsed_time(e["t4"]) for e in evs)
    ph["step_median"] = per_step[len(per_step) // 2]
    kern = {}
    import ctypes
    for name in KERNELS:
        tot = ctypes.c_double()
        n = ctypes.c_int64()
        _lib.check(L.seg_profile_read(name.encode(), ctypes.byref(tot), ctypes.byref(n)))
        if n.value:
            kern[name] = {"ms_per_step": tot.value / steps, "launches_per_step": n.value / steps}
    L.seg_profile_reset()
    return ph, kern, wall / steps * 1e3


# packed rows per trajectory group: about 40 KB of device memory per packed
# row (q, o, dq, dO, hidden states, k, v and their gradients, per-row fp32)
GROUP_ROWS = 4_500_000


def traj_groups(cfg, max_rows=GROUP_ROWS):
    """Consecutive trajectory ranges of the workload whose packed rows stay
    within max_rows each (a range holds at least one trajectory)."""
    from paper_2607_11185_amd import seg as S
    from paper_2607_11185_amd import workload as WL
    spans = WL.make_spans(cfg)
    groups, t0 = [], 0
    while t0 < spans.num_traj:
        t1 = t0 + 1
        while t1 < spans.num_traj:
            sub = spans.subset(t0, t1 + 1)
            pr = S.Problem.from_spans(sub, cfg.window, cfg.seg_steps, cfg.max_seg_tokens,
                                      cfg.buffer_tokens, 128, cfg.mode)
            if S.seg_layout_query(pr).packed_tokens > max_rows:
                break
            t1 += 1
        groups.append(spans.subset(t0, t1))
        t0 = t1
    return groups


def time_groups(cfg, dev, steps, warmup):
    """time_path and time_ref over the workload's trajectory groups, one
    group resident at a time; per-step times add up over the groups."""
    import torch
    groups = traj_groups(cfg)
    ph, kern, wall, ref, tot = {}, {}, 0.0, {}, {"pairs": 0, "packed": 0, "segments": 0,
                                                  "traj_tokens": 0, "flop": 0.0, "loss_rows": 0}
    for gi, sub in enumerate(groups):
        run = PathRun(cfg, dev, sub if len(groups) > 1 else None)
        if len(groups) > 1:
            log(f"  group {gi + 1}/{len(groups)}: {sub.num_traj} trajectories")
        p, k, w = time_path(run, steps, warmup)
        r = time_ref(run, steps, warmup)
        for n, v in p.items():
            ph[n] = ph.get(n, 0.0) + v
        for n, v in k.items():
            a = kern.setdefault(n, {"ms_per_step": 0.0, "launches_per_step": 0.0})
            a["ms_per_step"] += v["ms_per_step"]
            a["launches_per_step"] += v["launches_per_step"]
        for n, v in r.items():
            ref[n] = round(ref.get(n, 0.0) + v, 3)
        wall += w
        tot["pairs"] += run.pairs
        tot["packed"] += run.sizes.packed_tokens
        tot["segments"] += run.sizes.num_segments
        tot["traj_tokens"] += run.sizes.traj_tokens
        tot["loss_rows"] += run.sizes.loss_rows
        tot["flop"] += run.attn_flop()
        run.free()
        del run
        torch.cuda.empty_cache()
    tot["groups"] = len(groups)
    return ph, kern, wall, ref, tot


def time_ref(run, steps, warmup):
    """Mean device ms of the reference forward pass (attention, log-prob)."""
    import torch
    for _ in range(warmup):
        run.ref_forward()
    torch.cuda.synchronize()
    evs = [{n: torch.cuda.Event(enable_timing=True) for n in ("r0", "r1", "r2")}
           for _ in range(steps)]
    for i in range(steps):
        run.ref_forward(evs[i])
    torch.cuda.synchronize()
    att = sum(e["r0"].elapsed_time(e["r1"]) for e in evs) / steps
    lp = sum(e["r1"].elapsed_time(e["r2"]) for e in evs) / steps
    return {"attn_fwd": round(att, 3), "logprob": round(lp, 3), "total": round(att + lp, 3)}


def cpu_baseline(cfg):
    """The float64 oracle on a bounded sample (about 10-15 s on 16 threads):
    attention forward and backward of the first segment for up to four query
    heads of one kv head (every segment and head for the tiny workload), and
    the log-prob loss with its gradients for 16 action rows at the full
    vocabulary.  The oracle's rates, extrapolated by the FLOP counts of the
    whole step, give its trajectory tokens/s (labelled as extrapolated)."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import attention as OA
    from oracle import layout as OL
    from oracle import loss as OLS
    from paper_2607_11185_amd import workload as WL
    inp = WL.Inputs(cfg)
    ref = OL.build(inp.spans, cfg.window, cfg.seg_steps, 128, cfg.max_seg_tokens,
                   cfg.buffer_tokens, with_tiles=False, mode=cfg.mode)
    full = cfg.name == "tiny"
    segs = ref.segments if full else ref.segments[:1]
    if not full and segs[0].length > 16384:
        # a prefix of the segment is an attention problem of its own (rows see
        # no key after them): the first 16,384 tokens
        import dataclasses
        sg0 = segs[0]
        segs = [dataclasses.replace(sg0, canon=sg0.canon[:16384], kind=sg0.kind[:16384],
                                    step=sg0.step[:16384])]
    nh = cfg.hq if full else min(4, cfg.hq // cfg.hkv)  # query heads of kv head 0
    nkv = cfg.hkv if full else 1
    win = None if cfg.mode == "anchored" else cfg.window
    scale = 1.0 / math.sqrt(cfg.head_dim)
    t_attn, pairs_done, toks = 0.0, 0, 0
    for sg in segs:
        q = inp.q_np(sg.canon)[:, :nh]
        k = inp.k_np(sg.canon)[:, :nkv]
        v = inp.v_np(sg.canon)[:, :nkv]
        dout = inp.dout_np(np.arange(sg.start, sg.start + sg.length))[:, :nh]
        t0 = time.perf_counter()
        mask = OL.visibility(sg, win)
        OA.forward(q, k, v, mask, scale)
        OA.backward(q, k, v, mask, scale, dout)
        t_attn += time.perf_counter() - t0
        pairs_done += int(mask.sum())
        toks += sg.length
    attn_rate = 12.0 * cfg.head_dim * pairs_done * nh / t_attn
    # log-prob sample: the first rows of the batch's loss rows
    n_rows = min(16, len(ref.loss_pred_row))
    sel = np.arange(n_rows)
    h = inp.h_np(ref.tok_src[ref.loss_pred_row[sel]])
    w = inp.w_np()
    tgt = inp.tgt_np(ref.loss_tgt_src[sel])
    adv = inp.adv_np()[ref.loss_traj[sel]]
    t0 = time.perf_counter()
    lp, _, _ = OLS.logprob(h, w, tgt)
    OLS.loss_and_grads(h, w, tgt, lp + 0.1, adv, cfg.eps_low, cfg.eps_high,
                       loss_scale=1.0 / max(n_rows, 1))
    t_lp = time.perf_counter() - t0
    lp_rate = 8.0 * cfg.vocab * cfg.hidden * n_rows / t_lp  # logits twice (logp + loss), dH, dW
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    out = {"value": attn_rate / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
           "sample": (f"attention fwd+bwd of {'every segment' if full else 'segment 0'} "
                      f"({toks} tokens{', a prefix' if segs[0].length < ref.segments[0].length else ''}, "
                      f"{pairs_done} visible pairs per head), {nh} query heads / "
                      f"{nkv} kv head, d={cfg.head_dim}, {t_attn:.1f} s; log-prob loss with "
                      f"gradients of {n_rows} action rows at vocab {cfg.vocab}, hidden "
                      f"{cfg.hidden}, {t_lp:.1f} s; float64 NumPy"),
           "seconds": round(t_attn + t_lp, 2)}
    return out, attn_rate, lp_rate


def pmc_driver(cfg_name):
    """One launch of the f32->bf16 conversion kernel over a known number of
    bytes (the plain streaming kernel that calibrates the HBM byte counters),
    then one step on the workload: every kernel of the path (the layout
    build, attention forward, Delta, dK/dV, dQ, and the fused log-prob loss
    with its gradients) runs last, so the last dispatch of each kernel name
    (the last two of the transposed-operand GEMM: dH, then dW) is the step's.
    The layout and the loss targets come from the workload; q, k, v, dO,
    hidden states and the projection are drawn with torch.randn (a few large
    launches, left out of the counter tables by name).  Prints one JSON line
    with the sizes."""
    import numpy as np
    import torch

    from paper_2607_11185_amd import seg as S
    from paper_2607_11185_amd import workload as WL
    dev = torch.device("cuda:0")
    # calibration: 4096 one-turn samples of 256 tokens, 8 heads, d = 128, f32
    # inputs; the forward converts q, k and v with one streaming kernel each
    n_s, hc, d = 4096, 8, 128
    sp = WL.explicit_spans([1] * n_s, [236] * n_s, [0] * n_s, [20] * n_s, [4] * n_s)
    cal = S.seg_build_layout(S.Problem.from_spans(sp, 1, 1), device=dev)
    Pc = cal.sizes.packed_tokens
    zeros = np.zeros((Pc, hc, d), np.float32)
    qc = torch.from_numpy(zeros).to(dev)
    kc = torch.from_numpy(zeros).to(dev)
    vc = torch.from_numpy(zeros).to(dev)
    torch.cuda.synchronize()
    S.seg_attn_fwd(cal, qc, kc, vc, 1.0 / math.sqrt(d))
    torch.cuda.synchronize()
    n = Pc * hc * d
    del qc, kc, vc, cal
    torch.cuda.empty_cache()
    cfg = WL.CONFIGS[cfg_name]
    run = PathRun(cfg, dev, quick_inputs=True)
    torch.cuda.synchronize()
    log("inputs ready")
    run.step()
    torch.cuda.synchronize()
    log("step done")
    print(json.dumps({"config": cfg.name, "packed_tokens": run.sizes.packed_tokens,
                      "loss_rows": run.sizes.loss_rows, "visible_pairs_per_head": run.pairs,
                      "calibration": {"kernel": "k_f32_to_bf16", "elements": n,
                                      "read_bytes": 4 * n, "write_bytes": 2 * n,
                                      "launches": 3}}), flush=True)


LAYER_INTER = 18944   # MLP width of the 7B-class backbone (Qwen2-7B shape)
LAYER_GROUPS = 2      # trajectory groups (micro-batches) per layer step
LAYER_SCOPES = ["layout", "ly_norm", "ly_rope", "ly_proj", "ly_mlp", "ly_wgrad", "ly_misc",
                "attn_prep", "attn_fwd", "attn_delta", "attn_bwd_dkdv", "attn_bwd_dq"]


class LayerRun:
    """One decoder layer (projections, RoPE, segmented attention, SwiGLU MLP)
    over the batch, forward and backward, in trajectory groups: each group is
    packed and run on its own (a micro-batch), all groups' inputs resident."""

    def __init__(self, cfg, dev, inter, groups, chunk=0):
        import numpy as np
        import torch

        from paper_2607_11185_amd import seg as S
        from paper_2607_11185_amd import workload as WL
        self.S, self.cfg, self.dev = S, cfg, dev
        H, d = cfg.hidden, cfg.head_dim
        self.lc = S.LayerCfg(H, inter, cfg.hq, cfg.hkv, d, 1e-6, 1e6, chunk)
        spans = WL.make_spans(cfg)
        bounds = np.linspace(0, spans.num_traj, groups + 1).round().astype(int)
        self.w = WL.layer_weights_torch(cfg.seed, H, inter, cfg.hq, cfg.hkv, d, dev)
        n_canon = int(spans.canon_offsets()[-1])
        xc = WL.layer_rows_torch(cfg.seed, "x", n_canon, H, dev)
        coff = spans.canon_offsets()
        self.groups = []
        self.P = self.pairs = self.traj_tokens = 0
        for t0, t1 in zip(bounds[:-1], bounds[1:]):
            sub = spans.subset(int(t0), int(t1))
            prob = S.Problem.from_spans(sub, cfg.window, cfg.seg_steps, cfg.max_seg_tokens,
                                        cfg.buffer_tokens, 128, cfg.mode)
            sz = S.seg_layout_query(prob)
            lay = S.seg_build_layout(prob, sz, dev)
            host = lay.host()
            src = host["tok_src"].astype(np.int64)
            src = np.where(src >= 0, src + int(coff[t0]), 0)
            x = xc[torch.from_numpy(src).to(dev)].contiguous()
            P = sz.packed_tokens
            dy = WL.layer_rows_torch(cfg.seed + 1 + len(self.groups), "dy", P, H, dev)
            self.groups.append({"prob": prob, "lay": lay, "x": x, "dy": dy, "P": P})
            self.P += P
            self.pairs += int(host["seg_pairs"].sum())
            self.traj_tokens += sz.traj_tokens
        del xc
        torch.cuda.empty_cache()
        # outputs, saved activations and workspaces sized for the largest group
        big = max(self.groups, key=lambda g: g["P"])
        self.ws = S.layer_workspace(big["lay"], self.lc, True)
        self.y, self.saved = S.seg_layer_fwd(big["lay"], self.lc, self.w, big["x"], ws=self.ws)
        self.dx, self.grads = S.seg_layer_bwd(big["lay"], self.lc, self.w, big["x"], self.saved,
                                              big["dy"], ws=self.ws)
        torch.cuda.synchronize()
        log(f"[layer {cfg.name}] groups={len(self.groups)} packed={self.P} "
            f"(largest {big['P']}) pairs/head={self.pairs} inter={inter}")

    def _views(self, P):
        H, c = self.cfg.hidden, self.cfg
        sv = {"q": self.saved["q"][:P], "k": self.saved["k"][:P], "v": self.saved["v"][:P],
              "o": self.saved["o"][:P], "lse": self.saved["lse"].view(-1)[:c.hq * P].view(c.hq, P),
              "y1": self.saved["y1"][:P], "rstd1": self.saved["rstd1"][:P],
              "rstd2": self.saved["rstd2"][:P]}
        return self.y[:P], sv, self.dx[:P]

    def step(self, ev=None):
        S = self.S
        rec = (lambda name: ev[name].record()) if ev is not None else (lambda name: None)
        for gi, g in enumerate(self.groups):
            rec(f"l{gi}")
            sz = S.seg_layout_query(g["prob"])
            S.seg_build_layout(g["prob"], sz, self.dev, out=g["lay"])
            y, sv, dx = self._views(g["P"])
            rec(f"f{gi}")
            S.seg_layer_fwd(g["lay"], self.lc, self.w, g["x"], y=y, saved=sv, ws=self.ws)
            rec(f"b{gi}")
            S.seg_layer_bwd(g["lay"], self.lc, self.w, g["x"], sv, g["dy"], dx=dx, grads=self.grads,
                            ws=self.ws)
        rec("end")

    def gemm_flop(self):
        """Algorithmic GEMM FLOP of the step: forward projections and MLP, and
        twice that for the backward (data and weight gradients)."""
        c, I = self.cfg, self.lc.inter
        H, QD, KD = c.hidden, c.hq * c.head_dim, c.hkv * c.head_dim
        fwd = 2.0 * self.P * H * (QD + 2 * KD) + 2.0 * self.P * QD * H + 6.0 * self.P * H * I
        return 3.0 * fwd

    def attn_flop(self):
        c = self.cfg
        return 12.0 * c.head_dim * self.pairs * c.hq

    def free(self):
        for k in list(self.__dict__):
            if k not in ("cfg", "P", "pairs", "traj_tokens", "lc", "S", "dev"):
                delattr(self, k)


def time_layer(run, steps, warmup):
    import ctypes

    import torch

    from paper_2607_11185_amd import _lib
    L = _lib.lib()
    for _ in range(warmup):
        run.step()
    torch.cuda.synchronize()
    G = len(run.groups)
    names = [f"{p}{i}" for i in range(G) for p in "lfb"] + ["end"]
    evs = [{n: torch.cuda.Event(enable_timing=True) for n in names} for _ in range(steps)]
    L.seg_profile_reset()
    L.seg_profile_enable(1)
    torch.cuda.synchronize()
    for i in range(steps):
        run.step(evs[i])
    torch.cuda.synchronize()
    L.seg_profile_enable(0)
    ph = {"layout": 0.0, "fwd": 0.0, "bwd": 0.0, "step": 0.0}
    for e in evs:
        for i in range(G):
            nxt = e[f"l{i + 1}"] if i + 1 < G else e["end"]
            ph["layout"] += e[f"l{i}"].elapsed_time(e[f"f{i}"])
            ph["fwd"] += e[f"f{i}"].elapsed_time(e[f"b{i}"])
            ph["bwd"] += e[f"b{i}"].elapsed_time(nxt)
        ph["step"] += e["l0"].elapsed_time(e["end"])
    ph = {k: v / steps for k, v in ph.items()}
    scopes = {}
    for name in LAYER_SCOPES:
        tot = ctypes.c_double()
        n = ctypes.c_int64()
        _lib.check(L.seg_profile_read(name.encode(), ctypes.byref(tot), ctypes.byref(n)))
        if n.value:
            scopes[name] = round(tot.value / steps, 3)
    L.seg_profile_reset()
    return ph, scopes


def layer_bench(cfg, steps, warmup, inter, groups, stepwise=True, chunk=0):
    """Training step of one full decoder layer around the segmented attention
    (forward + backward, all weight gradients) over the batch, segmented and
    step-wise.  One JSON line (not the bench line)."""
    print(json.dumps(layer_result(cfg, steps, warmup, inter, groups, stepwise, chunk)), flush=True)


def layer_result(cfg, steps, warmup, inter, groups, stepwise=True, chunk=0):
    import torch
    dev = torch.device("cuda:0")
    res = {}
    cfgs = [("segmented", cfg)]
    if stepwise:
        cfgs.append(("stepwise", cfg.with_(name=cfg.name + "_stepwise", seg_steps=1,
                                           mode="sliding")))
    for label, c in cfgs:
        run = LayerRun(c, dev, inter, groups, chunk)
        ph, scopes = time_layer(run, steps, warmup)
        gemm_ms = sum(scopes.get(n, 0.0) for n in ("ly_proj", "ly_mlp", "ly_wgrad"))
        attn_ms = sum(scopes.get(n, 0.0) for n in ("attn_prep", "attn_fwd", "attn_delta",
                                                    "attn_bwd_dkdv", "attn_bwd_dq"))
        flop = run.gemm_flop() + run.attn_flop()
        res[label] = {
            "packed_tokens": run.P, "visible_pairs_per_head": run.pairs,
            "ms_per_step": round(ph["step"], 3),
            "traj_tokens_per_s": round(run.traj_tokens / (ph["step"] * 1e-3), 1),
            "layer_tflops": round(flop / ((ph["fwd"] + ph["bwd"]) * 1e-3) / 1e12, 2),
            "gemm_tflops": round(run.gemm_flop() / (gemm_ms * 1e-3) / 1e12, 2) if gemm_ms else None,
            "attn_tflops": round(run.attn_flop() / (attn_ms * 1e-3) / 1e12, 2) if attn_ms else None,
            "phases_ms": {k: round(v, 3) for k, v in ph.items()},
            "scopes_ms": scopes,
        }
        log(f"  {label}: {res[label]}")
        run.free()
        del run
        torch.cuda.empty_cache()
    out = {"layer": f"{cfg.name}: hidden {cfg.hidden}, MLP {inter}, {cfg.hq}q/{cfg.hkv}kv heads, "
                    f"d={cfg.head_dim}, RMSNorm + RoPE + SwiGLU, {groups} trajectory groups",
           "steps": steps, "warmup": warmup, "dtype": "bf16", **res}
    if stepwise:
        out["speedup_vs_stepwise"] = round(res["stepwise"]["ms_per_step"] /
                                           res["segmented"]["ms_per_step"], 3)
    return out


SWEEP_K = (1, 3, 5, 8, 10, 15)


def sweep(cfg, steps, warmup):
    """Kernel-level half of the paper's window sweep: W = L = K (sliding) or
    K = delta (anchored) over the same batch; per K the segmented step, the
    reference forward pass and the training-item and visible-pair counts.
    One JSON line."""
    import torch
    dev = torch.device("cuda:0")
    rows = []
    for K in SWEEP_K:
        c = cfg.with_(name=f"{cfg.name}_K{K}", window=K, seg_steps=K)
        run = PathRun(c, dev)
        ph, kern, _ = time_path(run, steps, warmup, profile=False)
        ref = time_ref(run, steps, warmup)
        attn = ph["attn_fwd"] + ph["attn_bwd"]
        rows.append({"K": K, "segments": run.sizes.num_segments,
                     "packed_tokens": run.sizes.packed_tokens,
                     "visible_pairs_per_head": run.pairs,
                     "step_ms": round(ph["step"], 3), "attn_ms": round(attn, 3),
                     "attn_tflops": round(run.attn_flop() / (attn * 1e-3) / 1e12, 2),
                     "traj_tokens_per_s": round(run.sizes.traj_tokens / (ph["step"] * 1e-3), 1),
                     "reference_forward_ms": ref["total"]})
        log(f"  K={K}: {rows[-1]}")
        run.free()
        del run
        torch.cuda.empty_cache()
    label = "K = delta" if cfg.mode == "anchored" else "W = L = K"
    print(json.dumps({"sweep": label, "workload": cfg.name, "steps": steps,
                      "warmup": warmup, "rows": rows}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="7b", help="workload name (7b, 7b_anchored, 7b_tp4_rank, small, long, tiny)")
    ap.add_argument("--no-stepwise", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sweep", action="store_true",
                    help="W = L = K sweep over K in (1, 3, 5, 8, 10, 15) on the workload "
                         "(one JSON line; not the bench line)")
    ap.add_argument("--pmc-driver", action="store_true",
                    help="one launch of each kernel of the step plus a calibration copy, for "
                         "rocprofv3 --pmc counter passes (no timing, no JSON bench line)")
    ap.add_argument("--layer", action="store_true",
                    help="training step of one full decoder layer (projections, RoPE, segmented "
                         "attention, SwiGLU MLP) segmented vs step-wise (one JSON line; not the "
                         "bench line)")
    ap.add_argument("--no-layer", action="store_true",
                    help="skip the decoder-layer measurement reported beside the bench line")
    ap.add_argument("--layer-inter", type=int, default=LAYER_INTER)
    ap.add_argument("--layer-groups", type=int, default=LAYER_GROUPS)
    ap.add_argument("--layer-chunk", type=int, default=0,
                    help="rows per projection / MLP chunk (0: the library default, 65536)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the segmented path runs on a single MI355X and this "
              "library has no multi-GPU code (run with --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2607_11185_amd import workload as WL
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.pmc_driver:
        pmc_driver(args.config)
        return
    if args.layer:
        layer_bench(WL.CONFIGS[args.config], args.steps, args.warmup, args.layer_inter,
                    args.layer_groups, not args.no_stepwise, args.layer_chunk)
        return
    if args.sweep:
        sweep(WL.CONFIGS[args.config], args.steps, args.warmup)
        return
    dev = torch.device("cuda:0")
    cfg = WL.CONFIGS[args.config]

    ph, kern, wall_ms, ref_seg, tot = time_groups(cfg, dev, args.steps, args.warmup)
    attn_ms = ph["attn_fwd"] + ph["attn_bwd"]
    value = tot["flop"] / (attn_ms * 1e-3) / 1e12
    traj_tokens = tot["traj_tokens"]
    # dominant attention kernel and its roofline from the live event timing
    dom = max(KERNEL_FLOP_PER_PAIR_D, key=lambda n: kern.get(n, {}).get("ms_per_step", 0.0))
    launches = kern[dom]["launches_per_step"]
    dom_ms = kern[dom]["ms_per_step"] / launches
    dom_flop = KERNEL_FLOP_PER_PAIR_D[dom] * cfg.head_dim * tot["pairs"] * cfg.hq / launches
    achieved = dom_flop / (dom_ms * 1e-3) / 1e12
    cut = (f"anchored K={cfg.window} delta={cfg.seg_steps}" if cfg.mode == "anchored"
           else f"W={cfg.window}, L={cfg.seg_steps}")
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ph["step"], 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded counter-based generator; no datasets or weights)",
        "config": {"workload": f"{cfg.name}-class segmented VCS step: {cfg.num_traj} trajectories "
                               f"x {cfg.steps[0]}-{cfg.steps[1]} turns, prompt {cfg.prompt_len}, "
                               f"{cfg.img_len} screenshot tokens, text {cfg.text_len[0]}-"
                               f"{cfg.text_len[1]} (last {cfg.action_len} trained), {cut}, "
                               f"{cfg.hq}q/{cfg.hkv}kv heads, d={cfg.head_dim}, "
                               f"hidden {cfg.hidden}, vocab {cfg.vocab}, clip {cfg.eps_low}/"
                               f"{cfg.eps_high}" + (f" cap {cfg.dual_clip}" if cfg.dual_clip else "")
                               + (f", {cfg.buffer_tokens}-token buffers" if cfg.buffer_tokens else ""),
                   "packed_tokens": tot["packed"], "traj_tokens": traj_tokens,
                   "segments": tot["segments"], "visible_pairs_per_head": tot["pairs"],
                   "loss_rows": tot["loss_rows"]},
        "traj_tokens_per_s": round(traj_tokens / (ph["step"] * 1e-3), 1),
        "attn_ms": round(attn_ms, 3),
        "attn_tflops_fa_convention": round(tot["flop"] * 14.0 / 12.0 / (attn_ms * 1e-3) / 1e12, 2),
        "phases_ms": {k: round(v, 3) for k, v in ph.items()},
        "kernels_ms": {k: round(v["ms_per_step"], 3) for k, v in kern.items()},
        "wall_ms_per_step": round(wall_ms, 3),
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic(cfg.name, dom),
                     "flop_per_launch": dom_flop, "ms_per_launch": round(dom_ms, 3)},
        "kl_coef": KL_COEF,
        "reference_forward_ms": ref_seg,
    }
    if tot["groups"] > 1:
        out["config"]["trajectory_groups"] = tot["groups"]

    if not args.no_stepwise:
        # step-wise decomposition: one item per turn holding its K (or W)
        # most recent screenshots; trajectory groups when it does not fit
        sw_cfg = cfg.with_(name=cfg.name + "_stepwise", seg_steps=1, mode="sliding")
        ph2, kern2, _, ref_sw, tot2 = time_groups(sw_cfg, dev, args.steps, args.warmup)
        attn2 = ph2["attn_fwd"] + ph2["attn_bwd"]
        out["stepwise"] = {
            "ms_per_step": round(ph2["step"], 3),
            "traj_tokens_per_s": round(traj_tokens / (ph2["step"] * 1e-3), 1),
            "attn_tflops": round(tot2["flop"] / (attn2 * 1e-3) / 1e12, 2),
            "attn_ms": round(attn2, 3), "packed_tokens": tot2["packed"],
            "segments": tot2["segments"], "visible_pairs_per_head": tot2["pairs"],
            "phases_ms": {k: round(v, 3) for k, v in ph2.items()},
        }
        if tot2["groups"] > 1:
            out["stepwise"]["trajectory_groups"] = tot2["groups"]
        out["speedup_vs_stepwise"] = round(ph2["step"] / ph["step"], 3)
        out["stepwise"]["reference_forward_ms"] = ref_sw
        out["reference_forward_speedup_vs_stepwise"] = round(ref_sw["total"] / ref_seg["total"], 3)

    if not args.no_layer and cfg.name in ("7b", "7b_anchored"):
        # one decoder layer around the attention (the next row past the hot
        # path), segmented vs step-wise, reported beside the bench numbers
        try:
            lr = layer_result(cfg, 2, 1, LAYER_INTER, LAYER_GROUPS, not args.no_stepwise)
            out["layer"] = {k: lr[k] for k in ("layer", "steps", "warmup", "speedup_vs_stepwise")
                            if k in lr}
            for k in ("segmented", "stepwise"):
                if k in lr:
                    out["layer"][k] = {n: lr[k][n] for n in ("packed_tokens", "ms_per_step",
                                                             "traj_tokens_per_s", "layer_tflops",
                                                             "gemm_tflops")}
        except Exception as e:  # the bench line is reported either way
            out["layer"] = {"error": f"{type(e).__name__}: {e}"}
        torch.cuda.empty_cache()

    if not args.no_cpu_baseline:
        cb, attn_rate, lp_rate = cpu_baseline(cfg)
        # the oracle's step time for the whole batch at the sampled rates
        # (extrapolated by FLOP counts; not a measurement of the whole batch)
        R = out["config"]["loss_rows"]
        t_or = tot["flop"] / attn_rate + 6.0 * cfg.vocab * cfg.hidden * R / lp_rate
        cb["gpu_over_oracle_attn"] = round(value * 1e12 / attn_rate, 1)
        cb["traj_tokens_per_s_extrapolated"] = round(traj_tokens / t_or, 3)
        cb["step_seconds_extrapolated"] = round(t_or, 1)
        out["cpu_baseline"] = cb
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
