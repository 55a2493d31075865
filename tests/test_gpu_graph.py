"""The compute entry points (attention forward / backward, fused log-prob
loss, decoder layer) captured in one HIP graph and replayed: every replay,
with other GPU work and synchronisations in between, reproduces the eager
results bit for bit (the kernels are deterministic and clear their outputs
with kernels, not memset nodes)."""
import numpy as np
import pytest

from paper_2607_11185_amd import seg as S
from paper_2607_11185_amd import workload as WL
from tests.gpu_helpers import GpuRun, say

pytestmark = pytest.mark.gpu

CFG = WL.Config("graph", 2, (4, 6), 48, 150, (30, 90), 6, 2, 3, 4, 2, 64, 128, 1000)


def _step(run, lc, wl, x, dy, lp_args, lp_cfg):
    o, lse = S.seg_attn_fwd(run.lay, run.q, run.k, run.v, run.scale)
    dq, dk, dv = S.seg_attn_bwd(run.lay, run.q, run.k, run.v, o, lse, run.dout, run.scale)
    lp = S.seg_logprob_loss(*lp_args, lp_cfg)
    y, saved = S.seg_layer_fwd(run.lay, lc, wl, x)
    dx, grads = S.seg_layer_bwd(run.lay, lc, wl, x, saved, dy)
    outs = {"o": o, "lse": lse, "dq": dq, "dk": dk, "dv": dv, "y": y, "dx": dx}
    outs.update({"lp_" + n: t for n, t in lp.items() if t is not None and n != "kl_tok"})
    outs.update({"g_" + n: t for n, t in grads.items()})
    return outs


def test_capture_and_replay_matches_eager():
    import torch
    say("graph capture")
    run = GpuRun(CFG).packed_inputs()
    dev = run.dev
    host = run.host
    R = run.lay.sizes.loss_rows
    src = torch.from_numpy(host["tok_src"].astype(np.int64)).to(dev)
    h = run.inp.h_torch(dev)[src].contiguous()
    w = run.inp.w_torch(dev)
    tgt = torch.from_numpy(run.inp.tgt_np(host["loss_tgt_src"])).to(dev)
    old = torch.from_numpy(run.inp.old_noise_np(host["loss_tgt_src"]).astype(np.float32)).to(dev)
    adv = torch.from_numpy(run.inp.adv_np().astype(np.float32)).to(dev)
    lp_args = (h, run.lay.loss_pred_row, w, tgt, old, adv, run.lay.loss_traj)
    lp_cfg = S.LossCfg(loss_scale=1.0 / R)
    H, I = CFG.hidden, 96
    lc = S.LayerCfg(H, I, CFG.hq, CFG.hkv, CFG.head_dim, 1e-6, 1e4, 500)
    wl = WL.layer_weights_torch(0, H, I, CFG.hq, CFG.hkv, CFG.head_dim, dev)
    x = WL.layer_rows_torch(0, "x", run.P, H, dev)
    dy = WL.layer_rows_torch(0, "dy", run.P, H, dev)

    eager = {n: t.clone() for n, t in _step(run, lc, wl, x, dy, lp_args, lp_cfg).items()}
    torch.cuda.synchronize()

    # warm the capture stream, then capture one whole step
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        _step(run, lc, wl, x, dy, lp_args, lp_cfg)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        captured = _step(run, lc, wl, x, dy, lp_args, lp_cfg)
    torch.cuda.synchronize()

    scratch = torch.randn(1 << 20, device=dev)
    for rep in range(3):
        # the program's own work between replays, touching other memory
        scratch.mul_(1.0001).add_(0.5)
        torch.cuda.synchronize()
        for t in captured.values():
            if t.dtype.is_floating_point:
                t.fill_(float("nan"))
            else:
                t.fill_(0)
        graph.replay()
        torch.cuda.synchronize()
        for n, t in captured.items():
            assert torch.equal(t, eager[n]), (rep, n)
        say(f"  replay {rep}: {len(captured)} outputs equal to the eager step")
