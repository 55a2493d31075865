"""Seeded synthetic workloads: step spans and per-token tensors.

This module is the only code that both the oracle-side tests and the HIP path
consume.  It holds no arithmetic of the method itself (no segmentation, no
visibility rule, no attention or loss): it only draws trajectory shapes and
input values.

Shapes follow the paper's setting (Sec. 3.3 and App. D): a trajectory is a
system prompt followed by T turns; each turn carries one screenshot
(image-token block) and one assistant text block whose last tokens are the
action tokens trained by the clipped policy-ratio objective (Eq. loss).

Random values come from a counter-based generator (a 32-bit integer hash of
the element index, "lowbias32" by C. Wellons) so that any element of any
tensor can be regenerated independently and bit-identically on the host
(NumPy) and on the device (PyTorch integer ops).  Normal variates use the
Irwin-Hall construction: the sum of four uniforms on 16-bit grids, centred and
scaled to unit variance; every step is an exactly rounded IEEE operation, so
both backends agree bit for bit.  Values are then rounded to float32 and, for
bf16 tensors, to bfloat16 with round-to-nearest-even.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

M32 = 0xFFFFFFFF
SQRT3 = math.sqrt(3.0)

# stream ids of the tensors (part of the generator's counter key)
STREAM = {"q": 1, "k": 2, "v": 3, "h": 4, "tgt": 5, "dout": 6, "w": 7, "adv": 8,
          "old_noise": 9}

# token kinds as carried in tok_meta = step << 2 | kind
KIND_PROMPT, KIND_IMAGE, KIND_TEXT, KIND_PAD = 0, 1, 2, 3


@dataclasses.dataclass(frozen=True)
class Config:
    """One synthetic workload.  Lengths are in tokens; ranges are inclusive."""
    name: str
    num_traj: int
    steps: tuple            # (lo, hi) turns per trajectory
    prompt_len: int
    img_len: int
    text_len: tuple         # (lo, hi) non-image tokens per turn
    action_len: int         # trained action tokens = last action_len text tokens
    window: int             # W screenshots kept visible
    seg_steps: int          # L turns per segment (1 = step-wise decomposition)
    hq: int
    hkv: int
    head_dim: int
    hidden: int
    vocab: int
    dtype: str = "bf16"     # dtype of q/k/v/dout/h: "bf16" or "f32"
    max_seg_tokens: int = 0
    buffer_tokens: int = 0
    eps_low: float = 0.2
    eps_high: float = 0.2
    dual_clip: float = 0.0  # ratio cap c of the dual clip (0: off)
    w_std: float = 0.02
    old_noise_std: float = 0.1
    seed: int = 0
    mode: str = "sliding"   # "sliding" window, or "anchored" (the App. D algorithm as printed)

    def with_(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


# The workloads (shapes of the paper's OSWorld/ScienceBoard
# style rollouts; 1920x1080 screenshots with 28-px merged patches give
# round(1920/28) * round(1080/28) = 69 * 39 = 2691 image tokens).
TINY = Config("tiny", 1, (8, 8), 64, 64, (32, 32), 8, 2, 4, 4, 1, 64, 128, 1024,
              dtype="f32")
SMALL = Config("small", 4, (16, 16), 256, 1024, (64, 192), 16, 3, 4, 16, 2, 128,
               2048, 32000)
SEVEN_B = Config("7b", 8, (30, 30), 512, 2691, (150, 400), 32, 3, 5, 28, 4, 128,
                 3584, 151936)
STEPWISE_7B = SEVEN_B.with_(name="7b_stepwise", seg_steps=1)
LONG = Config("long", 16, (10, 50), 512, 4096, (100, 600), 32, 5, 8, 28, 4, 128,
              3584, 151936, max_seg_tokens=65536, buffer_tokens=65536)
# The 7B-class batch cut the way the App. D algorithm does, with the paper's
# RL settings (hyperparameter table): K = 5 screenshots kept, removal
# threshold delta = 5, clip 0.2 / 0.28 with ratio cap c = 3.
SEVEN_B_ANCHORED = SEVEN_B.with_(name="7b_anchored", mode="anchored", window=5, seg_steps=5,
                                 eps_high=0.28, dual_clip=3.0)
# One rank's share of the 7B-class batch under the paper's tensor parallelism
# (TP = 4, heads and vocabulary split): 7 query heads of one kv head and a
# quarter of the vocabulary (the collectives themselves are not modelled).
SEVEN_B_TP4_RANK = SEVEN_B.with_(name="7b_tp4_rank", hq=7, hkv=1, vocab=151936 // 4)
CONFIGS = {c.name: c for c in (TINY, SMALL, SEVEN_B, STEPWISE_7B, LONG, SEVEN_B_ANCHORED,
                               SEVEN_B_TP4_RANK)}


@dataclasses.dataclass
class Spans:
    """Step spans of a batch of trajectories (all int32 host arrays)."""
    step_offsets: np.ndarray   # [num_traj+1]
    prompt_len: np.ndarray     # [num_traj]
    img_len: np.ndarray        # [num_steps]
    text_len: np.ndarray       # [num_steps]
    action_len: np.ndarray     # [num_steps]

    @property
    def num_traj(self) -> int:
        return len(self.prompt_len)

    @property
    def num_steps(self) -> int:
        return int(self.step_offsets[-1])

    def traj_tokens(self) -> np.ndarray:
        """Canonical token count of each trajectory: prompt + all turns."""
        out = np.zeros(self.num_traj, np.int64)
        for t in range(self.num_traj):
            a, b = self.step_offsets[t], self.step_offsets[t + 1]
            out[t] = int(self.prompt_len[t]) + int(self.img_len[a:b].sum()) + int(
                self.text_len[a:b].sum())
        return out

    def canon_offsets(self) -> np.ndarray:
        """[num_traj+1] start of each trajectory in the canonical token order."""
        return np.concatenate([[0], np.cumsum(self.traj_tokens())]).astype(np.int64)

    def subset(self, t0: int, t1: int) -> "Spans":
        """Trajectories t0 .. t1-1 as a batch of their own."""
        a, b = int(self.step_offsets[t0]), int(self.step_offsets[t1])
        return Spans(step_offsets=(self.step_offsets[t0:t1 + 1] - a).astype(np.int32),
                     prompt_len=self.prompt_len[t0:t1].copy(), img_len=self.img_len[a:b].copy(),
                     text_len=self.text_len[a:b].copy(), action_len=self.action_len[a:b].copy())


def make_spans(cfg: Config, seed: Optional[int] = None) -> Spans:
    """Draw turn counts and text lengths (NumPy PCG64, SeedSequence(seed))."""
    seed = cfg.seed if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0x5ea5])))
    lo, hi = cfg.steps
    T = rng.integers(lo, hi + 1, size=cfg.num_traj)
    n = int(T.sum())
    tl, th = cfg.text_len
    text = rng.integers(tl, th + 1, size=n).astype(np.int32)
    return Spans(
        step_offsets=np.concatenate([[0], np.cumsum(T)]).astype(np.int32),
        prompt_len=np.full(cfg.num_traj, cfg.prompt_len, np.int32),
        img_len=np.full(n, cfg.img_len, np.int32),
        text_len=text,
        action_len=np.minimum(np.full(n, cfg.action_len, np.int32), text),
    )


def explicit_spans(steps_per_traj, prompt, img, text, action) -> Spans:
    """Spans from explicit per-step lists (hand-worked and edge cases).

    ``prompt`` is one length per trajectory; ``img``/``text``/``action`` are
    flat per-step lists in trajectory order.
    """
    T = np.asarray(steps_per_traj, np.int64)
    return Spans(
        step_offsets=np.concatenate([[0], np.cumsum(T)]).astype(np.int32),
        prompt_len=np.asarray(prompt, np.int32),
        img_len=np.asarray(img, np.int32).reshape(-1),
        text_len=np.asarray(text, np.int32).reshape(-1),
        action_len=np.asarray(action, np.int32).reshape(-1),
    )


def canonical_tokens(spans: Spans):
    """Kind and step of every canonical token (prompt, then I_j, X_j per turn).

    Returns (kind[int8], step[int32], traj[int32]) over all trajectories in
    canonical order.  Pure bookkeeping of the span lists.
    """
    kinds, steps, trajs = [], [], []
    for t in range(spans.num_traj):
        a, b = spans.step_offsets[t], spans.step_offsets[t + 1]
        kinds.append(np.full(spans.prompt_len[t], KIND_PROMPT, np.int8))
        steps.append(np.zeros(spans.prompt_len[t], np.int32))
        for j, s in enumerate(range(a, b), start=1):
            kinds.append(np.full(spans.img_len[s], KIND_IMAGE, np.int8))
            steps.append(np.full(spans.img_len[s], j, np.int32))
            kinds.append(np.full(spans.text_len[s], KIND_TEXT, np.int8))
            steps.append(np.full(spans.text_len[s], j, np.int32))
        n = int(spans.prompt_len[t] + spans.img_len[a:b].sum() + spans.text_len[a:b].sum())
        trajs.append(np.full(n, t, np.int32))
    return np.concatenate(kinds), np.concatenate(steps), np.concatenate(trajs)


# ----------------------------------------------------------------------------
# counter-based generator (identical integer ops on NumPy and torch arrays)

def _mul32(x, c: int):
    """(x * c) mod 2^32 for x < 2^32 without leaving the signed int64 range."""
    lo, hi = c & 0xFFFF, c >> 16
    return (x * lo + (((x * hi) & 0xFFFF) << 16)) & M32


def hash32(x):
    """lowbias32 integer hash (C. Wellons), a bijection on 32-bit words.

    NumPy uint32 arrays use native wrap-around multiplication; other arrays
    (torch int64) use the split multiply of :func:`_mul32`.  Both compute the
    same function.
    """
    if isinstance(x, np.ndarray) and x.dtype == np.uint32:
        x = x ^ (x >> np.uint32(16))
        x *= np.uint32(0x7FEB352D)
        x ^= x >> np.uint32(15)
        x *= np.uint32(0x846CA68B)
        x ^= x >> np.uint32(16)
        return x
    x = x ^ (x >> 16)
    x = _mul32(x, 0x7FEB352D)
    x = x ^ (x >> 15)
    x = _mul32(x, 0x846CA68B)
    x = x ^ (x >> 16)
    return x


def _key(seed: int, stream: int, word: int) -> int:
    k = (seed * 0x9E3779B1 + stream * 0x85EBCA6B + word * 0xC2B2AE35) & M32
    # run the key itself through the hash so nearby seeds decorrelate
    x = k
    x ^= x >> 16
    x = (x * 0x7FEB352D) & M32
    x ^= x >> 15
    x = (x * 0x846CA68B) & M32
    x ^= x >> 16
    return x


def _words(idx, seed, stream, word):
    """32-bit random word for every element index in ``idx`` (int64 array)."""
    k = _key(seed, stream, word)
    if isinstance(idx, np.ndarray):
        lo = (idx & M32).astype(np.uint32)
        hi = (idx >> 32).astype(np.uint32)
        return hash32(hash32(lo ^ np.uint32(k)) ^ hi).astype(np.int64)
    lo = idx & M32
    hi = idx >> 32
    return hash32(hash32(lo ^ k) ^ hi)


def _normal_from_words(w0, w1, xp):
    """Irwin-Hall(4) normal from two words, as float64 (exact up to one rounding)."""
    s = (w0 & 0xFFFF) + (w0 >> 16) + (w1 & 0xFFFF) + (w1 >> 16)   # < 2^18
    num = s + 2 - 131072                                          # centred, exact
    if xp is np:
        z = num.astype(np.float64) / 65536.0
    else:
        z = num.to(xp.float64) / 65536.0
    return z * SQRT3


def bf16_round_np(x32: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 (as uint16 bits), round-to-nearest-even."""
    u = np.ascontiguousarray(x32, np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    return r


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _normal_np_chunk(seed, stream, idx, std, dtype):
    z = _normal_from_words(_words(idx, seed, stream, 0), _words(idx, seed, stream, 1), np)
    v32 = (z * std).astype(np.float32)
    if dtype == "bf16":
        return bf16_bits_to_f64(bf16_round_np(v32))
    return v32.astype(np.float64)


def normal_np(seed, stream, idx, std=1.0, dtype="bf16", chunk=1 << 18):
    """Values of elements ``idx`` of a normal tensor, as float64 host array.

    The returned float64 values are exactly the values stored in the tensor's
    dtype (bf16 or f32).  Large requests are split over threads.
    """
    idx = np.asarray(idx, np.int64)
    if idx.size <= chunk:
        return _normal_np_chunk(seed, stream, idx, std, dtype)
    flat = idx.reshape(-1)
    out = np.empty(flat.size, np.float64)

    def work(c0):
        c1 = min(flat.size, c0 + chunk)
        out[c0:c1] = _normal_np_chunk(seed, stream, flat[c0:c1], std, dtype)

    _parallel(work, range(0, flat.size, chunk))
    return out.reshape(idx.shape)


def normal_rows_np(seed, stream, rows, width, std=1.0, dtype="bf16", chunk=1 << 18):
    """Rows ``rows`` of a [*, width] normal tensor (element r*width + c)."""
    rows = np.asarray(rows, np.int64).reshape(-1)
    out = np.empty((rows.size, width), np.float64)
    per = max(1, chunk // width)
    cols = np.arange(width, dtype=np.int64)[None, :]

    def work(r0):
        r1 = min(rows.size, r0 + per)
        idx = rows[r0:r1, None] * width + cols
        out[r0:r1] = _normal_np_chunk(seed, stream, idx, std, dtype)

    _parallel(work, range(0, rows.size, per))
    return out


def _parallel(fn, starts):
    import concurrent.futures as cf
    import os
    starts = list(starts)
    if len(starts) <= 1:
        for s0 in starts:
            fn(s0)
        return
    with cf.ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
        list(ex.map(fn, starts))


def uniform_int_np(seed, stream, idx, n):
    idx = np.asarray(idx, np.int64)
    return ((_words(idx, seed, stream, 0) * n) >> 32).astype(np.int32)


def normal_torch(seed, stream, start, count, std=1.0, dtype="bf16", device="cuda",
                 chunk=1 << 25):
    """Device tensor of elements [start, start+count) of a normal tensor."""
    import torch
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    out = torch.empty(count, dtype=tdt, device=device)
    for c0 in range(0, count, chunk):
        c1 = min(count, c0 + chunk)
        idx = torch.arange(start + c0, start + c1, dtype=torch.int64, device=device)
        z = _normal_from_words(_words(idx, seed, stream, 0), _words(idx, seed, stream, 1),
                               torch)
        out[c0:c1] = (z * std).to(torch.float32).to(tdt)
        del idx, z
    return out


def uniform_int_torch(seed, stream, start, count, n, device="cuda"):
    import torch
    idx = torch.arange(start, start + count, dtype=torch.int64, device=device)
    return ((_words(idx, seed, stream, 0) * n) >> 32).to(torch.int32)


# ----------------------------------------------------------------------------
# the tensors of a workload

class Inputs:
    """Lazily generated input tensors of one workload.

    Canonical per-token tensors (q, k, v, h, targets, old-logp noise) are
    indexed by canonical token; ``dout`` is indexed by packed row; the vocab
    projection ``w`` and per-trajectory advantages are global.
    """

    def __init__(self, cfg: Config, spans: Optional[Spans] = None, seed: Optional[int] = None):
        self.cfg = cfg
        self.seed = cfg.seed if seed is None else seed
        self.spans = spans if spans is not None else make_spans(cfg, self.seed)
        self.canon_off = self.spans.canon_offsets()
        self.n_canon = int(self.canon_off[-1])

    # ---- host (float64 values exactly as stored) ----
    def _rows_np(self, name, rows, width, std, dtype):
        return normal_rows_np(self.seed, STREAM[name], rows, width, std, dtype)

    def q_np(self, rows):
        c = self.cfg
        return self._rows_np("q", rows, c.hq * c.head_dim, 1.0, c.dtype).reshape(
            -1, c.hq, c.head_dim)

    def k_np(self, rows):
        c = self.cfg
        return self._rows_np("k", rows, c.hkv * c.head_dim, 1.0, c.dtype).reshape(
            -1, c.hkv, c.head_dim)

    def v_np(self, rows):
        c = self.cfg
        return self._rows_np("v", rows, c.hkv * c.head_dim, 1.0, c.dtype).reshape(
            -1, c.hkv, c.head_dim)

    def dout_np(self, packed_rows):
        c = self.cfg
        return self._rows_np("dout", packed_rows, c.hq * c.head_dim, 1.0, c.dtype).reshape(
            -1, c.hq, c.head_dim)

    def h_np(self, rows):
        c = self.cfg
        return self._rows_np("h", rows, c.hidden, 1.0, c.dtype)

    def w_np(self, vocab_rows=None):
        c = self.cfg
        rows = np.arange(c.vocab) if vocab_rows is None else vocab_rows
        return self._rows_np("w", rows, c.hidden, c.w_std, "bf16" if c.dtype == "bf16" else "f32")

    def tgt_np(self, rows):
        return uniform_int_np(self.seed, STREAM["tgt"], rows, self.cfg.vocab)

    def adv_np(self):
        return normal_np(self.seed, STREAM["adv"], np.arange(self.spans.num_traj), 1.0, "f32")

    def old_noise_np(self, rows):
        return normal_np(self.seed, STREAM["old_noise"], rows, self.cfg.old_noise_std, "f32")

    # ---- device ----
    def _t(self, name, n_rows, width, std, dtype, device):
        return normal_torch(self.seed, STREAM[name], 0, n_rows * width, std, dtype,
                            device).view(n_rows, width)

    def q_torch(self, device="cuda"):
        c = self.cfg
        return self._t("q", self.n_canon, c.hq * c.head_dim, 1.0, c.dtype, device).view(
            self.n_canon, c.hq, c.head_dim)

    def k_torch(self, device="cuda"):
        c = self.cfg
        return self._t("k", self.n_canon, c.hkv * c.head_dim, 1.0, c.dtype, device).view(
            self.n_canon, c.hkv, c.head_dim)

    def v_torch(self, device="cuda"):
        c = self.cfg
        return self._t("v", self.n_canon, c.hkv * c.head_dim, 1.0, c.dtype, device).view(
            self.n_canon, c.hkv, c.head_dim)

    def dout_torch(self, n_packed, device="cuda"):
        c = self.cfg
        return self._t("dout", n_packed, c.hq * c.head_dim, 1.0, c.dtype, device).view(
            n_packed, c.hq, c.head_dim)

    def h_torch(self, device="cuda"):
        c = self.cfg
        return self._t("h", self.n_canon, c.hidden, 1.0, c.dtype, device)

    def w_torch(self, device="cuda"):
        c = self.cfg
        return self._t("w", c.vocab, c.hidden, c.w_std,
                       "bf16" if c.dtype == "bf16" else "f32", device)

    def tgt_torch(self, device="cuda"):
        return uniform_int_torch(self.seed, STREAM["tgt"], 0, self.n_canon, self.cfg.vocab,
                                 device)


# ----------------------------------------------------------------------------
# decoder-layer tensors (random-init weights of a Qwen-style layer)

LAYER_STREAM = {"x": 10, "dy": 11, "g1": 12, "wq": 13, "wk": 14, "wv": 15, "wo": 16, "g2": 17,
                "wg": 18, "wu": 19, "wd": 20}
LAYER_WEIGHTS = ("g1", "wq", "wk", "wv", "wo", "g2", "wg", "wu", "wd")


def layer_shapes(H, I, hq, hkv, d) -> dict:
    return {"g1": (H,), "wq": (hq * d, H), "wk": (hkv * d, H), "wv": (hkv * d, H),
            "wo": (H, hq * d), "g2": (H,), "wg": (I, H), "wu": (I, H), "wd": (H, I)}


def _gain_bits(seed, name, n):
    """Norm gains 1 + 0.1 z, rounded to float32 and then to bf16 (bits)."""
    z = normal_np(seed, LAYER_STREAM[name], np.arange(n), 1.0, "f32")
    return bf16_round_np((1.0 + 0.1 * z).astype(np.float32))


def layer_weights_np(seed, H, I, hq, hkv, d) -> dict:
    """bf16 layer weights as float64 values: gains 1 + 0.1 z, projections
    z / sqrt(fan_in)."""
    out = {}
    for n, shp in layer_shapes(H, I, hq, hkv, d).items():
        if len(shp) == 1:
            out[n] = bf16_bits_to_f64(_gain_bits(seed, n, shp[0]))
        else:
            out[n] = normal_np(seed, LAYER_STREAM[n], np.arange(shp[0] * shp[1]),
                               1.0 / math.sqrt(shp[1])).reshape(shp)
    return out


def layer_weights_torch(seed, H, I, hq, hkv, d, device="cuda") -> dict:
    """The same weights as layer_weights_np, as bf16 device tensors."""
    import torch
    out = {}
    for n, shp in layer_shapes(H, I, hq, hkv, d).items():
        if len(shp) == 1:
            bits = _gain_bits(seed, n, shp[0]).astype(np.int16)
            out[n] = torch.from_numpy(bits).view(torch.bfloat16).to(device)
        else:
            out[n] = normal_torch(seed, LAYER_STREAM[n], 0, shp[0] * shp[1],
                                  1.0 / math.sqrt(shp[1]), "bf16", device).view(*shp)
    return out


def layer_rows_np(seed, name, rows, width) -> np.ndarray:
    """Rows of a [*, width] standard-normal bf16 tensor ("x" or "dy")."""
    return normal_rows_np(seed, LAYER_STREAM[name], rows, width, 1.0, "bf16")


def layer_rows_torch(seed, name, n_rows, width, device="cuda"):
    return normal_torch(seed, LAYER_STREAM[name], 0, n_rows * width, 1.0, "bf16",
                        device).view(n_rows, width)
