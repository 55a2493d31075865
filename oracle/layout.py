"""Oracle layout: segments, packed tokens, visibility, tile map, loss rows.

TEST INFRASTRUCTURE ONLY (see the package docstring).  Pure Python loops
over small span lists, plus one dense boolean mask per segment.

Notation (Sec. 3.3 and App. D, Alg. "Sliding-window trajectory processing
with token-ID stream"): a trajectory has a prompt P of p tokens and turns
j = 1..T; turn j contributes a screenshot block I_j of m_j tokens and then a
text block X_j of x_j tokens whose last A_j tokens are the trained action
tokens.  Canonical order is P, I_1, X_1, ..., I_T, X_T.

Readings taken where the paper leaves the point open:

* Window (sliding): a query of turn s sees the screenshot of turn j only if
  j > s - W; it always sees every earlier text token.  The paper keeps the
  W most recent screenshots visible and keeps all text as context
  (Sec. 3.3; App. D "Token-ID stream").
* Segment cut: a segment covers at most L consecutive turns [a, b) (L plays
  the removal threshold Delta of Alg. 1/2), closed early when a token cap
  would be exceeded.
* Tokens of a segment [a, b): P, then for every turn j < b its screenshot if
  j > a - W and its text.  Older screenshots are dropped from the segment, as
  the re-tokenised history after pruning drops them; older text stays as
  loss-free context (App. D).
* Loss rows: the last A_j text tokens of each turn j in [a, b); the
  predicting row of a token at packed position t is t - 1 (the ratio uses
  pi(a_t | x_<t), Eq. loss); every action token is trained in exactly one
  segment ("each assistant response is optimized exactly once").
* Packing: segments in (trajectory, first turn) order; with a buffer size B,
  a segment that does not fit in the current buffer opens the next one and
  the tail of the closed buffer is padding.

Anchored mode (the algorithm as printed, App. D): K = W screenshots kept and
removal threshold Delta = L.  The screenshot count of the current token
stream is tracked turn by turn; when turn j's screenshot makes it exceed
K + Delta, the stream is saved as a segment (ending with turn j-1's text),
the oldest Delta screenshots leave the history and the re-tokenised history
(all earlier text, the remaining screenshots, turn j's included) starts the
next segment.  The loop is taken with the observation before the response
of a turn, the canonical order used here (a response follows the screenshot
it conditions on).  Inside a segment every token sees every earlier token:
the window is anchored at the segment start, not slid per query.
"""
from __future__ import annotations

import dataclasses
from typing import List

import numpy as np

KIND_PROMPT, KIND_IMAGE, KIND_TEXT, KIND_PAD = 0, 1, 2, 3
CLS_PARTIAL, CLS_FULL = 1, 2


class CapacityError(ValueError):
    """A single turn does not fit the token cap or the buffer size."""


@dataclasses.dataclass
class Segment:
    traj: int
    a: int                 # first turn (1-based)
    b: int                 # one past the last turn
    start: int             # packed row of the first token
    canon: np.ndarray      # canonical index of each token
    kind: np.ndarray
    step: np.ndarray

    @property
    def length(self) -> int:
        return len(self.canon)


def _traj_spans(spans, t):
    a, b = int(spans.step_offsets[t]), int(spans.step_offsets[t + 1])
    return (int(spans.prompt_len[t]), spans.img_len[a:b].astype(np.int64),
            spans.text_len[a:b].astype(np.int64), spans.action_len[a:b].astype(np.int64))


def segment_length(p, img, text, W, a, b):
    """Tokens of segment [a, b): prompt + text of turns < b + screenshots of
    turns j with max(1, a-W+1) <= j < b (turns are 1-based)."""
    lo = max(1, a - W + 1)
    return p + int(text[: b - 1].sum()) + int(img[lo - 1: b - 1].sum())


def segment_turns(p, img, text, W, L, cap=0):
    """Cut turns 1..T into [a, b) runs of at most L turns (closing early at
    the token cap).  Returns the list of (a, b)."""
    T = len(img)
    segs = []
    a = 1
    while a <= T:
        if cap and segment_length(p, img, text, W, a, a + 1) > cap:
            raise CapacityError(f"turn {a} alone needs more than {cap} tokens")
        b = a + 1
        while b - a < L and b <= T and (
                not cap or segment_length(p, img, text, W, a, b + 1) <= cap):
            b += 1
        segs.append((a, b))
        a = b
    return segs


def anchored_turns(T, K, delta):
    """The algorithm's segments of a T-turn trajectory: list of (a, b, images)
    with images the turns whose screenshot is in the segment's stream.  A
    trajectory without turns gives no segment (its final stream would hold
    no trainable token)."""
    segs = []
    history = []        # turns whose screenshot is in the text history
    stream = []         # turns whose screenshot is in the current stream
    n_img = 0
    a = 1
    for t in range(1, T + 1):
        n_img += 1      # observation with screenshot of turn t
        history.append(t)
        if n_img > K + delta:
            segs.append((a, t, tuple(stream)))      # saved before turn t's tokens
            history = history[delta:]               # oldest Delta screenshots removed
            n_img -= delta
            stream = list(history)                  # re-tokenised history
            a = t
        else:
            stream.append(t)                        # token-diff append
        # the response of turn t follows (trainable tokens)
    if a <= T:  # the final stream; an episode without turns has no trainable token
        segs.append((a, T + 1, tuple(stream)))
    return segs


def segment_tokens_with(p, img, text, images, b, canon0):
    """(canonical index, kind, step) of a segment whose turns are < b and
    whose screenshots are exactly those of the turns in ``images``."""
    keep = set(images)
    canon, kind, step = [], [], []
    canon.extend(range(canon0, canon0 + p))
    kind.extend([KIND_PROMPT] * p)
    step.extend([0] * p)
    c = canon0 + p
    for j in range(1, b):
        m, x = int(img[j - 1]), int(text[j - 1])
        if j in keep:
            canon.extend(range(c, c + m))
            kind.extend([KIND_IMAGE] * m)
            step.extend([j] * m)
        c += m
        canon.extend(range(c, c + x))
        kind.extend([KIND_TEXT] * x)
        step.extend([j] * x)
        c += x
    return (np.asarray(canon, np.int64), np.asarray(kind, np.int64),
            np.asarray(step, np.int64))


def segment_tokens(p, img, text, W, a, b, canon0):
    """(canonical index, kind, step) of every token of segment [a, b)."""
    canon, kind, step = [], [], []
    canon.extend(range(canon0, canon0 + p))
    kind.extend([KIND_PROMPT] * p)
    step.extend([0] * p)
    c = canon0 + p
    for j in range(1, b):
        m, x = int(img[j - 1]), int(text[j - 1])
        if j > a - W:
            canon.extend(range(c, c + m))
            kind.extend([KIND_IMAGE] * m)
            step.extend([j] * m)
        c += m
        canon.extend(range(c, c + x))
        kind.extend([KIND_TEXT] * x)
        step.extend([j] * x)
        c += x
    return (np.asarray(canon, np.int64), np.asarray(kind, np.int64),
            np.asarray(step, np.int64))


def visibility(seg: Segment, W) -> np.ndarray:
    """Dense mask[q, k]: key k visible to query q (same segment, k not after
    q, and k not a screenshot more than W-1 turns older than q's turn).
    W = None is the anchored mode: causal inside the segment."""
    n = seg.length
    qi = np.arange(n)[:, None]
    ki = np.arange(n)[None, :]
    causal = ki <= qi
    if W is None:
        return causal
    expired = (seg.kind[None, :] == KIND_IMAGE) & (seg.step[None, :] <= seg.step[:, None] - W)
    return causal & ~expired


def visibility_rows(seg: Segment, W, rows) -> np.ndarray:
    """Rows ``rows`` of the dense mask of :func:`visibility`."""
    rows = np.asarray(rows)
    ki = np.arange(seg.length)[None, :]
    causal = ki <= rows[:, None]
    if W is None:
        return causal
    expired = (seg.kind[None, :] == KIND_IMAGE) & (seg.step[None, :] <= seg.step[rows][:, None] - W)
    return causal & ~expired


def segment_tiles(seg: Segment, W: int, tile: int):
    """Class grid [nt, nt] of one segment (0 = skip, PARTIAL, FULL) and its
    exact visible-pair count, read off the dense mask: a tile is skipped when
    it holds no visible pair and FULL when it is tile x tile and every pair
    is visible."""
    mask = visibility(seg, W)
    n = seg.length
    nt = -(-n // tile)
    cls = np.zeros((nt, nt), np.int64)
    for i in range(nt):
        for j in range(nt):
            sub = mask[i * tile:(i + 1) * tile, j * tile:(j + 1) * tile]
            if not sub.any():
                continue
            full = sub.shape == (tile, tile) and bool(sub.all())
            cls[i, j] = CLS_FULL if full else CLS_PARTIAL
    return cls, int(mask.sum())


@dataclasses.dataclass
class Layout:
    segments: List[Segment]
    packed_tokens: int
    num_buffers: int
    tok_src: np.ndarray
    tok_meta: np.ndarray
    seg_info: np.ndarray        # [S, 8]
    loss_pred_row: np.ndarray
    loss_tgt_src: np.ndarray
    loss_traj: np.ndarray
    tile_seg: np.ndarray
    qt_ptr: np.ndarray
    qt_col: np.ndarray
    qt_cls: np.ndarray
    kt_ptr: np.ndarray
    kt_row: np.ndarray
    kt_cls: np.ndarray
    seg_pairs: np.ndarray
    tile: int
    window: int


def build(spans, W, L, tile, cap=0, buffer_tokens=0, with_tiles=True,
          mode="sliding") -> Layout:
    """All layout arrays of a batch (steps O1-O6 of the segmented path).

    mode "anchored": segments and screenshots from :func:`anchored_turns`
    with K = W and Delta = L, causal visibility (no token cap)."""
    if mode not in ("sliding", "anchored"):
        raise ValueError(mode)
    if mode == "anchored" and cap:
        raise ValueError("the anchored mode has no token cap")
    Wv = None if mode == "anchored" else W
    canon_off = [0]
    for t in range(spans.num_traj):
        p, img, text, _ = _traj_spans(spans, t)
        canon_off.append(canon_off[-1] + p + int(img.sum()) + int(text.sum()))

    # O1 + O3: segments and their tokens
    segs: List[Segment] = []
    for t in range(spans.num_traj):
        p, img, text, _ = _traj_spans(spans, t)
        if mode == "anchored":
            cuts = anchored_turns(len(img), W, L)
        else:
            cuts = [(a, b, None) for a, b in segment_turns(p, img, text, W, L, cap)]
        for a, b, images in cuts:
            if images is None:
                c, k, s = segment_tokens(p, img, text, W, a, b, canon_off[t])
            else:
                c, k, s = segment_tokens_with(p, img, text, images, b, canon_off[t])
            if len(c) == 0:
                raise ValueError(f"segment of trajectory {t}, turns {a}..{b - 1} holds no token")
            if buffer_tokens and len(c) > buffer_tokens:
                raise CapacityError(f"segment of {len(c)} tokens exceeds the buffer")
            segs.append(Segment(t, a, b, -1, c, k, s))

    # O2: packing
    pos, nbuf, fill = 0, 0, 0
    for sg in segs:
        if buffer_tokens:
            if nbuf == 0 or fill + sg.length > buffer_tokens:
                pos = nbuf * buffer_tokens
                nbuf += 1
                fill = 0
            sg.start = pos
            pos += sg.length
            fill += sg.length
        else:
            sg.start = pos
            pos += sg.length
    if buffer_tokens:
        packed = nbuf * buffer_tokens
    else:
        packed = pos
        nbuf = 1 if segs else 0

    tok_src = np.full(packed, -1, np.int64)
    tok_meta = np.full(packed, KIND_PAD, np.int64)
    for sg in segs:
        tok_src[sg.start: sg.start + sg.length] = sg.canon
        tok_meta[sg.start: sg.start + sg.length] = (sg.step << 2) | sg.kind

    # O6: loss rows (ordered by packed position)
    pred, tgt, trj, seg_nloss = [], [], [], []
    for sg in segs:
        p, img, text, act = _traj_spans(spans, sg.traj)
        n0 = len(pred)
        for j in range(sg.a, sg.b):        # earlier turns are context only
            xj = np.nonzero((sg.kind == KIND_TEXT) & (sg.step == j))[0]
            nact = int(act[j - 1])
            for i in (xj[len(xj) - nact:] if nact else []):
                if i == 0:
                    # pi(a_t | x_<t) needs a row before the token (Eq. loss)
                    raise ValueError(f"turn {j}: a trained token opens its segment")
                pred.append(sg.start + int(i) - 1)
                tgt.append(int(sg.canon[i]))
                trj.append(sg.traj)
        seg_nloss.append(len(pred) - n0)

    # O5: tiles (from the dense mask of every segment)
    tile_seg, qt_rows, kt_cols, pairs = [], [], [], []
    qbase = 0
    seg_info = np.zeros((len(segs), 8), np.int64)
    loss_base = 0
    for si, sg in enumerate(segs):
        n = sg.length
        nt = -(-n // tile)
        seg_info[si] = [sg.traj, sg.a, sg.b, sg.start, n, qbase, loss_base, seg_nloss[si]]
        loss_base += seg_nloss[si]
        if with_tiles:
            cls, npairs = segment_tiles(sg, Wv, tile)
            pairs.append(npairs)
            for i in range(nt):
                qt_rows.append([(qbase + j, int(cls[i, j])) for j in range(nt) if cls[i, j]])
            for j in range(nt):
                kt_cols.append([(qbase + i, int(cls[i, j])) for i in range(nt) if cls[i, j]])
        tile_seg.extend([si] * nt)
        qbase += nt

    def csr(rows):
        ptr = np.zeros(len(rows) + 1, np.int64)
        for i, r in enumerate(rows):
            ptr[i + 1] = ptr[i] + len(r)
        col = np.asarray([c for r in rows for c, _ in r], np.int64)
        cl = np.asarray([k for r in rows for _, k in r], np.int64)
        return ptr, col, cl

    qt_ptr, qt_col, qt_cls = csr(qt_rows)
    kt_ptr, kt_row, kt_cls = csr(kt_cols)
    return Layout(segs, packed, nbuf, tok_src, tok_meta, seg_info,
                  np.asarray(pred, np.int64), np.asarray(tgt, np.int64),
                  np.asarray(trj, np.int64), np.asarray(tile_seg, np.int64),
                  qt_ptr, qt_col, qt_cls, kt_ptr, kt_row, kt_cls,
                  np.asarray(pairs, np.int64), tile, Wv)
