"""Span-query attention, written out from its definition (float64, CPU).

Layout (Def. 2-4, section 4.3): the model input of a RAG/ITS span query
``G(cross-join(prefix, plus(F_1..F_n), cross))`` is the concatenation
``S = p | F_s1 | ... | F_sn | c`` of a shared prefix, the commuting fragments in
the order this query presents them, and the non-commuting cross segment (the
question or judge prompt).

Mask (section 5.6, span sparsity; footnote of section 5.1 on preparing
fragments independently of their context): a prefix token attends causally
within the prefix; a token of fragment i attends to the whole prefix and
causally within fragment i, and to nothing of the other fragments; a cross
token attends causally to everything before it.

Positions (section 5.5, repositioning): a fragment is prepared once, at
positions that do not depend on where it lands in a particular query
(canonical positions: prefix token t at t, fragment token j at P + j).  When
the cross segment reads the cached keys, each block is repositioned to where
the query places it (final positions: the index in S).  Prefix and fragment
rows therefore use canonical positions for their query and all their keys;
cross rows use final positions for their query and all their keys.

Rotary encoding (section 5.5 cites RoFormer): rotate-half pairing (i, i+d/2),
inverse frequency theta^(-2i/d), angles in float64.

Parity unpinned: nothing here.  Every function is pinned by tests against the
paper's statements and textbook reductions (causal attention, closed forms,
rotary identities).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Sequence

import numpy as np

SEG_PREFIX = -1
SEG_CROSS = -2


@dataclass
class Layout:
    seg: np.ndarray        # [N] segment id: SEG_PREFIX, fragment child index 0..n-1, SEG_CROSS
    idx: np.ndarray        # [N] index of the token inside its segment
    pos_canon: np.ndarray  # [N] canonical position
    pos_final: np.ndarray  # [N] final position (index in S)
    prefix_len: int
    frag_lens: tuple
    cross_len: int

    @property
    def n(self) -> int:
        return int(self.seg.shape[0])


def layout(prefix_len: int, frag_lens: Sequence[int], cross_len: int) -> Layout:
    """Segment ids and both position frames of S = p | F_1 | ... | F_n | c."""
    P = int(prefix_len)
    frag_lens = tuple(int(x) for x in frag_lens)
    total_frag = sum(frag_lens)
    seg, idx, canon = [], [], []
    for t in range(P):
        seg.append(SEG_PREFIX); idx.append(t); canon.append(t)
    for i, L in enumerate(frag_lens):
        for j in range(L):
            seg.append(i); idx.append(j); canon.append(P + j)
    for t in range(cross_len):
        seg.append(SEG_CROSS); idx.append(t); canon.append(P + total_frag + t)
    n = len(seg)
    return Layout(seg=np.array(seg, np.int64), idx=np.array(idx, np.int64),
                  pos_canon=np.array(canon, np.int64), pos_final=np.arange(n, dtype=np.int64),
                  prefix_len=P, frag_lens=frag_lens, cross_len=int(cross_len))


def mask_rows(lay: Layout, rows: np.ndarray) -> np.ndarray:
    """Boolean [len(rows), N]: may row r attend to key c."""
    rows = np.asarray(rows, np.int64)
    seg_r = lay.seg[rows][:, None]
    idx_r = lay.idx[rows][:, None]
    seg_c = lay.seg[None, :]
    idx_c = lay.idx[None, :]
    c = np.arange(lay.n)[None, :]
    prefix_row = (seg_c == SEG_PREFIX) & (idx_c <= idx_r)
    frag_row = (seg_c == SEG_PREFIX) | ((seg_c == seg_r) & (idx_c <= idx_r))
    cross_row = c <= rows[:, None]
    return np.where(seg_r == SEG_PREFIX, prefix_row, np.where(seg_r == SEG_CROSS, cross_row, frag_row))


def span_mask(lay: Layout) -> np.ndarray:
    """The full N x N mask."""
    return mask_rows(lay, np.arange(lay.n))


def inv_freq(head_dim: int, theta: float) -> np.ndarray:
    i = np.arange(head_dim // 2, dtype=np.float64)
    return theta ** (-2.0 * i / head_dim)


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half rotary encoding of x[..., N, (H,) d] at integer positions pos[N]."""
    x = np.asarray(x, np.float64)
    d = x.shape[-1]
    h = d // 2
    ang = np.asarray(pos, np.float64)[:, None] * inv_freq(d, theta)[None, :]   # [N, d/2]
    cos, sin = np.cos(ang), np.sin(ang)
    if x.ndim == 3:   # [N, H, d]
        cos, sin = cos[:, None, :], sin[:, None, :]
    a, b = x[..., :h], x[..., h:]
    return np.concatenate([a * cos - b * sin, b * cos + a * sin], axis=-1)


def attention_rows(q: np.ndarray, k: np.ndarray, v: np.ndarray, lay: Layout, rows: Sequence[int],
                   theta: float, block: int = 256) -> np.ndarray:
    """Output rows of span attention for the sequence S.

    q: [N, Hq, d], k, v: [N, Hkv, d] (pre-rotary, any float dtype; promoted to
    float64).  Returns float64 [len(rows), Hq, d].  Query head h reads kv head
    floor(h * Hkv / Hq).
    """
    q = np.asarray(q, np.float64); k = np.asarray(k, np.float64); v = np.asarray(v, np.float64)
    n, hq, d = q.shape
    hkv = k.shape[1]
    rows = np.asarray(rows, np.int64)
    out = np.zeros((rows.shape[0], hq, d), np.float64)
    scale = 1.0 / np.sqrt(d)
    # cross rows use final positions, prefix/fragment rows canonical positions
    phases = [(lay.seg[rows] != SEG_CROSS, lay.pos_canon), (lay.seg[rows] == SEG_CROSS, lay.pos_final)]
    for sel, pos in phases:
        sel_idx = np.nonzero(sel)[0]
        if sel_idx.size == 0:
            continue
        k_rot = rope(k, pos, theta)                                   # [N, Hkv, d]
        for b0 in range(0, sel_idx.size, block):
            out_at = sel_idx[b0: b0 + block]
            r = rows[out_at]
            q_rot = rope(q[r], pos[r], theta)                        # [B, Hq, d]
            allowed = mask_rows(lay, r)                              # [B, N]
            for h in range(hq):
                g = (h * hkv) // hq
                s = (q_rot[:, h, :] @ k_rot[:, g, :].T) * scale       # [B, N]
                s = np.where(allowed, s, -np.inf)
                m = np.max(s, axis=1, keepdims=True)
                w = np.exp(s - m)                                    # masked entries are exactly 0
                w /= np.sum(w, axis=1, keepdims=True)
                out[out_at, h, :] = w @ v[:, g, :]
    return out


def span_attention(q, k, v, lay: Layout, theta: float) -> np.ndarray:
    """All N output rows."""
    return attention_rows(q, k, v, lay, np.arange(lay.n), theta)


def cached_fragment_kv(k: np.ndarray, v: np.ndarray, lay: Layout, child: int, theta: float):
    """What the cache holds for fragment ``child``: its keys rotated at their
    canonical positions, and its values (section 5.5: the cached block carries
    the position of its preparation)."""
    sel = np.nonzero(lay.seg == child)[0]
    return rope(np.asarray(k, np.float64)[sel], lay.pos_canon[sel], theta), np.asarray(v, np.float64)[sel]


def allowed_pairs(lay: Layout) -> int:
    """Number of (query, key) pairs the mask allows (the algorithmic work)."""
    P, Ls, Q = lay.prefix_len, lay.frag_lens, lay.cross_len
    pre = P * (P + 1) // 2
    frag = sum(L * P + L * (L + 1) // 2 for L in Ls)
    base = P + sum(Ls)
    cross = Q * base + Q * (Q + 1) // 2
    return pre + frag + cross
