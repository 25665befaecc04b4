"""Oracle for the spatial and temporal attention branches: plain, exact, fp64, CPU.

TEST INFRASTRUCTURE ONLY, like ref_attention (whose per-head building blocks
it reuses): nothing on the product path imports it.

What it computes (Vchitect-2.0, Sec. III-B "Parallel Transformer
Architecture"): besides the full-sequence branch, the multimodal diffusion
block has a spatial and a temporal attention branch, obtained by regrouping
the video tokens of the [B, F, L, ...] video sequence (F frames of L tokens):
spatial attention runs on [B*F, L, ...] (each frame on its own) and temporal
attention on [B*L, F, ...] (each spatial position across the frames); the
three branch outputs are then added element-wise. The spatial branch also
attends to the text tokens, which join each frame's key set (Sec. V-B,
intra-node sequence-parallel workflow, where text is sharded together with the
spatial sequence for that reason).

Both branches act on the joint layout [B, N, H, D], N = T + F*L, with the
text slot first and video tokens frame-major (token T + f*L + l is frame f,
spatial position l), so no regrouped copy is ever made:

  spatial:  a video query of frame f attends to the valid text keys and to the
            keys of frame f;
  temporal: a video query at (f, l) attends to the keys (f', l), f' = 0..F-1.

Readings of points the paper leaves open (each is listed in the design notes):
  * only video tokens are queries of these branches; text rows of their
    outputs are O = 0, LSE = -inf and get no gradient from them (the text
    keys of the spatial branch still receive dK, dV);
  * key validity is that of the joint branch (padded text keys and keys with
    key_mask == 0 are excluded); the temporal branch has no text keys;
  * scale c = 1/sqrt(D) by default, exact softmax, no positional term.

Every function evaluates exact attention per (sample, group, head) with the
same two-pass definition as ref_attention; results are float64.
"""
from __future__ import annotations

import numpy as np

from .ref_attention import (_BlasOne, _as64, _head_backward, _head_forward, _pool_map, default_scale,
                            host_threads, key_validity)

__all__ = ["spatial_forward", "spatial_backward", "temporal_forward", "temporal_backward"]


def _frame_keys(text_slot: int, frame_len: int, f: int) -> np.ndarray:
    """Key positions of frame f's spatial sequence: the text slot, then the frame."""
    t0 = text_slot + f * frame_len
    return np.concatenate([np.arange(text_slot), np.arange(t0, t0 + frame_len)])


def _prep(q, k, v, text_slot, frames, text_len, key_mask, scale):
    q, k, v = _as64(q), _as64(k), _as64(v)
    B, N, H, D = q.shape
    assert (N - text_slot) % frames == 0, "video tokens must split into whole frames"
    L = (N - text_slot) // frames
    valid = key_validity(B, N, text_slot, text_len, key_mask)
    scale = default_scale(D) if scale is None else float(scale)
    return q, k, v, B, N, H, D, L, valid, scale


def spatial_forward(q, k, v, text_slot, frames, text_len=None, key_mask=None, scale=None, threads=None):
    """Spatial branch forward. Returns (o [B,N,H,D], lse [B,H,N]); text rows 0 / -inf."""
    q, k, v, B, N, H, D, L, valid, scale = _prep(q, k, v, text_slot, frames, text_len, key_mask, scale)
    threads = host_threads() if threads is None else threads
    o = np.zeros_like(q)
    lse = np.full((B, H, N), -np.inf)
    items = [(b, f, h) for b in range(B) for f in range(frames) for h in range(H)]

    def one(it):
        b, f, h = it
        keys = _frame_keys(text_slot, L, f)
        rows = np.arange(text_slot + f * L, text_slot + (f + 1) * L)
        return _head_forward(q[b, rows, h], k[b, keys, h], v[b, keys, h], valid[b, keys], scale)

    with _BlasOne():
        outs = _pool_map(one, items, threads)
    for (b, f, h), (oh, lh) in zip(items, outs):
        rows = slice(text_slot + f * L, text_slot + (f + 1) * L)
        o[b, rows, h] = oh
        lse[b, h, rows] = lh
    return o, lse


def spatial_backward(q, k, v, do, text_slot, frames, text_len=None, key_mask=None, scale=None, lse=None,
                     threads=None):
    """Spatial branch backward. Returns (dq, dk, dv) [B,N,H,D]; text keys collect the
    contributions of every frame (summed in frame order)."""
    q, k, v, B, N, H, D, L, valid, scale = _prep(q, k, v, text_slot, frames, text_len, key_mask, scale)
    do = _as64(do)
    threads = host_threads() if threads is None else threads
    if lse is None:
        _, lse = spatial_forward(q, k, v, text_slot, frames, text_len, key_mask, scale, threads)
    dq, dk, dv = (np.zeros_like(q) for _ in range(3))
    items = [(b, f, h) for b in range(B) for f in range(frames) for h in range(H)]

    def one(it):
        b, f, h = it
        keys = _frame_keys(text_slot, L, f)
        rows = np.arange(text_slot + f * L, text_slot + (f + 1) * L)
        return _head_backward(q[b, rows, h], k[b, keys, h], v[b, keys, h], do[b, rows, h], valid[b, keys], scale,
                              lse[b, h, rows])

    with _BlasOne():
        outs = _pool_map(one, items, threads)
    for (b, f, h), (a, bk, c) in zip(items, outs):
        keys = _frame_keys(text_slot, L, f)
        rows = slice(text_slot + f * L, text_slot + (f + 1) * L)
        dq[b, rows, h] = a
        dk[b, keys, h] += bk
        dv[b, keys, h] += c
    return dq, dk, dv


def _temporal_tokens(text_slot: int, frames: int, frame_len: int, l: int) -> np.ndarray:
    """Positions of spatial location l in every frame (the temporal sequence of l)."""
    return text_slot + np.arange(frames) * frame_len + l


def temporal_forward(q, k, v, text_slot, frames, key_mask=None, scale=None, threads=None):
    """Temporal branch forward. Returns (o [B,N,H,D], lse [B,H,N]); text rows 0 / -inf."""
    q, k, v, B, N, H, D, L, valid, scale = _prep(q, k, v, text_slot, frames, None, key_mask, scale)
    threads = host_threads() if threads is None else threads
    o = np.zeros_like(q)
    lse = np.full((B, H, N), -np.inf)
    items = [(b, l, h) for b in range(B) for l in range(L) for h in range(H)]

    def one(it):
        b, l, h = it
        t = _temporal_tokens(text_slot, frames, L, l)
        return _head_forward(q[b, t, h], k[b, t, h], v[b, t, h], valid[b, t], scale)

    with _BlasOne():
        outs = _pool_map(one, items, threads)
    for (b, l, h), (oh, lh) in zip(items, outs):
        t = _temporal_tokens(text_slot, frames, L, l)
        o[b, t, h] = oh
        lse[b, h, t] = lh
    return o, lse


def temporal_backward(q, k, v, do, text_slot, frames, key_mask=None, scale=None, lse=None, threads=None):
    """Temporal branch backward. Returns (dq, dk, dv) [B,N,H,D]; text rows zero."""
    q, k, v, B, N, H, D, L, valid, scale = _prep(q, k, v, text_slot, frames, None, key_mask, scale)
    do = _as64(do)
    threads = host_threads() if threads is None else threads
    if lse is None:
        _, lse = temporal_forward(q, k, v, text_slot, frames, key_mask, scale, threads)
    dq, dk, dv = (np.zeros_like(q) for _ in range(3))
    items = [(b, l, h) for b in range(B) for l in range(L) for h in range(H)]

    def one(it):
        b, l, h = it
        t = _temporal_tokens(text_slot, frames, L, l)
        return _head_backward(q[b, t, h], k[b, t, h], v[b, t, h], do[b, t, h], valid[b, t], scale, lse[b, h, t])

    with _BlasOne():
        outs = _pool_map(one, items, threads)
    for (b, l, h), (a, bk, c) in zip(items, outs):
        t = _temporal_tokens(text_slot, frames, L, l)
        dq[b, t, h] = a
        dk[b, t, h] = bk
        dv[b, t, h] = c
    return dq, dk, dv
