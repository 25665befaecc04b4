"""Oracle for the attention of the parallel multimodal diffusion block: the three
branches and the element-wise sum of their outputs. Plain, exact, fp64, CPU.

TEST INFRASTRUCTURE ONLY, like ref_attention and ref_branches (whose functions it
composes): nothing on the product path imports it.

What it computes (Vchitect-2.0, Sec. III-B "Parallel Transformer Architecture"):
the block runs a full-sequence (joint) attention branch, a spatial branch (each
frame on its own, with the text) and a temporal branch (each spatial position
across the frames), and adds the three branch outputs element-wise to form the
block's attention output. The backward of a sum hands the same output gradient to
every branch; each branch then back-propagates on its own.

Readings (listed in the design notes):
  * the sum is taken of the branch outputs as they leave the attention; per-branch
    projections, if a model has them, lie outside this path;
  * each branch takes its own q, k, v (a model may feed the same tensors to all
    three, in which case their gradients add);
  * the summed output is stored in bf16, rounded to nearest-even once from the sum
    of the three (bf16) branch outputs; `round_bf16` is that rounding.
"""
from __future__ import annotations

import numpy as np

from .ref_attention import attention_backward, attention_forward, key_validity
from .ref_branches import spatial_backward, spatial_forward, temporal_backward, temporal_forward

__all__ = ["BRANCHES", "branch_sum", "round_bf16", "block_forward", "block_backward"]

BRANCHES = ("joint", "spatial", "temporal")


def branch_sum(o_joint=None, o_spatial=None, o_temporal=None) -> np.ndarray:
    """Element-wise sum of the branch outputs in float64; a missing branch counts as zero."""
    parts = [np.asarray(x, dtype=np.float64) for x in (o_joint, o_spatial, o_temporal) if x is not None]
    if not parts:
        raise ValueError("branch_sum needs at least one branch output")
    out = np.zeros_like(parts[0])
    for p in parts:
        out = out + p
    return out


def round_bf16(x) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 (8 significant bits, ties to even),
    returned as float64. Written for the normal range of bfloat16 (magnitudes from 2^-126
    up to its largest finite value); zeros, infinities and NaNs pass through.
    """
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                      # x = m * 2^e, 0.5 <= |m| < 1
    r = np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)  # keep 8 significant bits, half to even
    return np.where(np.isfinite(x) & (x != 0), r, x)


def _branch_inputs(inputs, name):
    q, k, v = inputs[name]
    return q, k, v


def block_forward(inputs, text_slot, frames, text_len=None, key_mask=None, scale=None, threads=None):
    """Forward of the block's attention.

    inputs: {"joint": (q, k, v), "spatial": (q, k, v), "temporal": (q, k, v)}, each
    [B, N, H, D] on the joint layout (N = text_slot + frames * L).
    Returns (out, branches) with out = o_joint + o_spatial + o_temporal (float64, not
    rounded) and branches[name] = (o, lse) of each branch.
    """
    q, k, v = _branch_inputs(inputs, "joint")
    B, N = np.shape(q)[:2]
    joint = attention_forward(q, k, v, key_validity(B, N, text_slot, text_len, key_mask), scale, threads=threads)
    q, k, v = _branch_inputs(inputs, "spatial")
    spatial = spatial_forward(q, k, v, text_slot, frames, text_len, key_mask, scale, threads=threads)
    q, k, v = _branch_inputs(inputs, "temporal")
    temporal = temporal_forward(q, k, v, text_slot, frames, key_mask, scale, threads=threads)
    branches = {"joint": joint, "spatial": spatial, "temporal": temporal}
    return branch_sum(joint[0], spatial[0], temporal[0]), branches


def block_backward(inputs, dout, text_slot, frames, text_len=None, key_mask=None, scale=None,
                   branches=None, threads=None):
    """Backward of the block's attention for the gradient dout of the summed output.

    The sum passes dout unchanged to each branch. Returns {name: (dq, dk, dv)}; with
    shared inputs the caller adds the three.
    """
    lse = {n: (None if branches is None else branches[n][1]) for n in BRANCHES}
    q, k, v = _branch_inputs(inputs, "joint")
    B, N = np.shape(q)[:2]
    gj = attention_backward(q, k, v, dout, key_validity(B, N, text_slot, text_len, key_mask), scale,
                            lse=lse["joint"], threads=threads)
    q, k, v = _branch_inputs(inputs, "spatial")
    gs = spatial_backward(q, k, v, dout, text_slot, frames, text_len, key_mask, scale, lse=lse["spatial"],
                          threads=threads)
    q, k, v = _branch_inputs(inputs, "temporal")
    gt = temporal_backward(q, k, v, dout, text_slot, frames, key_mask, scale, lse=lse["temporal"],
                           threads=threads)
    return {"joint": gj, "spatial": gs, "temporal": gt}
