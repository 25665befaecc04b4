"""GPU parity of the spatial attention branch (through the C ABI) against the
fp64 branch oracle.

Small shapes are compared on every element, with frame lengths that put frame
boundaries inside 64-token tiles, text slots that are not tile multiples (so
workgroups mix text and video queries), ragged text, key masks, both head dims
and batches above one. The workload shapes are compared frame by frame on
sampled frames and heads: a frame's video rows (O, LSE, dQ) and video keys
(dK, dV) depend only on that frame and the text, so the oracle runs on the
text + frame sequence alone; text-key gradients sum the contributions of every
frame (one head). Tolerances as for the joint path (parity_util).
"""
import numpy as np
import pytest

import oracle.ref_branches as orb
import workloads as W
from parity_util import assert_close, bf16_values, log, to_gpu_bf16

pytestmark = pytest.mark.gpu


def _run(desc, g, text_len=None, key_mask=None):
    import torch
    import paper_2501_08453_amd as vc
    o, lse = vc.spatial_fwd(g["q"], g["k"], g["v"], desc, text_len, key_mask)
    dq, dk, dv = vc.spatial_bwd(g["q"], g["k"], g["v"], o, lse, g["do"], desc, text_len, key_mask)
    torch.cuda.synchronize()
    out = {n: bf16_values(t) for n, t in (("o", o), ("dq", dq), ("dk", dk), ("dv", dv))}
    out["lse"] = lse.cpu().numpy().astype(np.float64)
    return out


def _inputs(w, seed):
    import torch
    x = W.make_inputs(w, seed=seed)
    g = {n: to_gpu_bf16(x[n]) for n in ("q", "k", "v", "do")}
    h = {n: bf16_values(g[n]) for n in g}
    tl = x["text_len"]
    return g, h, tl, (None if tl is None else torch.from_numpy(tl).to("cuda"))


SMALL = [
    # (name, batch, heads, head_dim, text_slot, frames, grid_h, grid_w, ragged, masked)
    ("T0-F3-L50", 1, 2, 64, 0, 3, 5, 10, False, False),
    ("T16-F4-L100", 2, 2, 128, 16, 4, 10, 10, True, False),
    ("T100-F2-L130", 1, 3, 64, 100, 2, 10, 13, False, True),
    ("T256-F5-L64", 1, 2, 128, 256, 5, 8, 8, True, False),
    ("T40-F1-L200", 2, 1, 128, 40, 1, 10, 20, False, True),
    ("T8-F7-L33", 1, 2, 64, 8, 7, 3, 11, True, True),
    # text key blocks whose video query tiles are split over several workgroups (fp32
    # partials summed afterwards): 2 chunks; 2 text blocks, the second holding video keys
    # of three frames; 3 chunks with a batch of 2
    ("T100-F12-L60-split", 1, 2, 64, 100, 12, 6, 10, True, True),
    ("T300-F9-L100-split", 1, 2, 128, 300, 9, 10, 10, True, False),
    ("T64-F40-L30-split", 2, 1, 64, 64, 40, 5, 6, False, False),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_spatial_small_all_elements(case):
    import torch
    import paper_2501_08453_amd as vc
    name, B, H, D, T, F, gh, gw, ragged, masked = case
    w = W.custom(B, H, D, T, F, gh, gw, name=name, ragged_text=ragged)
    log("spatial case", name, w.shape)
    g, h, tl, tl_d = _inputs(w, seed=600 + len(name))
    km_np = W.random_key_mask(w, seed=88, keep=0.85) if masked else None
    km = None if km_np is None else torch.from_numpy(km_np).to("cuda")
    desc = vc.desc_for(w)
    split = vc.vc_spatialattn_bwd_workspace_bytes(desc) > vc.vc_jointattn_bwd_workspace_bytes(desc)
    assert split == name.endswith("-split")
    out = _run(desc, g, tl_d, km)
    o, lse = orb.spatial_forward(h["q"], h["k"], h["v"], T, F, tl, km_np)
    dq, dk, dv = orb.spatial_backward(h["q"], h["k"], h["v"], h["do"], T, F, tl, km_np, lse=lse)
    assert_close("O", out["o"], o)
    assert_close("LSE", out["lse"], lse)
    assert_close("dQ", out["dq"], dq)
    assert_close("dK", out["dk"], dk)
    assert_close("dV", out["dv"], dv)
    assert np.all(out["o"][:, :T] == 0) and np.all(np.isneginf(out["lse"][:, :, :T]))
    assert np.all(out["dq"][:, :T] == 0)


def _frame_view(a, T, L, f):
    """[B, T + L, H, D]: the text slot followed by frame f."""
    return np.concatenate([a[:, :T], a[:, T + f * L:T + (f + 1) * L]], axis=1)


@pytest.mark.parametrize("wid", [2, 3, 4, 5])
def test_spatial_workloads_sampled(wid):
    import paper_2501_08453_amd as vc
    w = W.WORKLOADS[wid]
    B, N, H, D = w.shape
    T, F, L = w.text_slot, w.frames, w.grid_h * w.grid_w
    log("spatial workload", w.name, w.shape)
    g, h, tl, tl_d = _inputs(w, seed=None)
    desc = vc.desc_for(w)
    out = _run(desc, g, tl_d)
    heads = [0, H - 1]
    frames = sorted({0, F // 2, F - 1})
    got = {n: [] for n in ("o", "lse", "dq", "dk", "dv")}
    ref = {n: [] for n in got}
    for f in frames:
        rows = slice(T + f * L, T + (f + 1) * L)
        sub = {n: _frame_view(h[n], T, L, f)[:, :, heads] for n in h}
        o, lse = orb.spatial_forward(sub["q"], sub["k"], sub["v"], T, 1, tl)
        dq, dk, dv = orb.spatial_backward(sub["q"], sub["k"], sub["v"], sub["do"], T, 1, tl, lse=lse)
        for n, r in (("o", o), ("dq", dq), ("dk", dk), ("dv", dv)):
            got[n].append(out[n][:, rows][:, :, heads])
            ref[n].append(r[:, T:])
        got["lse"].append(out["lse"][:, heads][:, :, rows])
        ref["lse"].append(lse[:, :, T:])
        log("   frame", f, "oracle done")
    for n in got:
        assert_close(n, np.concatenate(got[n], axis=1 if n != "lse" else 2),
                     np.concatenate(ref[n], axis=1 if n != "lse" else 2))
    # text keys collect gradients from every frame: head 0, all frames
    if T > 0:
        dk_t = np.zeros((B, T, 1, D))
        dv_t = np.zeros((B, T, 1, D))
        for f in range(F):
            sub = {n: _frame_view(h[n], T, L, f)[:, :, :1] for n in h}
            _, lse = orb.spatial_forward(sub["q"], sub["k"], sub["v"], T, 1, tl)
            _, dk, dv = orb.spatial_backward(sub["q"], sub["k"], sub["v"], sub["do"], T, 1, tl, lse=lse)
            dk_t += dk[:, :T]
            dv_t += dv[:, :T]
        assert_close("dK text", out["dk"][:, :T, :1], dk_t)
        assert_close("dV text", out["dv"][:, :T, :1], dv_t)


def test_spatial_frame_independence_and_joint_reduction():
    """One frame: the spatial branch equals the joint branch on the video rows; and
    changing another frame's tokens leaves a frame's outputs bit-identical."""
    import paper_2501_08453_amd as vc
    w1 = W.custom(1, 2, 128, 64, 1, 10, 20)
    g, h, _, _ = _inputs(w1, seed=4321)
    desc = vc.desc_for(w1)
    sp = _run(desc, g)
    o_j, lse_j = vc.fwd(g["q"], g["k"], g["v"], desc)
    np.testing.assert_array_equal(sp["o"][:, 64:], bf16_values(o_j)[:, 64:])
    np.testing.assert_array_equal(sp["lse"][:, :, 64:], lse_j.cpu().numpy()[:, :, 64:])
    w = W.custom(1, 2, 64, 32, 3, 6, 10)
    g, h, _, _ = _inputs(w, seed=99)
    desc = vc.desc_for(w)
    a = _run(desc, g)
    g2 = dict(g)
    L = 60
    for n in ("q", "k", "v"):
        t = g[n].clone()
        t[:, 32 + 2 * L:] = 2.0  # frame 2
        g2[n] = t
    b = _run(desc, g2)
    np.testing.assert_array_equal(a["o"][:, :32 + 2 * L], b["o"][:, :32 + 2 * L])
    np.testing.assert_array_equal(a["lse"][:, :, :32 + 2 * L], b["lse"][:, :, :32 + 2 * L])
