"""GPU parity of the temporal attention branch (through the C ABI) against the
fp64 branch oracle.

Small shapes are compared on every element, for frame counts that pack one to
sixteen positions into a matrix-core block, position counts that leave a
ragged last block, both head dims, with and without text and a key mask; long
clips (33 to 144 frames, one position per workgroup step, frames in blocks of
32 with a ragged last block) likewise, including positions whose keys are all
masked or all but one. The workload shapes, and a 144-frame clip, are compared
on sampled spatial positions (positions are
independent in this branch, so the oracle runs on the sliced positions only)
plus identities that hold on every head at full size. Tolerances as for the
joint path (parity_util).
"""
import numpy as np
import pytest

import oracle.ref_branches as orb
import workloads as W
from parity_util import assert_close, bf16_values, log, to_gpu_bf16

pytestmark = pytest.mark.gpu


def _run(desc, g, key_mask=None):
    import torch
    import paper_2501_08453_amd as vc
    o, lse = vc.temporal_fwd(g["q"], g["k"], g["v"], desc, key_mask)
    dq, dk, dv = vc.temporal_bwd(g["q"], g["k"], g["v"], o, lse, g["do"], desc, key_mask)
    torch.cuda.synchronize()
    out = {n: bf16_values(t) for n, t in (("o", o), ("dq", dq), ("dk", dk), ("dv", dv))}
    out["lse"] = lse.cpu().numpy().astype(np.float64)
    return out


def _inputs(w, seed):
    x = W.make_inputs(w, seed=seed)
    g = {n: to_gpu_bf16(x[n]) for n in ("q", "k", "v", "do")}
    h = {n: bf16_values(g[n]) for n in g}
    return g, h


SMALL = [
    # (name, batch, heads, head_dim, text_slot, frames, grid_h, grid_w, masked)
    ("F1", 1, 2, 64, 4, 1, 3, 5, False),
    ("F2-ragged", 2, 3, 128, 16, 2, 7, 3, False),
    ("F5-ragged", 1, 2, 64, 0, 5, 4, 5, True),
    ("F8", 2, 2, 128, 8, 8, 4, 4, False),
    ("F16-ragged", 1, 3, 128, 12, 16, 3, 3, True),
    ("F32", 1, 2, 64, 4, 32, 2, 3, False),
    ("F13-d128", 1, 1, 128, 0, 13, 5, 3, True),
    # one position per group with many padding slots, and a ragged last group
    ("F17-masked", 2, 2, 128, 8, 17, 3, 5, True),
    ("F11-d64", 1, 3, 64, 4, 11, 5, 5, False),
    ("F31-d64", 1, 2, 64, 0, 31, 2, 4, True),
]


LONG = [
    # frame counts past one 32-slot block: blocks of 32 with a ragged last one
    ("F33-d64-masked", 1, 2, 64, 8, 33, 3, 5, True),
    ("F37-d128-one-position", 1, 1, 128, 0, 37, 1, 1, True),
    ("F64-d128-masked", 2, 2, 128, 16, 64, 3, 3, True),
    ("F100-d128", 1, 1, 128, 40, 100, 4, 4, False),
    ("F144-d128-masked", 1, 2, 128, 12, 144, 2, 5, True),
    ("F144-d64", 1, 3, 64, 0, 144, 3, 3, False),
    ("F129-d128-one-frame-last-block", 1, 2, 128, 8, 129, 2, 2, True),
    ("F97-d64", 2, 1, 64, 0, 97, 1, 3, False),
]


@pytest.mark.parametrize("case", SMALL + LONG, ids=[c[0] for c in SMALL + LONG])
def test_temporal_small_all_elements(case):
    import torch
    import paper_2501_08453_amd as vc
    name, B, H, D, T, F, gh, gw, masked = case
    w = W.custom(B, H, D, T, F, gh, gw, name=name)
    log("temporal case", name, w.shape)
    g, h = _inputs(w, seed=500 + len(name))
    km_np = None
    km = None
    if masked:
        km_np = W.random_key_mask(w, seed=77, keep=0.8)
        km = torch.from_numpy(km_np).to("cuda")
    desc = vc.desc_for(w)
    out = _run(desc, g, km)
    o, lse = orb.temporal_forward(h["q"], h["k"], h["v"], T, F, km_np)
    dq, dk, dv = orb.temporal_backward(h["q"], h["k"], h["v"], h["do"], T, F, km_np, lse=lse)
    assert_close("O", out["o"], o)
    assert_close("LSE", out["lse"], lse)
    assert_close("dQ", out["dq"], dq)
    assert_close("dK", out["dk"], dk)
    assert_close("dV", out["dv"], dv)
    # text rows exactly zero / -inf
    assert np.all(out["o"][:, :T] == 0) and np.all(np.isneginf(out["lse"][:, :, :T]))
    assert np.all(out["dq"][:, :T] == 0) and np.all(out["dk"][:, :T] == 0) and np.all(out["dv"][:, :T] == 0)


@pytest.mark.parametrize("wid", [2, 3, 4, 5])
def test_temporal_workloads_sampled(wid):
    import torch
    import paper_2501_08453_amd as vc
    w = W.WORKLOADS[wid]
    B, N, H, D = w.shape
    T, F, L = w.text_slot, w.frames, w.grid_h * w.grid_w
    log("temporal workload", w.name, w.shape)
    g, h = _inputs(w, seed=None)
    desc = vc.desc_for(w)
    out = _run(desc, g)
    rng = np.random.Generator(np.random.PCG64(9000 + wid))
    pos = np.sort(rng.choice(L, size=min(L, 48), replace=False))
    pos = np.unique(np.concatenate([pos, [0, L - 1]]))
    rows = (T + np.arange(F)[:, None] * L + pos[None, :]).reshape(-1)  # frame-major, like the layout
    sub = lambda a: a[:, rows]  # noqa: E731
    o, lse = orb.temporal_forward(sub(h["q"]), sub(h["k"]), sub(h["v"]), 0, F)
    dq, dk, dv = orb.temporal_backward(sub(h["q"]), sub(h["k"]), sub(h["v"]), sub(h["do"]), 0, F, lse=lse)
    assert_close("O", sub(out["o"]), o)
    assert_close("LSE", out["lse"][:, :, rows], lse)
    assert_close("dQ", sub(out["dq"]), dq)
    assert_close("dK", sub(out["dk"]), dk)
    assert_close("dV", sub(out["dv"]), dv)
    # identities on every head at full size: sum_j dV_j = sum_i dO_i over the video rows
    # (each video query's probabilities sum to 1) and sum_j dK_j = 0. Each dV_j sums only F
    # rows here, so the bf16 rounding of the outputs and of P (relative 2^-9 per term,
    # independent signs) accumulates like a random walk over the rows: the bound is six
    # standard deviations of that walk, per (sample, head, dim).
    dv_sum = out["dv"].sum(axis=1)
    do_sum = h["do"][:, T:].sum(axis=1)
    walk = 2.0 ** -9 * (np.sqrt((h["do"][:, T:] ** 2).sum(axis=1)) + np.sqrt((out["dv"] ** 2).sum(axis=1)))
    ratio = (np.abs(dv_sum - do_sum) / walk).max()
    err_dk = np.abs(out["dk"].sum(axis=1)).max()
    dk_mag = np.abs(out["dk"]).sum(axis=1).mean()
    log("   |sum dV - sum dO| / rounding walk: max %.2f; |sum dK| max %.3e (sum |dK| ~ %.3e)"
        % (ratio, err_dk, dk_mag))
    assert ratio <= 6.0
    assert err_dk <= 5e-3 * dk_mag
    del torch


def test_temporal_long_clip_masked_positions():
    """A 40-frame clip: position 0 has every key masked (its queries get O = 0, LSE = -inf,
    zero gradients), position 1 a single valid frame (O = that frame's v, LSE = its score,
    dQ = dK = 0), the others a random mask; every element against the oracle."""
    import torch
    import paper_2501_08453_amd as vc
    w = W.custom(1, 2, 128, 8, 40, 2, 3, name="F40-masked-positions")
    T, F, L = w.text_slot, w.frames, w.grid_h * w.grid_w
    g, h = _inputs(w, seed=4040)
    km_np = W.random_key_mask(w, seed=41, keep=0.7)
    frames = T + np.arange(F) * L
    km_np[0, frames + 0] = 0
    km_np[0, frames + 1] = 0
    km_np[0, T + 17 * L + 1] = 1
    km = torch.from_numpy(km_np).to("cuda")
    out = _run(vc.desc_for(w), g, km)
    o, lse = orb.temporal_forward(h["q"], h["k"], h["v"], T, F, km_np)
    dq, dk, dv = orb.temporal_backward(h["q"], h["k"], h["v"], h["do"], T, F, km_np, lse=lse)
    assert np.all(out["o"][0, frames + 0] == 0) and np.all(np.isneginf(out["lse"][0, :, frames + 0]))
    assert np.all(out["dq"][0, frames + 0] == 0) and np.all(out["dk"][0, frames + 0] == 0)
    assert np.all(out["dv"][0, frames + 0] == 0)
    masked1 = np.setdiff1d(frames + 1, [T + 17 * L + 1])  # position 1's masked keys: exact zeros
    assert np.all(out["dk"][0, masked1] == 0) and np.all(out["dv"][0, masked1] == 0)
    for n, a, r in (("O", out["o"], o), ("LSE", out["lse"], lse), ("dQ", out["dq"], dq), ("dK", out["dk"], dk),
                    ("dV", out["dv"], dv)):
        assert_close(n, a, r)


def test_temporal_144_frames_sampled():
    """A 144-frame clip (the paper's longest input length in frames) at a reduced 24x40 grid
    and 4 heads (138,496 tokens): 48 sampled spatial positions of every head against the
    oracle, the gradient-sum identities on every head."""
    import torch
    import paper_2501_08453_amd as vc
    w = W.custom(1, 4, 128, 256, 144, 24, 40, name="clip-144f")
    B, N, H, D = w.shape
    T, F, L = w.text_slot, w.frames, w.grid_h * w.grid_w
    log("temporal 144 frames", w.shape)
    g, h = _inputs(w, seed=144)
    out = _run(vc.desc_for(w), g)
    rng = np.random.Generator(np.random.PCG64(1440))
    pos = np.unique(np.concatenate([rng.choice(L, size=46, replace=False), [0, L - 1]]))
    rows = (T + np.arange(F)[:, None] * L + pos[None, :]).reshape(-1)
    sub = lambda a: a[:, rows]  # noqa: E731
    o, lse = orb.temporal_forward(sub(h["q"]), sub(h["k"]), sub(h["v"]), 0, F)
    dq, dk, dv = orb.temporal_backward(sub(h["q"]), sub(h["k"]), sub(h["v"]), sub(h["do"]), 0, F, lse=lse)
    assert_close("O", sub(out["o"]), o)
    assert_close("LSE", out["lse"][:, :, rows], lse)
    assert_close("dQ", sub(out["dq"]), dq)
    assert_close("dK", sub(out["dk"]), dk)
    assert_close("dV", sub(out["dv"]), dv)
    dv_sum = out["dv"].sum(axis=1)
    do_sum = h["do"][:, T:].sum(axis=1)
    walk = 2.0 ** -9 * (np.sqrt((h["do"][:, T:] ** 2).sum(axis=1)) + np.sqrt((out["dv"] ** 2).sum(axis=1)))
    ratio = (np.abs(dv_sum - do_sum) / walk).max()
    err_dk = np.abs(out["dk"].sum(axis=1)).max()
    dk_mag = np.abs(out["dk"]).sum(axis=1).mean()
    log("   |sum dV - sum dO| / rounding walk: max %.2f; |sum dK| max %.3e (sum |dK| ~ %.3e)"
        % (ratio, err_dk, dk_mag))
    assert ratio <= 6.0
    assert err_dk <= 5e-3 * dk_mag
    del torch


def test_temporal_deterministic_and_text_independent():
    import torch
    import paper_2501_08453_amd as vc
    w = W.custom(1, 2, 128, 24, 8, 6, 5)
    g, h = _inputs(w, seed=1234)
    desc = vc.desc_for(w)
    a = _run(desc, g)
    b = _run(desc, g)
    for n in a:
        np.testing.assert_array_equal(a[n], b[n])
    # text tokens take no part: changing them changes nothing
    g2 = dict(g)
    for n in ("q", "k", "v"):
        t = g[n].clone()
        t[:, :w.text_slot] = 3.0
        g2[n] = t
    c = _run(desc, g2)
    for n in a:
        np.testing.assert_array_equal(a[n], c[n])
    del torch
