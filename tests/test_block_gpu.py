"""GPU parity of the block's branch sum (through the C ABI) against the fp64 block
oracle: the standalone sum, the sum fused into the temporal forward, and the block
backward (every branch takes the same output gradient).

Small shapes are compared on every element. The standalone sum is also held to the
exact rounding of the fp64 sum of its (bf16) inputs, which the oracle's round_bf16
defines: identical for inputs of like magnitude; where their exponents lie far apart
and the terms cancel, within one bf16 spacing plus the error bound of summing in fp32.
At the long workload the fused sum
must equal the standalone one bit for bit, and sampled rows (text rows, video rows of
the first and last frame at several positions, two heads) are compared with the
three branch oracles summed.
"""
import numpy as np
import pytest

import oracle.ref_attention as ora
import oracle.ref_block as obl
import oracle.ref_branches as orb
import workloads as W
from parity_util import MAX_ABS, assert_close, bf16_values, log, to_gpu_bf16

pytestmark = pytest.mark.gpu


def _bf16_spacing(x):
    """Spacing of bf16 numbers at |x| (normal range)."""
    _, e = np.frexp(np.abs(x))
    return np.ldexp(1.0, e - 8)


def test_branch_sum_rounds_the_exact_sum():
    import torch
    import paper_2501_08453_amd as vc
    w = W.custom(2, 3, 64, 10, 3, 4, 5)
    desc = vc.desc_for(w)
    rng = np.random.Generator(np.random.PCG64(77))
    g = []
    for _ in range(3):
        x = rng.standard_normal(w.shape) * np.exp(rng.uniform(-8, 8, w.shape))
        g.append(to_gpu_bf16(x.astype(np.float32)))
    h = [bf16_values(t) for t in g]
    out = bf16_values(vc.branch_sum(desc, *g))
    ref = obl.round_bf16(obl.branch_sum(*h))
    diff = np.abs(out - ref)
    same = float((diff == 0).mean())
    # summing in fp32 rounds (a + b) and then (a + b) + c, each by at most 2^-24 of its
    # magnitude; where the terms cancel, that error is not small next to the result
    fp32_err = 2.0 ** -23 * (np.abs(h[0]) + np.abs(h[1]) + np.abs(h[2]))
    log("   identical %.6f, max diff / (spacing + fp32 bound) %.2f"
        % (same, (diff / (_bf16_spacing(ref) + fp32_err)).max()))
    assert same > 0.999
    assert np.all(diff <= _bf16_spacing(ref) + fp32_err)
    # branch outputs of like magnitude (as attention outputs are): the exact rounding
    y = [to_gpu_bf16((0.05 * rng.standard_normal(w.shape)).astype(np.float32)) for _ in range(3)]
    hy = [bf16_values(t) for t in y]
    np.testing.assert_array_equal(bf16_values(vc.branch_sum(desc, *y)), obl.round_bf16(obl.branch_sum(*hy)))
    # missing branches count as zero; one input is returned unchanged
    np.testing.assert_array_equal(bf16_values(vc.branch_sum(desc, None, None, g[2])), h[2])
    two = bf16_values(vc.branch_sum(desc, g[0], None, g[2]))
    ref2 = obl.round_bf16(obl.branch_sum(h[0], None, h[2]))
    assert np.all(np.abs(two - ref2) <= _bf16_spacing(ref2) + 2.0 ** -23 * (np.abs(h[0]) + np.abs(h[2])))
    # in place: out is the first input
    acc = g[0].clone()
    vc.vc_branchsum(desc, acc, g[1], g[2], acc)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(bf16_values(acc), out)


SMALL = [
    # (name, batch, heads, head_dim, text_slot, frames, grid_h, grid_w, ragged, masked)
    ("T16-F4-L20", 1, 2, 64, 16, 4, 4, 5, False, False),
    ("T100-F3-L70-ragged", 2, 2, 128, 100, 3, 7, 10, True, False),
    ("T8-F8-L33-masked", 1, 3, 64, 8, 8, 3, 11, True, True),
    ("T0-F5-L64", 1, 2, 128, 0, 5, 8, 8, False, False),
    ("T24-F40-L12-masked", 1, 2, 128, 24, 40, 3, 4, True, True),  # temporal: long-clip kernel
]


def _branch_inputs(w, seed):
    """Separate q, k, v for each branch (on the GPU) and their exact values (host)."""
    g, h = {}, {}
    for j, name in enumerate(obl.BRANCHES):
        x = W.make_inputs(w, seed=seed + 10 * j)
        g[name] = tuple(to_gpu_bf16(x[n]) for n in ("q", "k", "v"))
        h[name] = tuple(bf16_values(t) for t in g[name])
        if j == 0:
            tl = x["text_len"]
            g["do"] = to_gpu_bf16(x["do"])
            h["do"] = bf16_values(g["do"])
    return g, h, tl


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_fused_temporal_sum(case):
    import torch
    import paper_2501_08453_amd as vc
    name, B, H, D, T, F, gh, gw, ragged, masked = case
    w = W.custom(B, H, D, T, F, gh, gw, name=name, ragged_text=ragged)
    log("block case", name, w.shape)
    g, h, tl = _branch_inputs(w, seed=900 + len(name))
    tl_d = None if tl is None else torch.from_numpy(tl).to("cuda")
    km_np = W.random_key_mask(w, seed=31, keep=0.85) if masked else None
    km = None if km_np is None else torch.from_numpy(km_np).to("cuda")
    desc = vc.desc_for(w)
    o_j, _ = vc.fwd(*g["joint"], desc, text_len=tl_d, key_mask=km)
    o_s, _ = vc.spatial_fwd(*g["spatial"], desc, tl_d, km)
    o_t, lse_t, out = vc.temporal_fwd_sum(*g["temporal"], desc, o_joint=o_j, o_spatial=o_s, key_mask=km)
    o_t0, lse_t0 = vc.temporal_fwd(*g["temporal"], desc, km)
    standalone = vc.branch_sum(desc, o_j, o_s, o_t0)
    # the fused pass writes the same temporal output and exactly the standalone sum
    np.testing.assert_array_equal(bf16_values(o_t), bf16_values(o_t0))
    np.testing.assert_array_equal(lse_t.cpu().numpy(), lse_t0.cpu().numpy())
    np.testing.assert_array_equal(bf16_values(out), bf16_values(standalone))
    # accumulating into the joint output's buffer gives the same
    acc = o_j.clone()
    vc.vc_temporalattn_fwd_sum(desc, *g["temporal"], km, acc, o_s, o_t, lse_t, acc)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(bf16_values(acc), bf16_values(out))
    ref, _ = obl.block_forward({n: h[n] for n in obl.BRANCHES}, T, F, tl, km_np)
    assert_close("sum", bf16_values(out), ref)


@pytest.mark.parametrize("case", SMALL[:3], ids=[c[0] for c in SMALL[:3]])
def test_block_backward_shared_inputs(case):
    """One set of q, k, v feeds all three branches; the block's input gradients are the
    sums of the branches' gradients for the same dout."""
    import torch
    import paper_2501_08453_amd as vc
    name, B, H, D, T, F, gh, gw, ragged, masked = case
    w = W.custom(B, H, D, T, F, gh, gw, name=name, ragged_text=ragged)
    x = W.make_inputs(w, seed=321 + len(name))
    q, k, v, do = (to_gpu_bf16(x[n]) for n in ("q", "k", "v", "do"))
    tl = x["text_len"]
    tl_d = None if tl is None else torch.from_numpy(tl).to("cuda")
    km_np = W.random_key_mask(w, seed=32, keep=0.85) if masked else None
    km = None if km_np is None else torch.from_numpy(km_np).to("cuda")
    desc = vc.desc_for(w)
    o_j, l_j = vc.fwd(q, k, v, desc, text_len=tl_d, key_mask=km)
    o_s, l_s = vc.spatial_fwd(q, k, v, desc, tl_d, km)
    o_t, l_t, out = vc.temporal_fwd_sum(q, k, v, desc, o_joint=o_j, o_spatial=o_s, key_mask=km)
    gj = vc.bwd(q, k, v, o_j, l_j, do, desc, text_len=tl_d, key_mask=km)
    gs = vc.spatial_bwd(q, k, v, o_s, l_s, do, desc, tl_d, km)
    gt = vc.temporal_bwd(q, k, v, o_t, l_t, do, desc, km)
    torch.cuda.synchronize()
    got = [sum(bf16_values(gr[i]) for gr in (gj, gs, gt)) for i in range(3)]
    hq, hk, hv, hdo = (bf16_values(t) for t in (q, k, v, do))
    inputs = {n: (hq, hk, hv) for n in obl.BRANCHES}
    ref_out, br = obl.block_forward(inputs, T, F, tl, km_np)
    ref = obl.block_backward(inputs, hdo, T, F, tl, km_np, branches=br)
    assert_close("sum", bf16_values(out), ref_out)
    for i, n in enumerate(("dQ", "dK", "dV")):
        assert_close(n, got[i], sum(ref[b][i] for b in obl.BRANCHES))


def test_block_sum_long_workload_sampled():
    import torch
    import paper_2501_08453_amd as vc
    w = W.WORKLOADS[3]
    B, N, H, D = w.shape
    T, F, L = w.text_slot, w.frames, w.grid_h * w.grid_w
    log("block long workload", w.shape)
    x = W.make_inputs(w, with_do=False)
    q, k, v = (to_gpu_bf16(x[n]) for n in ("q", "k", "v"))
    del x
    desc = vc.desc_for(w)
    o_j, _ = vc.fwd(q, k, v, desc)
    o_s, _ = vc.spatial_fwd(q, k, v, desc)
    o_t, _, out = vc.temporal_fwd_sum(q, k, v, desc, o_joint=o_j, o_spatial=o_s)
    standalone = vc.branch_sum(desc, o_j, o_s, o_t)
    torch.cuda.synchronize()
    assert torch.equal(out, standalone)
    log("   fused sum equals the standalone sum over all", out.numel(), "elements")
    rng = np.random.Generator(np.random.PCG64(4242))
    pos = np.unique(np.r_[0, L - 1, rng.integers(0, L, 6)])
    frames = [0, F - 1]
    text_rows = np.array([0, T // 2, T - 1])
    video_rows = (T + np.array(frames)[:, None] * L + pos[None, :]).reshape(-1)
    rows = np.r_[text_rows, video_rows]
    rows_t = torch.from_numpy(rows).to("cuda")
    c = ora.default_scale(D)
    valid = ora.key_validity(B, N, T, None)
    got, ref = [], []
    for h in (0, H - 1):
        qh, kh, vh = (bf16_values(t[:, :, h:h + 1]) for t in (q, k, v))
        o_jr, _ = ora.forward_rows(qh, kh, vh, valid[0], c, 0, 0, rows)
        o_sr = np.zeros_like(o_jr)
        o_tr = np.zeros_like(o_jr)
        for f in frames:  # spatial: text + frame f alone
            sub = [np.concatenate([a[:, :T], a[:, T + f * L:T + (f + 1) * L]], axis=1) for a in (qh, kh, vh)]
            o_f, _ = orb.spatial_forward(*sub, T, 1)
            for i, r in enumerate(rows):
                if T + f * L <= r < T + (f + 1) * L:
                    o_sr[i] = o_f[0, T + r - (T + f * L), 0]
        for p in pos:  # temporal: the F tokens of position p alone
            idx = T + np.arange(F) * L + p
            o_p, _ = orb.temporal_forward(*(a[:, idx] for a in (qh, kh, vh)), 0, F)
            for i, r in enumerate(rows):
                if r >= T and (r - T) % L == p:
                    o_tr[i] = o_p[0, (r - T) // L, 0]
        ref.append(obl.branch_sum(o_jr, o_sr, o_tr))
        got.append(bf16_values(out[0, :, h].index_select(0, rows_t)))
        log("   head", h, "oracle done")
    assert_close("sum", np.concatenate(got), np.concatenate(ref))


def test_autograd_wrappers():
    """The differentiable wrappers give what the direct calls give, bit for bit (the
    deterministic backward, so that no dQ is summed by atomics): each branch alone, and the
    block, whose output is the fused sum and whose input gradients are the branch sums of
    the three branches' gradients. The block's are also compared with the block oracle: a
    gradient is then bf16(g_joint + g_spatial + g_temporal) of three bf16 results, so its
    max-abs bound is the sum of the three results' own bounds plus half a bf16 spacing of
    the sum (mean-rel keeps its bar)."""
    import torch
    import paper_2501_08453_amd as vc
    w = W.custom(1, 2, 128, 24, 40, 3, 4, name="autograd", ragged_text=True)  # long-clip temporal
    x = W.make_inputs(w, seed=77)
    q, k, v, do = (to_gpu_bf16(x[n]) for n in ("q", "k", "v", "do"))
    tl = x["text_len"]
    tl_d = torch.from_numpy(tl).to("cuda")
    km_np = W.random_key_mask(w, seed=5, keep=0.9)
    km = torch.from_numpy(km_np).to("cuda")
    desc = vc.desc_for(w, deterministic=True)

    def run(f, *extra):
        leaves = [t.clone().requires_grad_(True) for t in (q, k, v)]
        out = f(*leaves, desc, *extra)
        out.backward(do)
        torch.cuda.synchronize()
        return out.detach(), [t.grad for t in leaves]

    direct = {
        "joint": (vc.joint_attention, (tl_d, km), lambda: vc.fwd(q, k, v, desc, tl_d, km),
                  lambda o, l: vc.bwd(q, k, v, o, l, do, desc, tl_d, km)),
        "spatial": (vc.spatial_attention, (tl_d, km), lambda: vc.spatial_fwd(q, k, v, desc, tl_d, km),
                    lambda o, l: vc.spatial_bwd(q, k, v, o, l, do, desc, tl_d, km)),
        "temporal": (vc.temporal_attention, (km,), lambda: vc.temporal_fwd(q, k, v, desc, km),
                     lambda o, l: vc.temporal_bwd(q, k, v, o, l, do, desc, km)),
    }
    grads = {}
    for name, (wrap, extra, f, b) in direct.items():
        out, g = run(wrap, *extra)
        o_d, l_d = f()
        g_d = b(o_d, l_d)
        torch.cuda.synchronize()
        assert torch.equal(out, o_d), name
        for t, r, n in zip(g, g_d, ("dq", "dk", "dv")):
            assert torch.equal(t, r), (name, n)
        grads[name] = g_d
        log("   wrapper", name, "equals the direct calls")

    out, g = run(vc.parallel_block_attention, tl_d, km)
    o_j, _ = vc.fwd(q, k, v, desc, tl_d, km)
    o_s, _ = vc.spatial_fwd(q, k, v, desc, tl_d, km)
    _, _, out_d = vc.temporal_fwd_sum(q, k, v, desc, o_joint=o_j, o_spatial=o_s, key_mask=km)
    torch.cuda.synchronize()
    assert torch.equal(out, out_d)
    for i, n in enumerate(("dq", "dk", "dv")):
        s = vc.branch_sum(desc, *(grads[b][i] for b in ("joint", "spatial", "temporal")))
        torch.cuda.synchronize()
        assert torch.equal(g[i], s), n
    hq, hk, hv, hdo = (bf16_values(t) for t in (q, k, v, do))
    inputs = {n: (hq, hk, hv) for n in obl.BRANCHES}
    T, F = w.text_slot, w.frames
    ref_out, br = obl.block_forward(inputs, T, F, tl, km_np)
    ref = obl.block_backward(inputs, hdo, T, F, tl, km_np, branches=br)
    assert_close("block out", bf16_values(out), ref_out)
    for i, n in enumerate(("dQ", "dK", "dV")):
        total = sum(ref[b][i] for b in obl.BRANCHES)
        bound = sum(max(MAX_ABS, float(_bf16_spacing(np.max(np.abs(ref[b][i]))))) for b in obl.BRANCHES)
        bound += 0.5 * float(_bf16_spacing(np.max(np.abs(total))))
        assert_close("block " + n, bf16_values(g[i]), total, max_abs=bound)
