"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Small shapes are compared on every element; the full-size workloads on the
oracle's sampled rows (queries) and columns (keys) of chosen heads, plus
identities that hold at any size on every head. Tolerances are in
parity_util (max-abs 2e-2, L1 mean-relative 5e-3 per output tensor).
"""
import zlib

import numpy as np
import pytest

import oracle.ref_attention as ora
import workloads as W
from parity_util import assert_close, bf16_values, log, run_gpu, to_gpu_bf16

pytestmark = pytest.mark.gpu


def _vc():
    import paper_2501_08453_amd as vc
    return vc


def _inputs_on_gpu(x):
    import torch
    g = {n: to_gpu_bf16(x[n]) for n in ("q", "k", "v", "do")}
    g["text_len"] = None if x["text_len"] is None else torch.from_numpy(x["text_len"]).to("cuda")
    return g


def _full_compare(w, x, scale=None, key_mask=None, use_bf16_oracle=True, heads=None, samples=None, det=False):
    """Whole-tensor comparison on the given (sample, head) pairs (all if None). det: the
    deterministic backward (separate dQ pass) instead of the default fused one."""
    import torch
    vc = _vc()
    g = _inputs_on_gpu(x)
    km = None if key_mask is None else torch.from_numpy(key_mask).to("cuda")
    desc = vc.desc_for(w, scale, deterministic=det)
    out = run_gpu(desc, g["q"], g["k"], g["v"], g["do"], g["text_len"], km)
    if use_bf16_oracle:
        q, k, v, do = (bf16_values(g[n]) for n in ("q", "k", "v", "do"))
    else:
        q, k, v, do = (x[n].astype(np.float64) for n in ("q", "k", "v", "do"))
    B, N, H, D = w.shape
    valid = ora.key_validity(B, N, w.text_slot, x["text_len"], key_mask)
    c = ora.default_scale(D) if scale is None else scale
    bs = range(B) if samples is None else samples
    hs = range(H) if heads is None else heads
    sel = (list(bs), list(hs))
    qs, ks, vs, dos = (a[sel[0]][:, :, sel[1]] for a in (q, k, v, do))
    o, lse = ora.attention_forward(qs, ks, vs, valid[sel[0]], c)
    dq, dk, dv = ora.attention_backward(qs, ks, vs, dos, valid[sel[0]], c, lse=lse)
    pick = lambda a: a[sel[0]][:, :, sel[1]]  # noqa: E731
    assert_close("O", pick(out["o"]), o)
    assert_close("LSE", out["lse"][sel[0]][:, sel[1]], lse)
    assert_close("dQ", pick(out["dq"]), dq)
    assert_close("dK", pick(out["dk"]), dk)
    assert_close("dV", pick(out["dv"]), dv)
    return out, valid


MODES = [False, True]
MODE_IDS = ["fused", "deterministic"]


def _same_up_to_order(a, b, what=""):
    """Two backward results that differ only in the order of their fp32 sums (atomics in
    the fused dQ; the order of query tiles; dP - D formed as (-D + dO V^T) or as
    (dO V^T) - D, which can flip the bf16 rounding of a dS term): elementwise within two
    bf16 spacings plus 2^-7 of the tensor's rms (where terms cancel, a small result moves by
    much more than its own spacing), and within 2^-8 of its mean magnitude on average."""
    d = np.abs(a - b)
    spacing = np.ldexp(1.0, np.frexp(np.maximum(np.abs(a), np.abs(b)))[1] - 8)
    rms = float(np.sqrt(np.mean(b * b)))
    bound = 2 * spacing + 2.0 ** -7 * rms
    log("   %s: max diff / bound %.3f, mean diff / mean |b| %.2e, identical %.4f"
        % (what, (d / bound).max(), d.mean() / max(np.abs(b).mean(), 1e-30), float((d == 0).mean())))
    return bool(np.all(d <= bound) and d.mean() <= 2.0 ** -8 * np.abs(b).mean())


@pytest.mark.parametrize("det", MODES, ids=MODE_IDS)
def test_split_tail_of_last_round_head_dim_64(det):
    """As below at head_dim 64, where the fused backward carries every key block's dQ, the
    14 split items' chunks included (the dQ stage then only converts the accumulator)."""
    import paper_2501_08453_amd as vc
    w = W.custom(1, 9, 64, 100, 4, 43, 43, name="tail64", ragged_text=True)
    assert (w.tokens + 255) // 256 == 30
    assert vc.vc_jointattn_fused_dq_keys(vc.desc_for(w)) == w.tokens
    x = W.make_inputs(w, seed=73)
    km = W.random_key_mask(w, seed=74, keep=0.9)
    log("split tail, head_dim 64: 270 items of 256 rows", w.shape, "deterministic" if det else "fused")
    _full_compare(w, x, key_mask=km, heads=[0, 8], det=det)


@pytest.mark.parametrize("det", MODES, ids=MODE_IDS)
def test_split_tail_of_last_round(det):
    """Joint kernels split the items of their last, partial round of workgroups over several
    workgroups (fp32 partials merged or summed afterwards). 9 heads x 30 blocks of 256 rows
    = 270 items: on 256 compute units the last 14 items (blocks 16-29 of head 8) are split
    into 17 chunks of 7 query (key) tiles each. head_dim 128, so that the two ids run different backwards: the
    fused one (key blocks 0-19 add their dQ share with atomics, 4 of them inside the split
    tail; the dQ pass covers blocks 20-29) and the deterministic one (separate dK/dV pass,
    dQ pass over every key). Head 8 (and head 0, unsplit) on every element, with ragged
    text and a key mask so that split items hold masked keys too."""
    import paper_2501_08453_amd as vc
    w = W.custom(1, 9, 128, 100, 4, 43, 43, name="tail", ragged_text=True)
    assert (w.tokens + 255) // 256 == 30
    fused_keys = vc.vc_jointattn_fused_dq_keys(vc.desc_for(w))
    assert fused_keys == 20 * 256, fused_keys
    x = W.make_inputs(w, seed=71)
    km = W.random_key_mask(w, seed=72, keep=0.9)
    log("split tail: 270 items of 256 rows", w.shape, "deterministic" if det else "fused")
    _full_compare(w, x, key_mask=km, heads=[0, 8], det=det)


def test_tiny_workload_fp32_oracle():
    """Workload 1 (144 tokens): oracle on the fp32 draws, GPU on their bf16 casts."""
    w = W.WORKLOADS[1]
    log("tiny workload, oracle on fp32 inputs")
    _full_compare(w, W.make_inputs(w), use_bf16_oracle=False)


def test_tiny_workload_bf16_oracle():
    w = W.WORKLOADS[1]
    log("tiny workload, oracle on the bf16 inputs")
    _full_compare(w, W.make_inputs(w))


EDGE = [
    # (name, B, H, D, T, F, Hp, Wp, text_len, mask_keep, scale)
    ("fewer-keys-than-a-wave", 1, 1, 64, 0, 1, 1, 5, None, None, None),
    ("text-only-padding", 2, 3, 128, 7, 3, 5, 7, [3, 7], None, None),
    ("ragged-tail-d128", 1, 2, 128, 40, 2, 10, 13, [40], None, None),
    ("ragged-tail-d64", 3, 2, 64, 64, 4, 9, 11, [1, 64, 0], None, None),
    ("key-mask-d128", 2, 2, 128, 16, 3, 7, 9, [5, 16], 0.8, None),
    ("key-mask-d64", 2, 2, 64, 16, 2, 9, 9, None, 0.6, None),
    ("skipped-text-tiles", 1, 2, 128, 256, 1, 10, 10, [8], None, None),
    # scale 0.3 on q drawn with std 0.3: logits of order one, as in the workloads
    ("scale-0.3", 1, 2, 128, 32, 2, 8, 8, [20], None, 0.3),
    ("two-query-tiles-exact", 1, 1, 128, 0, 2, 8, 16, None, None, None),
]


@pytest.mark.parametrize("det", MODES, ids=MODE_IDS)
@pytest.mark.parametrize("case", EDGE, ids=[e[0] for e in EDGE])
def test_edge_shapes(case, det):
    name, B, H, D, T, F, Hp, Wp, tl, keep, scale = case
    log("edge case", name, "deterministic" if det else "fused")
    w = W.custom(B, H, D, T, F, Hp, Wp)
    x = W.make_inputs(w, seed=zlib.crc32(name.encode()) % 10000)
    if scale is not None:
        x["q"] *= np.float32(scale)
    if tl is not None:
        x["text_len"] = np.array(tl, dtype=np.int32)
    km = None if keep is None else W.random_key_mask(w, 7, keep)
    _full_compare(w, x, scale=scale, key_mask=km, det=det)


def test_sample_without_valid_keys_and_single_key():
    """Sample 0: every key masked (O = 0, LSE = -inf, grads 0); sample 1: one valid key."""
    import torch
    w = W.custom(2, 2, 128, 8, 2, 6, 6)
    x = W.make_inputs(w, seed=5)
    km = np.zeros((2, w.tokens), np.uint8)
    km[1, 17] = 1
    log("no valid keys / single valid key")
    out, _ = _full_compare(w, x, key_mask=km)
    assert np.all(out["o"][0] == 0) and np.all(np.isneginf(out["lse"][0]))
    assert np.all(out["dq"][0] == 0) and np.all(out["dk"][0] == 0) and np.all(out["dv"][0] == 0)
    assert np.all(out["dk"][1][np.arange(w.tokens) != 17] == 0)
    del torch


def test_medium_workload_sampled_heads():
    """Workload 2 (8,320 tokens, D=64, flat logits) on four (sample, head) pairs, every element."""
    w = W.WORKLOADS[2]
    x = W.make_inputs(w)
    log("medium workload, samples 0-1 x heads 0, 3, 15")
    _full_compare(w, x, heads=[0, 3, 15], samples=[0, 1])


def test_ragged_workload_sampled_heads():
    """Workload 4 (4 x 9,856 tokens, text lengths drawn in [8, 256])."""
    w = W.WORKLOADS[4]
    x = W.make_inputs(w)
    log("ragged workload, text_len =", x["text_len"].tolist())
    _full_compare(w, x, heads=[0, 15], samples=[0, 1, 2, 3])


def _sampled_large(wid, heads, n_rows, with_cols, det=False):
    """Workload `wid` through the C ABI (fused backward, or det: the deterministic one),
    against the oracle on sampled query rows (O, LSE, dQ) and, with_cols, the same
    positions as key columns (dK, dV) of the given heads. The sample holds n_rows random
    rows, 16 random rows among the last 48 blocks of 256 rows (they hold the items of the
    last, split round of dispatch at these sizes, all of the last head) and the text
    boundary and ends."""
    import torch
    vc = _vc()
    w = W.WORKLOADS[wid]
    log("workload", wid, "generating inputs", w.shape, "deterministic" if det else "fused")
    x = W.make_inputs(w)
    g = _inputs_on_gpu(x)
    del x
    desc = vc.desc_for(w, deterministic=det)
    out = run_gpu(desc, g["q"], g["k"], g["v"], g["do"], g["text_len"], None, host=False)
    log("workload", wid, "GPU done")
    B, N, H, D = w.shape
    c = ora.default_scale(D)
    valid = ora.key_validity(B, N, w.text_slot, None)
    rng = np.random.Generator(np.random.PCG64(2024 + wid))
    rows = np.unique(np.r_[0, 1, w.text_slot - 1, w.text_slot, N - 1, rng.integers(0, N, n_rows),
                           rng.integers(max(0, N - 48 * 256), N, 16)])
    rows_t = torch.from_numpy(rows).to("cuda")
    res = {n: [] for n in ("o", "lse", "dq", "dk", "dv")}
    ref = {n: [] for n in res}
    for h in heads:
        qh, kh, vh, doh = (bf16_values(g[n][:, :, h:h + 1]) for n in ("q", "k", "v", "do"))
        o_r, l_r = ora.forward_rows(qh, kh, vh, valid[0], c, 0, 0, rows)
        dq_r = ora.backward_rows(qh, kh, vh, doh, valid[0], c, 0, 0, rows)
        pick = lambda n: bf16_values(out[n][0, :, h].index_select(0, rows_t))  # noqa: E731
        res["o"].append(pick("o")); ref["o"].append(o_r)
        res["lse"].append(out["lse"][0, h].index_select(0, rows_t).double().cpu().numpy()); ref["lse"].append(l_r)
        res["dq"].append(pick("dq")); ref["dq"].append(dq_r)
        if with_cols:
            dk_c, dv_c = ora.backward_cols(qh, kh, vh, doh, valid[0], c, 0, 0, rows)
            res["dk"].append(pick("dk")); ref["dk"].append(dk_c)
            res["dv"].append(pick("dv")); ref["dv"].append(dv_c)
        log("workload", wid, "head", h, "oracle done")
    for n in res:
        if res[n]:
            assert_close(n, np.concatenate(res[n]), np.concatenate(ref[n]))
    # identities at any size, every head: sum_j dK_j = 0 and sum_j dV_j = sum_i dO_i
    dk_sum = out["dk"].double().sum(dim=1)            # [B, H, D]
    dv_sum = out["dv"].double().sum(dim=1)
    do_sum = g["do"].double().sum(dim=1)
    scale_dv = do_sum.abs().mean().item()
    err_dv = (dv_sum - do_sum).abs().max().item()
    err_dk = dk_sum.abs().max().item()
    dk_mag = out["dk"].double().abs().sum(dim=1).mean().item()
    log("   sum dV - sum dO: max %.3e (sum dO ~ %.3e); |sum dK| max %.3e (sum |dK| ~ %.3e)"
        % (err_dv, scale_dv, err_dk, dk_mag))
    assert err_dv <= 5e-3 * scale_dv
    assert err_dk <= 5e-3 * dk_mag


def test_long_workload_sampled():
    """Workload 3 (57,856 tokens, 24 heads, D=128): rows and columns of heads 0 and 23."""
    _sampled_large(3, heads=[0, 23], n_rows=48, with_cols=True)


def test_long_workload_sampled_deterministic():
    """Workload 3 with the deterministic backward (separate dK/dV pass with token-major Q and
    dO copies, dQ pass over every key, both with their split last round and tail sums):
    rows and columns of heads 0 and 23."""
    _sampled_large(3, heads=[0, 23], n_rows=48, with_cols=True, det=True)


def test_max_workload_sampled():
    """Workload 5 (123,136 tokens): rows and columns of heads 0 and 23, identities on all
    heads."""
    _sampled_large(5, heads=[0, 23], n_rows=48, with_cols=True)


@pytest.mark.parametrize("det", MODES, ids=MODE_IDS)
def test_masked_key_values_have_no_effect(det):
    import torch
    vc = _vc()
    w = W.custom(2, 2, 128, 32, 2, 8, 9)
    x = W.make_inputs(w, seed=11)
    x["text_len"] = np.array([5, 30], np.int32)
    km = W.random_key_mask(w, 3, 0.7)
    g = _inputs_on_gpu(x)
    kmg = torch.from_numpy(km).to("cuda")
    desc = vc.desc_for(w, deterministic=det)
    a = run_gpu(desc, g["q"], g["k"], g["v"], g["do"], g["text_len"], kmg)
    valid = ora.key_validity(2, w.tokens, w.text_slot, x["text_len"], km)
    inv = torch.from_numpy(~valid).to("cuda")[:, :, None, None]
    # 30: large finite probabilities at the masked keys; 3000: their exponentials
    # overflow (inf, and NaN in dS), which must stay confined to those keys
    for mag in (30.0, 3000.0):
        noise = torch.randn(g["k"].shape, device="cuda", generator=torch.Generator("cuda").manual_seed(1)) * mag
        k2 = torch.where(inv, noise.to(torch.bfloat16), g["k"]).contiguous()
        v2 = torch.where(inv, (-noise).to(torch.bfloat16), g["v"]).contiguous()
        b = run_gpu(desc, g["q"], k2, v2, g["do"], g["text_len"], kmg)
        assert np.array_equal(a["o"], b["o"]) and np.array_equal(a["lse"], b["lse"])
        assert np.all(b["dk"][~valid] == 0) and np.all(b["dv"][~valid] == 0)
        if det:
            assert np.array_equal(a["dk"][valid], b["dk"][valid]) and np.array_equal(a["dv"][valid], b["dv"][valid])
            assert np.array_equal(a["dq"], b["dq"])
        else:  # dK, dV without atomics; dQ summed by atomics, and finite (no inf or NaN leaked)
            assert np.array_equal(a["dk"][valid], b["dk"][valid]) and np.array_equal(a["dv"][valid], b["dv"][valid])
            assert np.all(np.isfinite(b["dq"])) and _same_up_to_order(a["dq"], b["dq"], "dQ, masked values changed")


def test_forward_is_deterministic_and_batch_independent():
    import torch
    vc = _vc()
    w = W.custom(3, 2, 128, 64, 2, 9, 10, ragged_text=True)
    x = W.make_inputs(w, seed=21)
    g = _inputs_on_gpu(x)
    desc = vc.desc_for(w)
    o1, l1 = vc.fwd(g["q"], g["k"], g["v"], desc, g["text_len"])
    o2, l2 = vc.fwd(g["q"], g["k"], g["v"], desc, g["text_len"])
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    for b in range(3):
        d1 = vc.make_desc(1, 2, 128, 64, 2, 9, 10)
        ob, lb = vc.fwd(g["q"][b:b + 1].contiguous(), g["k"][b:b + 1].contiguous(), g["v"][b:b + 1].contiguous(),
                        d1, g["text_len"][b:b + 1].contiguous())
        assert torch.equal(ob, o1[b:b + 1]) and torch.equal(lb, l1[b:b + 1])


def test_autograd_wrapper_matches_direct_calls():
    import torch
    vc = _vc()
    w = W.custom(1, 2, 64, 16, 2, 8, 8)
    x = W.make_inputs(w, seed=4)
    g = _inputs_on_gpu(x)
    desc = vc.desc_for(w, deterministic=True)
    q = g["q"].clone().requires_grad_(True)
    k = g["k"].clone().requires_grad_(True)
    v = g["v"].clone().requires_grad_(True)
    o = vc.joint_attention(q, k, v, desc)
    o.backward(g["do"])
    ref = run_gpu(desc, g["q"], g["k"], g["v"], g["do"])
    assert np.array_equal(bf16_values(o.detach()), ref["o"])
    assert np.array_equal(bf16_values(q.grad), ref["dq"])
    assert np.array_equal(bf16_values(k.grad), ref["dk"])
    assert np.array_equal(bf16_values(v.grad), ref["dv"])


def test_backward_reproducibility():
    """Deterministic backward: two runs agree bit for bit. Fused backward: dK, dV (no
    atomics) bit for bit run to run; dQ, and all three against the deterministic ones, up
    to one bf16 spacing (the order of fp32 additions differs)."""
    import torch
    vc = _vc()
    w = W.custom(2, 3, 128, 40, 3, 7, 9, ragged_text=True)
    x = W.make_inputs(w, seed=12)
    g = _inputs_on_gpu(x)
    runs = {}
    for det in (True, False):
        desc = vc.desc_for(w, deterministic=det)
        o, lse = vc.fwd(g["q"], g["k"], g["v"], desc, g["text_len"])
        runs[det] = [(o, lse) + vc.bwd(g["q"], g["k"], g["v"], o, lse, g["do"], desc, g["text_len"]) for _ in range(2)]
    torch.cuda.synchronize()
    for a, b in zip(*runs[True]):
        assert torch.equal(a, b)
    f0, f1 = runs[False]
    for i in (0, 1, 3, 4):  # o, lse, dk, dv
        assert torch.equal(f0[i], f1[i])
    for i, n in ((2, "dQ"), (3, "dK"), (4, "dV")):  # against the deterministic backward
        for f in (f0, f1):
            assert _same_up_to_order(bf16_values(f[i]), bf16_values(runs[True][0][i]), n + " fused vs deterministic")


@pytest.mark.parametrize("head_dim", [128, 64])
def test_staged_backward_calls(head_dim):
    """The stage entry points reproduce vc_jointattn_bwd in both modes, and the separate
    dK/dV stage refuses a descriptor of the fused backward (whose stage 1 does not make the
    token-major copies it reads). With head_dim 64 the fused pass carries every key's dQ
    (stage 3 then only converts the accumulator); with 128, the leading 65% of the keys'."""
    import torch
    vc = _vc()
    w = W.custom(1, 2, head_dim, 24, 3, 9, 10, ragged_text=True)
    x = W.make_inputs(w, seed=77)
    g = _inputs_on_gpu(x)
    q, k, v, do, tl = g["q"], g["k"], g["v"], g["do"], g["text_len"]
    for det in (True, False):
        desc = vc.desc_for(w, deterministic=det)
        o, lse = vc.fwd(q, k, v, desc, tl)
        ref = vc.bwd(q, k, v, o, lse, do, desc, tl)
        dq, dk, dv = (torch.empty_like(q) for _ in range(3))
        ws = vc.workspace(desc, "cuda")
        s = torch.cuda.current_stream().cuda_stream
        vc.vc_jointattn_bwd_prepare(desc, q, k, o, lse, do, ws, ws.numel(), s)
        if det:
            vc.vc_jointattn_bwd_dkdv(desc, q, k, v, do, tl, None, dk, dv, ws, ws.numel(), s)
        else:
            with pytest.raises(vc.JointAttnError) as e:
                vc.vc_jointattn_bwd_dkdv(desc, q, k, v, do, tl, None, dk, dv, ws, ws.numel(), s)
            assert e.value.status == -8
            vc.vc_jointattn_bwd_fused(desc, q, k, v, do, tl, None, dk, dv, ws, ws.numel(), s)
        vc.vc_jointattn_bwd_dq(desc, q, k, v, do, tl, None, dq, ws, ws.numel(), s)
        torch.cuda.synchronize()
        assert torch.equal(dk, ref[1]) and torch.equal(dv, ref[2])
        if not det and head_dim == 64:
            assert vc.vc_jointattn_fused_dq_keys(desc) == w.tokens
        if det:
            assert torch.equal(dq, ref[0])
        else:
            assert _same_up_to_order(bf16_values(dq), bf16_values(ref[0]), "dQ staged vs one call")
