"""GPU test of the no-allocation forward (vc_jointattn_fwd_noalloc), through the C ABI.

Its output is compared with the workspace-taking forward's (vc_jointattn_fwd, the same
kernels) bit for bit, and with the fp64 oracle to the parity bar, on two calls in a row,
the second with a smaller input: the ragged-text workload first (4 x 9,856 tokens, 216 MB
of the 256 MiB scratch array), then a small ragged, key-masked problem at head_dim 64.
A problem larger than the array is refused before anything runs.
"""
import numpy as np
import pytest

import oracle.ref_attention as ora
import workloads as W
from parity_util import assert_close, bf16_values, log, to_gpu_bf16

pytestmark = pytest.mark.gpu


def _call_both(w, x, key_mask=None):
    import torch
    import paper_2501_08453_amd as vc
    q, k, v = (to_gpu_bf16(x[n]) for n in ("q", "k", "v"))
    tl = None if x["text_len"] is None else torch.from_numpy(x["text_len"]).to("cuda")
    km = None if key_mask is None else torch.from_numpy(key_mask).to("cuda")
    desc = vc.desc_for(w)
    B, N, H, D = w.shape
    assert vc.vc_jointattn_fwd_workspace_bytes(desc) <= vc.NOALLOC_SCRATCH_BYTES
    o_n = torch.full_like(q, float("nan"))
    l_n = torch.full((B, H, N), float("nan"), dtype=torch.float32, device="cuda")
    vc.vc_jointattn_fwd_noalloc(desc, q, k, v, tl, km, o_n, l_n)
    o_w, l_w = vc.fwd(q, k, v, desc, tl, km)
    torch.cuda.synchronize()
    assert torch.equal(o_n, o_w), "no-allocation forward differs from vc_jointattn_fwd (O)"
    assert torch.equal(l_n, l_w), "no-allocation forward differs from vc_jointattn_fwd (LSE)"
    return q, k, v, o_n, l_n


def test_noalloc_forward_two_calls_then_refusal():
    import torch
    import paper_2501_08453_amd as vc
    # call 1: the ragged-text workload; oracle on sampled rows of two (sample, head) pairs
    w1 = W.WORKLOADS[4]
    x1 = W.make_inputs(w1, with_do=False)
    log("no-alloc forward, call 1:", w1.shape, "text_len", x1["text_len"].tolist())
    q, k, v, o, lse = _call_both(w1, x1)
    B, N, H, D = w1.shape
    valid = ora.key_validity(B, N, w1.text_slot, x1["text_len"])
    rng = np.random.Generator(np.random.PCG64(5))
    rows = np.unique(np.r_[0, w1.text_slot - 1, w1.text_slot, N - 1, rng.integers(0, N, 40)])
    rows_t = torch.from_numpy(rows).to("cuda")
    for b, h in ((0, 0), (3, 15)):
        qh, kh, vh = (bf16_values(t[b:b + 1, :, h:h + 1]) for t in (q, k, v))
        o_r, l_r = ora.forward_rows(qh, kh, vh, valid[b], ora.default_scale(D), 0, 0, rows)
        assert_close("O", bf16_values(o[b, :, h].index_select(0, rows_t)), o_r)
        assert_close("LSE", lse[b, h].index_select(0, rows_t).double().cpu().numpy(), l_r)
    del q, k, v, o, lse
    # call 2: smaller, head_dim 64, ragged text and a key mask; oracle on every element
    w2 = W.custom(2, 2, 64, 16, 2, 8, 9, ragged_text=True)
    x2 = W.make_inputs(w2, seed=31, with_do=False)
    km = W.random_key_mask(w2, seed=32, keep=0.85)
    log("no-alloc forward, call 2:", w2.shape)
    q, k, v, o, lse = _call_both(w2, x2, km)
    B, N, H, D = w2.shape
    valid = ora.key_validity(B, N, w2.text_slot, x2["text_len"], km)
    o_r, l_r = ora.attention_forward(bf16_values(q), bf16_values(k), bf16_values(v), valid)
    assert_close("O", bf16_values(o), o_r)
    assert_close("LSE", lse.double().cpu().numpy(), l_r)
    # a problem beyond the array: refused with VC_ERR_SCRATCH, nothing launched
    big = vc.make_desc(1, 24, 128, 256, 16, 45, 80)
    with pytest.raises(vc.JointAttnError) as e:
        vc.vc_jointattn_fwd_noalloc(big, q, k, v, None, None, o, lse)
    assert e.value.status == -10
