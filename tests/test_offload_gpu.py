"""GPU tests of the activation offload engine (vc_offload_*, through the C ABI) and of
the block's memory strategies: keeping the branch outputs, recomputing them before
the backward, or offloading them to pinned host memory and loading them back. The
attention path is deterministic (with the separate dQ pass), so all three give
bit-identical gradients.
"""
import pytest

import workloads as W
from parity_util import log, to_gpu_bf16

pytestmark = pytest.mark.gpu


def test_round_trip_is_bitwise():
    import torch
    import paper_2501_08453_amd as vc
    x = torch.randn(3, 1000, 7, device="cuda").to(torch.bfloat16)
    host = torch.empty(x.shape, dtype=x.dtype, pin_memory=True)
    back = torch.empty_like(x)
    with vc.Offload() as off:
        off.store(host, x)
        off.wait()
        off.load(back, host)
        off.wait()
        torch.cuda.synchronize()
    assert torch.equal(host, x.cpu())
    assert torch.equal(back, x)


def test_store_is_ordered_after_queued_kernels():
    """A store issued right after a long kernel on the stream, with no host
    synchronisation, copies the kernel's result."""
    import torch
    import paper_2501_08453_amd as vc
    w = W.WORKLOADS[2]
    x = W.make_inputs(w, with_do=False)
    q, k, v = (to_gpu_bf16(x[n]) for n in ("q", "k", "v"))
    desc = vc.desc_for(w)
    tl = None if x["text_len"] is None else torch.from_numpy(x["text_len"]).to("cuda")
    torch.cuda.synchronize()
    o = torch.zeros_like(q)
    lse = torch.empty((w.batch, w.heads, w.tokens), device="cuda")
    host_o = torch.empty(o.shape, dtype=o.dtype, pin_memory=True)
    host_l = torch.empty(lse.shape, dtype=lse.dtype, pin_memory=True)
    with vc.Offload() as off:
        vc.fwd(q, k, v, desc, text_len=tl, out=o, lse=lse)
        off.store(host_o, o)
        off.store(host_l, lse)
        off.wait()
        o.fill_(0)  # ordered after the copies on this stream
        torch.cuda.synchronize()
    ref_o, ref_l = vc.fwd(q, k, v, desc, text_len=tl)
    torch.cuda.synchronize()
    assert torch.equal(host_o, ref_o.cpu())
    assert torch.equal(host_l, ref_l.cpu())


def test_rejects_pageable_and_out_of_range_memory():
    import torch
    import paper_2501_08453_amd as vc
    x = torch.randn(4096, device="cuda")
    pageable = torch.empty(4096)
    pinned = torch.empty(4096, pin_memory=True)
    with vc.Offload() as off:
        with pytest.raises(vc.JointAttnError) as e:
            off.store(pageable, x)
        assert e.value.status == -8
        lib = vc._lib()
        # ranges running past the allocations (the device one may be a larger segment of
        # torch's caching allocator, so go far past it)
        n = x.numel() * 4
        assert lib.vc_offload_store(off._h, pinned.data_ptr(), x.data_ptr(), 1 << 40, None) == -8
        assert lib.vc_offload_load(off._h, x.data_ptr(), pinned.data_ptr(), n + (1 << 30), None) == -8
        assert lib.vc_offload_store(off._h, None, x.data_ptr(), n, None) == -1
        off.store(pinned, x)  # the valid copy still works
        off.wait()
        torch.cuda.synchronize()
    assert torch.equal(pinned, x.cpu())


def _block(vc, q, k, v, do, desc, strategy, off=None):
    """Block forward (three branches + fused sum) then backward, with the branch outputs
    kept, recomputed, or offloaded and loaded back. Returns (sum, grads)."""
    import torch
    o_j, l_j = vc.fwd(q, k, v, desc)
    o_s, l_s = vc.spatial_fwd(q, k, v, desc)
    o_t, l_t, out = vc.temporal_fwd_sum(q, k, v, desc, o_joint=o_j, o_spatial=o_s)
    saved = [o_j, l_j, o_s, l_s, o_t, l_t]
    if strategy == "offload":
        host = [torch.empty(t.shape, dtype=t.dtype, pin_memory=True) for t in saved]
        for hbuf, t in zip(host, saved):
            off.store(hbuf, t)
        off.wait()
        for t in saved:  # the device copies are free for reuse once the wait is queued
            t.fill_(float("nan"))
        for hbuf, t in zip(host, saved):
            off.load(t, hbuf)
        off.wait()
    elif strategy == "recompute":
        for t in saved:
            t.fill_(float("nan"))
        vc.fwd(q, k, v, desc, out=o_j, lse=l_j)
        vc.spatial_fwd(q, k, v, desc, out=o_s, lse=l_s)
        vc.temporal_fwd(q, k, v, desc, out=o_t, lse=l_t)
    grads = [vc.bwd(q, k, v, o_j, l_j, do, desc), vc.spatial_bwd(q, k, v, o_s, l_s, do, desc),
             vc.temporal_bwd(q, k, v, o_t, l_t, do, desc)]
    torch.cuda.synchronize()
    return out, grads


def test_keep_recompute_offload_give_identical_gradients():
    import torch
    import paper_2501_08453_amd as vc
    w = W.custom(1, 4, 128, 64, 6, 10, 16)
    x = W.make_inputs(w, seed=2718)
    q, k, v, do = (to_gpu_bf16(x[n]) for n in ("q", "k", "v", "do"))
    desc = vc.desc_for(w, deterministic=True)
    keep = _block(vc, q, k, v, do, desc, "keep")
    rec = _block(vc, q, k, v, do, desc, "recompute")
    with vc.Offload() as off:
        offl = _block(vc, q, k, v, do, desc, "offload", off)
    for other, name in ((rec, "recompute"), (offl, "offload")):
        assert torch.equal(other[0], keep[0]), name
        for gk, go in zip(keep[1], other[1]):
            for a, b in zip(gk, go):
                assert torch.equal(a, b), name
        log("   %s: bitwise equal to keep" % name)


def test_selective_plans_give_identical_results():
    """Five stacked layers with their own q, k, v and upstream gradient, run under plans that
    recompute and/or offload a share of the layers (memory.BlockStack: one or two device
    sets for the offloaded layers in turn, loads overlapping another layer's backward):
    every layer's block output and the gradients of all three branches are bitwise those of
    keeping every layer's saved outputs."""
    import torch
    import paper_2501_08453_amd as vc
    from paper_2501_08453_amd import memory as mem
    K = 5
    assert mem.ring_size(mem.plan(K, 0.4, "offload")) == 1 and mem.ring_size(mem.plan(K, 0.6, "offload")) == 2
    w = W.custom(1, 2, 128, 16, 4, 6, 8)
    desc = vc.desc_for(w, deterministic=True)
    inputs, douts = [], []
    for i in range(K):
        x = W.make_inputs(w, seed=3100 + i)
        inputs.append(tuple(to_gpu_bf16(x[n]) for n in ("q", "k", "v")))
        douts.append(to_gpu_bf16(x["do"]))

    def run(strategies):
        outs = [torch.full_like(inputs[0][0], float("nan")) for _ in range(K)]
        grads = [tuple(tuple(torch.full_like(inputs[0][0], float("nan")) for _ in range(3)) for _ in range(3))
                 for _ in range(K)]
        bs = mem.BlockStack(desc, inputs, strategies, outs, grads)
        bs.forward()
        bs.backward(douts)
        torch.cuda.synchronize()
        bs.close()
        return outs, grads

    ref = run(mem.plan(K, 0.0, "keep"))
    # offload 0.4: two spaced layers sharing one device set; 0.6 and 1.0: adjacent ones, two
    # sets; combination: one offloaded layer and recomputed ones
    for mode, ratio in (("recompute", 0.6), ("offload", 0.4), ("offload", 0.6), ("offload", 1.0),
                        ("combination", 1.0), ("combination", 0.2)):
        st = mem.plan(K, ratio, mode)
        got = run(st)
        for i in range(K):
            assert torch.equal(got[0][i], ref[0][i]), (mode, ratio, i)
            for br in range(3):
                for a, b in zip(got[1][i][br], ref[1][i][br]):
                    assert torch.equal(a, b), (mode, ratio, i, br)
        log("   %s at ratio %.1f (%s): bitwise equal to keep" % (mode, ratio, ",".join(s[0] for s in st)))
