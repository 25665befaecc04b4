#!/usr/bin/env python3
"""Throughput of joint text-video attention (forward + backward) on one MI355X.

One step = one pass of the whole path over one batch of synthetic input:
forward (O, LSE), backward prepare (D = rowsum(dO o O), token-major copies),
backward dK/dV and backward dQ, all through the C ABI on torch's current
stream. Inputs are resident in HBM before timing.

Prints one JSON line. `value` is algorithmic TFLOP/s of the whole step:
12 * H * N * N_kv * D per sample (forward 4, backward 8; the backward's
recomputation of Q K^T is not counted).

--branch spatial / temporal measure the other two attention branches of the
block instead (same inputs, forward + backward): the spatial branch in
algorithmic TFLOP/s (each video query against the valid text keys and its own
frame), the temporal branch, which is bound by memory traffic, in algorithmic
GB/s (bytes the step must move at least).

--branch block measures the whole attention of the parallel block (the three
branches and their fused sum) over --layers stacked layers, forward through all
of them and backward in reverse, with the branch outputs each layer saves for
its backward kept in HBM, or, for a selective ratio of the layers, recomputed
before its backward, offloaded to pinned host memory and loaded back, or both
combined (the memory strategies of Sec. V-B / VI-D).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import workloads as W  # noqa: E402

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 matrix-core peak (published)
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E bandwidth (published)
METRIC = "joint-attention fwd+bwd TFLOP/s and % bf16 MFMA peak at 57,856 tokens"
METRIC_SPATIAL = "spatial-attention fwd+bwd TFLOP/s (per-frame text+frame keys)"
METRIC_TEMPORAL = "temporal-attention fwd+bwd GB/s (algorithmic HBM bytes)"
METRIC_BLOCK = ("parallel-block attention (joint + spatial + temporal, summed) fwd+bwd TFLOP/s; saved branch "
                "outputs kept, recomputed or offloaded")


def valid_keys_per_sample(w, text_len):
    if text_len is None:
        return [w.tokens] * w.batch
    tl = np.clip(np.asarray(text_len), 0, w.text_slot)
    return [int(w.tokens - (w.text_slot - t)) for t in tl]


def flops(w, text_len):
    nkv = valid_keys_per_sample(w, text_len)
    fwd = sum(4.0 * w.heads * w.tokens * n * w.head_dim for n in nkv)
    return fwd, 2.0 * fwd


def spatial_flops(w, text_len):
    """Forward, backward algorithmic flops of the spatial branch: each of the F*L video
    queries against the valid text keys and the L keys of its frame."""
    L = w.grid_h * w.grid_w
    tl = [w.text_slot] * w.batch if text_len is None else np.clip(np.asarray(text_len), 0, w.text_slot)
    fwd = sum(4.0 * w.heads * w.frames * L * (L + int(t)) * w.head_dim for t in tl)
    return fwd, 2.0 * fwd


def temporal_bytes(w):
    """Forward, backward algorithmic HBM bytes of the temporal branch (bf16 tensors of the
    video rows, fp32 LSE): the least the step must move. Forward reads q, k, v and writes
    o, lse; backward reads q, k, v, o, dO, lse and writes dq, dk, dv (D = rowsum(dO o O)
    needs no bytes of its own: o and dO are read anyway)."""
    rows = w.batch * w.frames * w.grid_h * w.grid_w * w.heads
    t = rows * w.head_dim * 2.0
    r = rows * 4.0
    return 3 * t + t + r, 5 * t + r + 3 * t


def cpu_baseline_branch(kind, w, g, text_len, target_s):
    """The branch oracle timed on a bounded sample: whole frames of head 0 (spatial) or a
    block of spatial positions of head 0 (temporal), forward + backward."""
    import torch
    import oracle.ref_branches as orb
    T, F, L = w.text_slot, w.frames, w.grid_h * w.grid_w
    tl = None if text_len is None else text_len[:1]
    threads = __import__("oracle").host_threads()
    if kind == "spatial":
        # one frame of sample 0 with every head per round (the oracle's pool runs the heads
        # in parallel), frames added until the target time is reached
        done, fl, t = 0, 0.0, 0.0
        while done < F and t < target_s:
            def sl(name):
                a = g[name][:1]
                a = torch.cat([a[:, :T], a[:, T + done * L:T + (done + 1) * L]], dim=1)
                return a.to(torch.float64).cpu().numpy()
            q, k, v, do = (sl(n) for n in ("q", "k", "v", "do"))
            t0 = time.perf_counter()
            _, lse = orb.spatial_forward(q, k, v, T, 1, tl)
            orb.spatial_backward(q, k, v, do, T, 1, tl, lse=lse)
            t += time.perf_counter() - t0
            tv = T if tl is None else int(min(max(tl[0], 0), T))
            fl += 12.0 * w.heads * L * (L + tv) * w.head_dim
            done += 1
        return {"value": fl / t / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
                "sample": "%d frame(s) of sample 0, all %d heads (text + frame keys), fwd+bwd, %.1f s"
                % (done, w.heads, t)}
    h0 = lambda t: t[:1, :, :1].to(torch.float64).cpu().numpy()  # noqa: E731
    q, k, v, do = (h0(g[n]) for n in ("q", "k", "v", "do"))
    n_pos = 64
    while True:
        pos = np.arange(min(n_pos, L))
        rows = (T + np.arange(F)[:, None] * L + pos[None, :]).reshape(-1)
        sl = lambda a: a[:, rows]  # noqa: E731
        t0 = time.perf_counter()
        _, lse = orb.temporal_forward(sl(q), sl(k), sl(v), 0, F)
        orb.temporal_backward(sl(q), sl(k), sl(v), sl(do), 0, F, lse=lse)
        t = time.perf_counter() - t0
        if t >= target_s / 4 or n_pos >= L:
            break
        n_pos *= 2
    wsub = W.custom(1, 1, w.head_dim, 0, F, 1, len(pos))
    bf, bb = temporal_bytes(wsub)
    return {"value": (bf + bb) / t / 1e9, "unit": "GB/s", "cores": __import__("oracle").host_threads(),
            "kind": "oracle", "sample": "%d spatial positions x %d frames of sample 0, head 0, fwd+bwd, %.1f s"
            % (len(pos), F, t)}


def cpu_baseline(w, g, text_len, target_s):
    """Time the fp64 oracle on a bounded block of query rows of head 0, sample 0.

    Rows are doubled from 1024 until one run takes a quarter of the target, then the
    block is scaled to about the target (at most every row of the head). The oracle's
    thread pool uses every host core it may run on.
    """
    import torch
    import oracle.ref_attention as ora
    N, D = w.tokens, w.head_dim
    qh, kh, vh, doh = (g[n][0:1, :, 0:1].to(torch.float64).cpu().numpy() for n in ("q", "k", "v", "do"))
    valid = ora.key_validity(1, N, w.text_slot, None if text_len is None else text_len[:1])
    c = ora.default_scale(D)
    nkv = int(valid[0].sum())

    def run(rows):
        t0 = time.perf_counter()
        ora.rowblock_fwd_bwd(qh, kh, vh, doh, valid[0], c, 0, 0, np.arange(rows))
        return time.perf_counter() - t0

    rows = min(N, 1024)
    t = run(rows)
    while t < target_s / 4 and rows < N:
        rows = min(N, rows * 2)
        t = run(rows)
    if t < target_s * 0.75 and rows < N:
        rows = int(min(N, rows * target_s / max(t, 1e-3)))
        t = run(rows)
    fl = 12.0 * rows * nkv * D
    return {
        "value": fl / t / 1e12,
        "unit": "TFLOP/s",
        "cores": ora.host_threads(),
        "kind": "oracle",
        "sample": "query rows 0..%d of head 0, sample 0 (%d of %d queries x %d keys, D=%d), forward + "
                  "backward in fp64 (%.1f s); same algorithmic flop count as the GPU figure"
                  % (rows - 1, rows, N, nkv, D, t),
    }


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_bwd_dkdv_long720p.json")
KERNEL_SOURCES = ["paper_2501_08453_amd/csrc/bwd.hip", "paper_2501_08453_amd/csrc/common.hpp"]
# Traffic records of the temporal backward, per workload: the short-clip kernel at the long
# workload, the long-clip kernel at the 144-frame clip.
TEMPORAL_TRAFFIC = {
    3: (os.path.join(ROOT, "profiles", "traffic_temporal_bwd_long720p.json"),
        ["paper_2501_08453_amd/csrc/temporal.hip", "paper_2501_08453_amd/csrc/common.hpp"]),
    6: (os.path.join(ROOT, "profiles", "traffic_temporal_bwd_clip144f.json"),
        ["paper_2501_08453_amd/csrc/temporal_long.hip", "paper_2501_08453_amd/csrc/common.hpp"]),
}


def code_only(text: str) -> str:
    """Source text without // comments, trailing blanks and blank lines, so that a traffic
    record stays tied to the code it was measured on, not to its commentary. (The kernel
    sources keep no // inside string literals.)"""
    out = []
    for line in text.splitlines():
        line = line.split("//", 1)[0].rstrip()
        if line:
            out.append(line)
    return "\n".join(out)


def kernel_source_digest(sources=KERNEL_SOURCES) -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in sources:
        with open(os.path.join(ROOT, rel), encoding="utf-8") as f:
            h.update(code_only(f.read()).encode())
    return h.hexdigest()


def traffic_record(path=TRAFFIC_FILE, sources=KERNEL_SOURCES):
    """HBM bytes per launch measured with hardware counters (FETCH_SIZE + WRITE_SIZE,
    scaled by a plain copy of known size), if the record matches the current kernel
    sources; None otherwise."""
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_digest") != kernel_source_digest(sources):
        return None
    return rec.get("bytes_per_launch")


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=W.HEADLINE, choices=sorted(W.WORKLOADS) + sorted(W.EXTRA),
                    help="1-5: the five configurations; 6: a 144-frame clip (branch measurements)")
    ap.add_argument("--branch", default="joint", choices=["joint", "spatial", "temporal", "block"],
                    help="attention branch to measure (joint = the headline; block = all three and their sum)")
    ap.add_argument("--layers", type=int, default=10, help="stacked layers for --branch block")
    ap.add_argument("--ratios", default="0.2,0.5,0.8,1",
                    help="selective ratios measured by --branch block (share of layers recomputed/offloaded)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target length of the oracle timing")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--deterministic", action="store_true",
                    help="joint backward as separate dK/dV and dQ passes (bitwise reproducible) instead of "
                         "the fused pass")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after the run, copy this many MiB device-to-device with one plain copy "
                         "kernel (reference for hardware byte counters)")
    args = ap.parse_args(argv)
    if args.gpus != 1:
        print("bench.py measures one GPU only: the path shards by heads with no communication inside "
              "attention, so run --gpus 1 (got --gpus %d)" % args.gpus, file=sys.stderr)
        return 2

    import torch
    import paper_2501_08453_amd as vc

    w = W.get(args.workload)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.workload in W.EXTRA:
        g = W.make_inputs_device(w, device=dev)
        text_len = g.pop("text_len")
    else:
        x = W.make_inputs(w)
        g = {n: torch.from_numpy(x[n]).to(dev).to(torch.bfloat16).contiguous() for n in ("q", "k", "v", "do")}
        text_len = x["text_len"]
        del x
    tl = None if text_len is None else torch.from_numpy(text_len).to(dev)
    desc = vc.desc_for(w, deterministic=args.deterministic)
    # The joint backward bench.py times is the one vc_jointattn_bwd runs by default: fused,
    # unless the fused pass would carry no keys (head_dim 64), then the separate passes.
    separate = args.deterministic or vc.vc_jointattn_fused_dq_keys(desc) == 0
    if separate and not args.deterministic:
        desc = vc.desc_for(w, deterministic=True)
    B, N, H, D = w.shape
    o = torch.empty_like(g["q"])
    lse = torch.empty((B, H, N), dtype=torch.float32, device=dev)
    dq, dk, dv = (torch.empty_like(g["q"]) for _ in range(3))
    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream
    q, k, v, do = g["q"], g["k"], g["v"], g["do"]
    if args.branch == "temporal":  # no joint workspaces
        return branch_main(args, w, g, text_len, tl, desc, o, lse, dq, dk, dv, None, None, stream)
    if args.branch == "block":
        del o, lse, dq, dk, dv
        return block_main(args, w, g, text_len, tl, desc, stream)
    fws = vc.fwd_workspace(desc, dev)
    ws = vc.spatial_workspace(desc, dev) if args.branch == "spatial" else vc.workspace(desc, dev)
    fwsb, wsb = fws.numel(), ws.numel()
    if args.branch != "joint":
        return branch_main(args, w, g, text_len, tl, desc, o, lse, dq, dk, dv, fws, ws, stream)

    # Events bracket each stage on the stream the library launches on. Default: the fused
    # backward (stage 1; the key-stationary pass for dK, dV and, for the leading key
    # blocks, their dQ share: the accumulator fill, the kernel, the split tail's sum; the
    # dQ pass over the other keys); --deterministic: stage 1 with all token-major copies,
    # the dK/dV pass, the dQ pass over all keys.
    def step(ev=None):
        if ev:
            ev[0].record(stream)
        vc.vc_jointattn_fwd(desc, q, k, v, tl, None, o, lse, fws, fwsb, sh)
        if ev:
            ev[1].record(stream)
        vc.vc_jointattn_bwd_prepare(desc, q, k, o, lse, do, ws, wsb, sh)
        if ev:
            ev[2].record(stream)
        if separate:
            vc.vc_jointattn_bwd_dkdv(desc, q, k, v, do, tl, None, dk, dv, ws, wsb, sh)
        else:
            vc.vc_jointattn_bwd_fused(desc, q, k, v, do, tl, None, dk, dv, ws, wsb, sh)
        if ev:
            ev[3].record(stream)
        vc.vc_jointattn_bwd_dq(desc, q, k, v, do, tl, None, dq, ws, wsb, sh)
        if ev:
            ev[4].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    k_fwd = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    k_prep = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    k_dkdv = float(np.mean([e[2].elapsed_time(e[3]) for e in evs]))
    k_dq = float(np.mean([e[3].elapsed_time(e[4]) for e in evs]))

    f_fwd, f_bwd = flops(w, text_len)
    value = (f_fwd + f_bwd) / (ms_step * 1e-3) / 1e12
    # The dominant kernel is the key-stationary backward pass: it carries 3/4 of the
    # backward's algorithmic flops (the dP, dV, dK products of dP, dV, dK, dQ) and, fused,
    # the dQ product of its leading keys too (with text_len ragged the count is approximate
    # by the masked text keys); the dQ pass the rest of the dQ product (plus recomputation).
    fused_share = 0.0 if separate else vc.vc_jointattn_fused_dq_keys(desc) / N
    dkdv_flops = (0.75 + 0.25 * fused_share) * f_bwd
    dkdv_tflops = dkdv_flops / (k_dkdv * 1e-3) / 1e12
    line = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) q, k, v, dO of the workload's shape)",
        "config": {
            "workload": "%s: B=%d, H=%d, D=%d, %d text + %dx%dx%d video = %d tokens"
                        % (w.name, B, H, D, w.text_slot, w.frames, w.grid_h, w.grid_w, N),
            "batch": B, "heads": H, "head_dim": D, "tokens": N, "text_slot": w.text_slot,
            "frames": w.frames, "grid": [w.grid_h, w.grid_w],
        },
        "pct_of_peak": round(100.0 * value / PEAK_BF16_TFLOPS, 2),
        "algorithmic_tflop_per_step": round((f_fwd + f_bwd) / 1e12, 4),
        # The FlashAttention convention counts the backward as 2.5 forwards (its recomputed
        # Q K^T included): 14 instead of 12 flops per (query, key, dim) triple.
        "fa_convention_tflops": round((f_fwd + 2.5 * f_fwd) / (ms_step * 1e-3) / 1e12, 2),
        "backward": "separate dK/dV and dQ passes (deterministic)" if separate
                    else "fused (dQ of every key by fp32 atomics in the dK/dV pass)" if fused_share >= 1.0
                    else "fused (dQ of the leading %.0f%% of keys by fp32 atomics in the dK/dV pass)"
                    % (100 * fused_share),
        "kernels_ms": {"fwd": round(k_fwd, 4), "bwd_prepare": round(k_prep, 4),
                       ("bwd_dkdv" if separate else "bwd_fused"): round(k_dkdv, 4),
                       "bwd_dq": round(k_dq, 4)},
        "fwd_tflops": round(f_fwd / (k_fwd * 1e-3) / 1e12, 2),
        "bwd_tflops": round(f_bwd / ((k_prep + k_dkdv + k_dq) * 1e-3) / 1e12, 2),
        "roofline": {
            "bound": "mfma",
            "kernel": "bwd_dkdv_kernel" + ("" if separate else " (dQ fused)"),
            "achieved": round(dkdv_tflops, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(dkdv_tflops / PEAK_BF16_TFLOPS, 4),
            "traffic": None,
            "algorithmic_flops_per_launch": dkdv_flops,
        },
    }
    # the record is the fused kernel's, on the headline workload
    tr = None if separate or args.workload != W.HEADLINE else traffic_record()
    if tr is not None:
        line["roofline"]["traffic"] = tr
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, g, text_len, args.cpu_seconds)
    print(json.dumps(line), flush=True)
    copy_calibration(args.copy_calibration_mib, dev)
    return 0


def copy_calibration(mib, dev):
    """One plain device-to-device copy of `mib` MiB: the reference the hardware byte
    counters are scaled by."""
    if not mib:
        return
    import torch
    n = mib << 20
    src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()


def branch_main(args, w, g, text_len, tl, desc, o, lse, dq, dk, dv, fws, ws, stream):
    """Forward + backward of the spatial or temporal branch, events around each call."""
    import torch
    import paper_2501_08453_amd as vc
    q, k, v, do = g["q"], g["k"], g["v"], g["do"]
    sh = stream.cuda_stream
    B, N, H, D = w.shape

    def step(ev=None):
        if ev:
            ev[0].record(stream)
        if args.branch == "spatial":
            vc.vc_spatialattn_fwd(desc, q, k, v, tl, None, o, lse, fws, fws.numel(), sh)
        else:
            vc.vc_temporalattn_fwd(desc, q, k, v, None, o, lse, sh)
        if ev:
            ev[1].record(stream)
        if args.branch == "spatial":
            vc.vc_spatialattn_bwd(desc, q, k, v, o, lse, do, tl, None, dq, dk, dv, ws, ws.numel(), sh)
        else:
            vc.vc_temporalattn_bwd(desc, q, k, v, o, lse, do, None, dq, dk, dv, None, 0, sh)
        if ev:
            ev[2].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    k_fwd = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    k_bwd = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    if args.branch == "spatial":
        a_fwd, a_bwd = spatial_flops(w, text_len)
        scale, unit, peak, bound, metric = 1e12, "TFLOP/s", PEAK_BF16_TFLOPS, "mfma", METRIC_SPATIAL
    else:
        a_fwd, a_bwd = temporal_bytes(w)
        scale, unit, peak, bound, metric = 1e9, "GB/s", PEAK_HBM_GBS, "hbm", METRIC_TEMPORAL
    value = (a_fwd + a_bwd) / (ms_step * 1e-3) / scale
    # Dominant call: the backward (spatial: preparation and gradient kernels; temporal: one
    # gradient kernel that forms D and LSE*log2(e) itself, persistent for clips of more than
    # 32 frames, after the text-row fill).
    if args.branch == "spatial":
        bwd_label = "spatial backward (prepare + gradient kernels)"
    elif w.frames > 32:
        bwd_label = "temporal backward (one persistent kernel, D and LSE*log2(e) formed inside)"
    else:
        bwd_label = "temporal backward (gradient kernel, D and LSE*log2(e) formed inside)"
    bwd_rate = a_bwd / (k_bwd * 1e-3) / scale
    line = {
        "metric": metric, "value": round(value, 2), "unit": unit, "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) q, k, v, dO of the workload's shape)",
        "config": {
            "workload": "%s, %s branch: B=%d, H=%d, D=%d, %d text + %dx%dx%d video = %d tokens"
                        % (w.name, args.branch, B, H, D, w.text_slot, w.frames, w.grid_h, w.grid_w, N),
            "branch": args.branch, "batch": B, "heads": H, "head_dim": D, "tokens": N,
            "text_slot": w.text_slot, "frames": w.frames, "grid": [w.grid_h, w.grid_w],
        },
        "kernels_ms": {"fwd": round(k_fwd, 4), "bwd": round(k_bwd, 4)},
        "fwd_rate": round(a_fwd / (k_fwd * 1e-3) / scale, 2),
        "roofline": {"bound": bound, "kernel": bwd_label,
                     "achieved": round(bwd_rate, 2), "peak": peak, "unit": unit,
                     "frac": round(bwd_rate / peak, 4), "traffic": None,
                     "algorithmic_per_launch": a_bwd},
    }
    tr = (traffic_record(*TEMPORAL_TRAFFIC[args.workload])
          if args.branch == "temporal" and args.workload in TEMPORAL_TRAFFIC else None)
    if tr is not None:
        line["roofline"]["traffic"] = tr
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline_branch(args.branch, w, g, text_len, args.cpu_seconds)
    print(json.dumps(line), flush=True)
    copy_calibration(args.copy_calibration_mib, q.device)
    return 0


def pcie_rates(dev, mib=1024):
    """Device -> pinned host and pinned host -> device copy rates (GB/s) of one large copy."""
    import torch
    n = mib << 20
    d = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
    h = torch.empty(n, dtype=torch.uint8, pin_memory=True)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    h.copy_(d, non_blocking=True)  # warm
    torch.cuda.synchronize()
    ev[0].record()
    h.copy_(d, non_blocking=True)
    ev[1].record()
    d.copy_(h, non_blocking=True)
    ev[2].record()
    torch.cuda.synchronize()
    return n / (ev[0].elapsed_time(ev[1]) * 1e-3) / 1e9, n / (ev[1].elapsed_time(ev[2]) * 1e-3) / 1e9


def block_main(args, w, g, text_len, tl, desc, stream):
    """`--layers` stacked attention blocks (joint, spatial and temporal branches with the
    sum fused into the temporal forward), forward through every layer, then backward in
    reverse, as in a training step; q, k, v, dO are shared by the layers. Each layer saves
    the O and LSE of its three branches for its backward, and a plan (memory.plan) decides
    per layer whether that set is kept in HBM, recomputed before the layer's backward or
    offloaded to pinned host memory and loaded back (Sec. V-B). Measured: every layer kept,
    then recomputation, offloading and their combination (offloaded share 0.2, the rest
    recomputed) at each selective ratio of --ratios (the paper's tuned ratios by default).
    """
    import torch
    import paper_2501_08453_amd as vc
    from paper_2501_08453_amd import memory as mem
    q, k, v, do = g["q"], g["k"], g["v"], g["do"]
    B, N, H, D = w.shape
    K = max(1, args.layers)
    dev = q.device
    out = torch.empty_like(q)
    grads = tuple(tuple(torch.empty_like(q) for _ in range(3)) for _ in range(3))
    ratios = [float(x) for x in args.ratios.split(",") if x]

    def run(strategies):
        bs = mem.BlockStack(desc, [(q, k, v)] * K, strategies, [out] * K, [grads] * K, text_len=tl)
        try:
            for _ in range(args.warmup):
                bs.forward(stream)
                bs.backward([do] * K, stream)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(args.steps):
                bs.forward(stream)
                bs.backward([do] * K, stream)
            torch.cuda.synchronize()
            return (time.perf_counter() - t0) * 1e3 / args.steps, bs.set_bytes
        finally:
            bs.close()
            del bs
            torch.cuda.empty_cache()

    keep_ms, set_bytes = run(mem.plan(K, 0.0, "keep"))
    runs = []
    for ratio in ratios:
        for mode in ("recompute", "offload", "combination"):
            st = mem.plan(K, ratio, mode)
            ms, _ = run(st)
            n_off = st.count("offload")
            runs.append({"mode": mode, "selective_ratio": ratio, "offloaded_layers": n_off,
                         "recomputed_layers": st.count("recompute"), "ms_per_step": round(ms, 3),
                         "overhead": round(ms / keep_ms - 1.0, 4),
                         "device_saved_bytes": mem.device_sets(st) * set_bytes,
                         "host_bytes": n_off * set_bytes, "pcie_bytes_per_step": 2 * n_off * set_bytes})
            print("  %-11s ratio %.2f: %d offloaded, %d recomputed: %.2f ms (%+.1f%%)"
                  % (mode, ratio, n_off, st.count("recompute"), ms, 100 * (ms / keep_ms - 1)), file=sys.stderr,
                  flush=True)
    d2h, h2d = pcie_rates(dev)

    fj, bj = flops(w, text_len)
    fs, bs_ = spatial_flops(w, text_len)
    L = w.grid_h * w.grid_w
    ft = 4.0 * w.batch * w.heads * L * w.frames * w.frames * w.head_dim  # every video query, F keys
    block_flops = K * (fj + bj + fs + bs_ + 3.0 * ft)
    value = block_flops / (keep_ms * 1e-3) / 1e12
    line = {
        "metric": METRIC_BLOCK, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(keep_ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) q, k, v, dO of the workload's shape, shared by the layers)",
        "config": {
            "workload": "%s, parallel block x %d layers: B=%d, H=%d, D=%d, %d text + %dx%dx%d video = %d tokens"
                        % (w.name, K, B, H, D, w.text_slot, w.frames, w.grid_h, w.grid_w, N),
            "branch": "block", "layers": K, "batch": B, "heads": H, "head_dim": D, "tokens": N,
            "text_slot": w.text_slot, "frames": w.frames, "grid": [w.grid_h, w.grid_w],
        },
        "roofline": {"bound": "mfma", "kernel": "whole block step (all kernels)", "achieved": round(value, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(value / PEAK_BF16_TFLOPS, 4),
                     "traffic": None, "algorithmic_per_launch": block_flops},
        "memory_strategies": {
            "saved_bytes_per_layer": set_bytes, "offload_share_in_combination": mem.OFFLOAD_SHARE,
            "keep": {"ms_per_step": round(keep_ms, 3), "device_saved_bytes": K * set_bytes},
            "selective": runs,
            "pcie_GBps": {"d2h": round(d2h, 2), "h2d": round(h2d, 2)},
        },
        "cpu_baseline": None,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
