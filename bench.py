#!/usr/bin/env python3
"""Throughput of joint text-video attention (forward + backward) on one MI355X.

One step = one pass of the whole path over one batch of synthetic input:
forward (O, LSE), backward prepare (D = rowsum(dO o O), token-major copies),
backward dK/dV and backward dQ, all through the C ABI on torch's current
stream. Inputs are resident in HBM before timing.

Prints one JSON line. `value` is algorithmic TFLOP/s of the whole step:
12 * H * N * N_kv * D per sample (forward 4, backward 8; the backward's
recomputation of Q K^T is not counted).
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
METRIC = "joint-attention fwd+bwd TFLOP/s and % bf16 MFMA peak at 57,856 tokens"


def valid_keys_per_sample(w, text_len):
    if text_len is None:
        return [w.tokens] * w.batch
    tl = np.clip(np.asarray(text_len), 0, w.text_slot)
    return [int(w.tokens - (w.text_slot - t)) for t in tl]


def flops(w, text_len):
    nkv = valid_keys_per_sample(w, text_len)
    fwd = sum(4.0 * w.heads * w.tokens * n * w.head_dim for n in nkv)
    return fwd, 2.0 * fwd


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


def kernel_source_digest() -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def traffic_record():
    """HBM bytes per launch of the dK/dV kernel measured with hardware counters (FETCH_SIZE
    + WRITE_SIZE, scaled by a plain copy of known size), if the record matches the current
    kernel sources; None otherwise."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_digest") != kernel_source_digest():
        return None
    return rec.get("bytes_per_launch")


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=W.HEADLINE, choices=sorted(W.WORKLOADS))
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target length of the oracle timing")
    ap.add_argument("--no-cpu-baseline", action="store_true")
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

    w = W.WORKLOADS[args.workload]
    x = W.make_inputs(w)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    g = {n: torch.from_numpy(x[n]).to(dev).to(torch.bfloat16).contiguous() for n in ("q", "k", "v", "do")}
    text_len = x["text_len"]
    tl = None if text_len is None else torch.from_numpy(text_len).to(dev)
    del x
    desc = vc.desc_for(w)
    B, N, H, D = w.shape
    o = torch.empty_like(g["q"])
    lse = torch.empty((B, H, N), dtype=torch.float32, device=dev)
    dq, dk, dv = (torch.empty_like(g["q"]) for _ in range(3))
    fws = vc.fwd_workspace(desc, dev)
    ws = vc.workspace(desc, dev)
    fwsb, wsb = fws.numel(), ws.numel()
    q, k, v, do = g["q"], g["k"], g["v"], g["do"]
    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream

    # Events bracket each stage on the stream the library launches on.
    def step(ev=None):
        if ev:
            ev[0].record(stream)
        vc.vc_jointattn_fwd(desc, q, k, v, tl, None, o, lse, fws, fwsb, sh)
        if ev:
            ev[1].record(stream)
        vc.vc_jointattn_bwd_prepare(desc, q, k, o, lse, do, ws, wsb, sh)
        if ev:
            ev[2].record(stream)
        vc.vc_jointattn_bwd_dkdv(desc, q, k, v, do, tl, None, dk, dv, ws, wsb, sh)
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
    # The dK/dV kernel carries 3/4 of the backward's algorithmic flops (dP, dV, dK of
    # dP, dV, dK, dQ); the dQ kernel the remaining dQ product (plus its recomputation).
    dkdv_flops = 0.75 * f_bwd
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
        "kernels_ms": {"fwd": round(k_fwd, 4), "bwd_prepare": round(k_prep, 4), "bwd_dkdv": round(k_dkdv, 4),
                       "bwd_dq": round(k_dq, 4)},
        "fwd_tflops": round(f_fwd / (k_fwd * 1e-3) / 1e12, 2),
        "bwd_tflops": round(f_bwd / ((k_prep + k_dkdv + k_dq) * 1e-3) / 1e12, 2),
        "roofline": {
            "bound": "mfma",
            "kernel": "bwd_dkdv_kernel",
            "achieved": round(dkdv_tflops, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(dkdv_tflops / PEAK_BF16_TFLOPS, 4),
            "traffic": None,
            "algorithmic_flops_per_launch": dkdv_flops,
        },
    }
    tr = traffic_record()
    if tr is not None:
        line["roofline"]["traffic"] = tr
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, g, text_len, args.cpu_seconds)
    print(json.dumps(line), flush=True)
    if args.copy_calibration_mib:
        n = args.copy_calibration_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
    return 0


if __name__ == "__main__":
    sys.exit(main())
