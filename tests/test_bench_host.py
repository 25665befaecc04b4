"""Host-side logic of bench.py (CPU only): the one-GPU guard, the algorithmic work counts
behind the reported rates, and the tie between a traffic record and the kernel sources."""
import json
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import workloads as W  # noqa: E402


def test_more_than_one_gpu_is_refused():
    assert bench.main(["--gpus", "2"]) == 2
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "8"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""  # no JSON line for a configuration that was not measured


def test_joint_flops_of_the_headline_workload():
    w = W.WORKLOADS[W.HEADLINE]
    fwd, bwd = bench.flops(w, None)
    # 4 N^2 D per (sample, head) forward: QK^T and PV, two flops per multiply-add
    assert fwd == 4.0 * 24 * 57856 * 57856 * 128
    assert bwd == 2.0 * fwd
    assert round((fwd + bwd) / 1e12, 4) == 123.3955


def _valid_keys_by_count(w, text_len):
    """Keys a query attends to, counted one by one: text keys below the sample's text length,
    every video key."""
    out = []
    for t in text_len:
        keys = np.arange(w.tokens)
        valid = (keys >= w.text_slot) | (keys < min(max(int(t), 0), w.text_slot))
        out.append(int(valid.sum()))
    return out


@pytest.mark.parametrize("text_len", [[0, 5, 16, 40], [16, 16, 16, 16], [-3, 99, 7, 1]])
def test_joint_flops_with_padded_text(text_len):
    w = W.custom(4, 3, 64, 16, 2, 4, 5)
    fwd, bwd = bench.flops(w, np.asarray(text_len, dtype=np.int32))
    nkv = _valid_keys_by_count(w, text_len)
    assert fwd == sum(4.0 * w.heads * w.tokens * n * w.head_dim for n in nkv)
    assert bwd == 2.0 * fwd


def test_spatial_flops_count_text_and_own_frame_keys():
    w = W.custom(2, 3, 64, 16, 3, 4, 5)
    text_len = np.asarray([7, 16], dtype=np.int32)
    fwd, bwd = bench.spatial_flops(w, text_len)
    L = w.grid_h * w.grid_w
    pairs = 0
    for t in text_len:  # every video query: the valid text keys and the L keys of its frame
        for f in range(w.frames):
            for _ in range(L):
                pairs += int(t) + L
    assert fwd == 4.0 * w.heads * w.head_dim * pairs
    assert bwd == 2.0 * fwd


def test_temporal_bytes_of_the_headline_workload():
    w = W.WORKLOADS[W.HEADLINE]
    fwd, bwd = bench.temporal_bytes(w)
    rows = 16 * 45 * 80 * 24
    tensor = rows * 128 * 2  # one bf16 [video rows, heads, D] tensor
    assert fwd == 4 * tensor + 4 * rows  # q, k, v read; o written; fp32 LSE written
    assert bwd == 8 * tensor + 4 * rows  # q, k, v, o, dO read; dq, dk, dv written; LSE read
    assert round(fwd / 1e9, 2) == 1.42 and round(bwd / 1e9, 2) == 2.84


def test_extra_workloads_are_bench_only():
    """The 144-frame clip is selectable by id but is none of the five configurations."""
    w = W.get(6)
    assert 6 not in W.WORKLOADS and w.frames == 144 and w.tokens == 256 + 144 * 45 * 80
    assert W.get(3) is W.WORKLOADS[3]


def test_code_only_drops_comments_and_blank_lines():
    src = "int a = 1;  // one\n\n// a whole comment line\n   \nint b = a;\n"
    assert bench.code_only(src) == "int a = 1;\nint b = a;"


def _write(path, text):
    with open(path, "w", encoding="utf-8") as f:
        f.write(text)


def test_traffic_record_follows_the_code_not_the_comments(tmp_path):
    src = tmp_path / "kernel.hip"
    _write(src, "__global__ void k() {}  // first\n")
    sources = [str(src)]  # absolute: os.path.join keeps it as is
    rec = tmp_path / "traffic.json"
    _write(rec, json.dumps({"bytes_per_launch": 1234, "source_digest": bench.kernel_source_digest(sources)}))
    assert bench.traffic_record(str(rec), sources) == 1234
    _write(src, "// a new comment\n__global__ void k() {}  // reworded\n\n")
    assert bench.traffic_record(str(rec), sources) == 1234  # commentary changed only
    _write(src, "__global__ void k() { int x = 0; }\n")
    assert bench.traffic_record(str(rec), sources) is None  # the code changed: the record is stale
    assert bench.traffic_record(str(tmp_path / "missing.json"), sources) is None
    _write(rec, "not json")
    assert bench.traffic_record(str(rec), sources) is None
