"""Properties of the compiled gfx950 kernels that the compiler does not check for us (CPU only:
hipcc cross-compiles the device code to assembly).

- The inline-assembly LDS copies set M0 themselves; a kernel that uses them must not rely on
  M0 anywhere else. Every M0 write must therefore be one copy's own, right before its
  global -> LDS instruction, and every such instruction must come from those copies.
- Packed fp32 arithmetic is disabled at build time; no packed fp32 add, multiply or fma may
  appear in any kernel.
- The hot joint-attention kernels and the long-clip temporal kernels fit their register
  budget without scratch spills; the spatial dK/dV instances, at the limit, touch scratch
  only outside the blocks that issue matrix-core work or LDS copies.
- No kernel waits for vector memory between the LDS copies of a batch: a compiler-inserted
  wait there (e.g. for a spill reload) would make each copy wait for the previous one.
"""
import os
import re
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2501_08453_amd import build as B  # noqa: E402

SOURCES = ["fwd.hip", "bwd.hip", "temporal.hip", "temporal_long.hip", "layout.hip", "offload.hip"]


@pytest.fixture(scope="module")
def device_asm(tmp_path_factory):
    try:
        cc = B.hipcc()
    except Exception as e:  # pragma: no cover - toolchain missing
        pytest.skip("hipcc not available: %s" % e)
    if not shutil.which(cc) and not os.path.exists(cc):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("asm")
    flags = [f for f in B.HIPCC_FLAGS if f not in ("-shared", "-fPIC")]
    asm = {}
    for fn in SOURCES:
        dst = str(out / (fn + ".s"))
        r = subprocess.run([cc, *flags, "-I", os.path.join(ROOT, "include"), "--cuda-device-only", "-S",
                            os.path.join(B.CSRC, fn), "-o", dst], capture_output=True, text=True, timeout=600)
        assert r.returncode == 0, r.stderr[-2000:]
        with open(dst) as f:
            asm[fn] = f.read()
    return asm


def kernels(text):
    """(mangled name, body) of every kernel in an assembly file."""
    for m in re.finditer(r"^(_Z\w+):", text, re.M):
        end = text.find(".Lfunc_end", m.end())
        yield m.group(1), text[m.end():end]


def instructions(body):
    for line in body.split("\n"):
        line = line.split(";", 1)[0].strip()
        if line and not line.startswith(".") and not line.endswith(":"):
            yield line


def test_m0_is_set_only_by_the_lds_copies(device_asm):
    seen_copies = 0
    for fn, text in device_asm.items():
        for name, body in kernels(text):
            ins = list(instructions(body))
            for i, line in enumerate(ins):
                if re.search(r"\bm0\b", line):
                    assert re.match(r"s_mov_b32 m0, (s\d+|vcc_lo|vcc_hi)$", line), (fn, name, line)  # an SGPR
                    nxt = [x for x in ins[i + 1:i + 3] if not x.startswith("s_nop")]
                    assert nxt and nxt[0].startswith("global_load_lds_dwordx4"), (fn, name, ins[i:i + 3])
                if line.startswith("global_load_lds") or re.match(r"buffer_load\w*.*\blds\b", line):
                    prev = [x for x in ins[max(0, i - 2):i] if not x.startswith("s_nop")]
                    assert prev and prev[-1].startswith("s_mov_b32 m0,"), (fn, name, ins[max(0, i - 2):i + 1])
                    seen_copies += 1
    assert seen_copies > 0  # the forward, dK/dV and dQ kernels all copy tiles this way


def test_no_packed_fp32_arithmetic(device_asm):
    for fn, text in device_asm.items():
        hits = re.findall(r"\bv_pk_(?:add|mul|fma)_f32\b", text)
        assert not hits, (fn, hits[:3])


HOT = [
    ("fwd.hip", "fwd_kernelILi128ELb0EE"),
    ("fwd.hip", "fwd_kernelILi64ELb0EE"),
    ("fwd.hip", "fwd_kernelILi128ELb1EE"),  # with a key mask
    ("bwd.hip", "bwd_dkdv_kernelILi128ELb0ELb1EE"),  # fused joint dK/dV (+dQ)
    ("bwd.hip", "bwd_dkdv_kernelILi128ELb0ELb0EE"),  # separate joint dK/dV
    ("bwd.hip", "bwd_dq_kernelILi128ELb0EE"),
    ("bwd.hip", "bwd_dq_kernelILi64ELb0EE"),
    ("bwd.hip", "bwd_dq_kernelILi128ELb1EE"),
    ("temporal_long.hip", "temporal_long_fwd_kernelILi128ELb0EE"),  # clips of 33-144 frames
    ("temporal_long.hip", "temporal_long_fwd_kernelILi128ELb1EE"),
    ("temporal_long.hip", "temporal_long_bwd_kernelILi128EE"),
]


@pytest.mark.parametrize("fn,kernel", HOT, ids=[k for _, k in HOT])
def test_hot_kernels_do_not_spill(device_asm, fn, kernel):
    text = device_asm[fn]
    m = re.search(r"\.name:\s+_Z\w*%s\w*\n(?:.*\n){0,40}?\s+\.vgpr_spill_count:\s+(\d+)" % kernel, text)
    assert m, kernel
    assert int(m.group(1)) == 0, (kernel, "spills", m.group(1))


def basic_blocks(body):
    return re.split(r"\n\.LBB\d+_\d+:", body)


def test_no_vector_memory_wait_among_lds_copies(device_asm):
    """In a basic block that issues LDS copies, the only vector-memory waits are the
    kernels' own waits for a stage's copies: full waits right before a barrier, or the
    explicit wait for every counter (s_waitcnt 0, which names expcnt) of a one-wave
    workgroup. Any other vmcnt wait there, e.g. one the compiler inserts for a spill reload
    at the head of a copy loop, waits for every copy in flight, the ones just issued
    included."""
    checked = 0
    for fn, text in device_asm.items():
        for name, body in kernels(text):
            for blk in basic_blocks(body):
                ins = list(instructions(blk))
                if not any(l.startswith("global_load_lds") for l in ins):
                    continue
                checked += 1
                for i, line in enumerate(ins):
                    if line.startswith("s_waitcnt") and "vmcnt" in line:
                        nxt = ins[i + 1] if i + 1 < len(ins) else ""
                        explicit = all(c in line for c in ("vmcnt(0)", "expcnt(0)", "lgkmcnt(0)"))
                        assert nxt.startswith("s_barrier") or explicit, (fn, name, line, ins[max(0, i - 3):i + 3])
    assert checked > 0


@pytest.mark.parametrize("kernel", ["bwd_dkdv_kernelILi128ELb1ELb1EE", "bwd_dkdv_kernelILi128ELb1ELb0EE"])
def test_spatial_dkdv_scratch_outside_hot_blocks(device_asm, kernel):
    """The spatial dK/dV instances (the default fused one and the deterministic one) use all
    256 registers; what they spill is set up and read back outside the walk's blocks: no
    basic block holds both a scratch access and a matrix-core op or an LDS copy."""
    text = device_asm["bwd.hip"]
    bodies = [b for n, b in kernels(text) if kernel in n]
    assert len(bodies) == 1, kernel
    for blk in basic_blocks(bodies[0]):
        ins = list(instructions(blk))
        if any(l.startswith("scratch_") for l in ins):
            assert not any(l.startswith("v_mfma") or l.startswith("global_load_lds") for l in ins), (kernel, ins[:8])
