"""Host-side checks of the C ABI: the library loads, exports what the header
declares, and reports argument errors before touching a device.

No call here reaches a kernel launch: every call fails validation first (the
device-error case runs only where no GPU is present).
"""
import ctypes

import pytest

import paper_2501_08453_amd as vc


@pytest.fixture(scope="module")
def lib():
    return vc._lib()


def good_desc(**kw):
    d = dict(batch=1, heads=2, head_dim=64, text_slot=16, frames=2, grid_h=8, grid_w=8)
    d.update(kw)
    return vc.make_desc(**d)


def test_exports_every_declared_function(lib):
    names = vc.header_functions()
    assert set(names) >= {"vc_jointattn_fwd", "vc_jointattn_bwd", "vc_jointattn_bwd_workspace_bytes",
                          "vc_status_string", "vc_jointattn_abi_version"}
    for n in names:
        assert hasattr(lib, n), n
    assert set(vc._SIGS) == set(names)


def test_version_and_strings(lib):
    assert vc.vc_jointattn_abi_version() == vc.ABI_VERSION
    for code in vc.STATUS:
        assert isinstance(vc.vc_status_string(code), str) and vc.vc_status_string(code)
    assert vc.vc_status_string(12345) == "unknown status"


def test_tokens_and_workspace():
    d = good_desc()
    assert vc.vc_jointattn_tokens(d) == 16 + 2 * 8 * 8
    d3 = vc.make_desc(1, 24, 128, 256, 16, 45, 80)
    n = 57856
    assert vc.vc_jointattn_tokens(d3) == n
    npad = (n + 63) // 64 * 64
    al = lambda x: (x + 255) // 256 * 256  # noqa: E731
    rows = al(24 * npad * 4)
    tiles = al(24 * (npad // 64) * 128 * 72 * 2)
    # V^T tiles, then per row of up to 256 split workgroups: fp32 O, base and sum
    assert vc.vc_jointattn_fwd_workspace_bytes(d3) == tiles + 256 * 256 * (128 + 2) * 4
    # fp32 partial dK, dV of up to 256 split workgroups of 256 keys (the last, partial round
    # of the 5,424 workgroups)
    tail = 2 * 256 * 256 * 128 * 4
    assert vc.vc_jointattn_bwd_workspace_bytes(d3) == 2 * rows + 3 * tiles + tail
    assert vc.vc_jointattn_tokens(good_desc(head_dim=96)) == -3
    assert vc.vc_jointattn_bwd_workspace_bytes(good_desc(frames=0)) == 0
    # spatial: the 900 video query tiles of the text key block split into 16 chunks of
    # about one frame (57 tiles), fp32 partial dK and dV of its 256 keys per chunk
    part = 2 * 16 * 24 * 256 * 128 * 4
    assert vc.vc_spatialattn_bwd_workspace_bytes(d3) == 2 * rows + 3 * tiles + tail + part
    # no text, or too few video tiles to split: the joint size
    for kw in (dict(text_slot=0), dict()):
        dd = good_desc(**kw)
        assert vc.vc_spatialattn_bwd_workspace_bytes(dd) == vc.vc_jointattn_bwd_workspace_bytes(dd)
    assert vc.vc_spatialattn_bwd_workspace_bytes(good_desc(frames=0)) == 0


@pytest.mark.parametrize("kw,code", [
    (dict(head_dim=96), -3), (dict(head_dim=0), -3), (dict(batch=0), -2), (dict(heads=0), -2),
    (dict(text_slot=-1), -2), (dict(frames=0), -2), (dict(grid_h=-3), -2), (dict(grid_w=0), -2),
    (dict(frames=1 << 20, grid_h=1 << 10, grid_w=4), -2),
])
def test_bad_descriptor(lib, kw, code):
    d = good_desc(**kw)
    p = 1 << 20  # never dereferenced: validation fails first
    assert lib.vc_jointattn_fwd(ctypes.byref(d), p, p, p, None, None, p, p, p, 1 << 30, None) == code
    assert lib.vc_jointattn_bwd(ctypes.byref(d), p, p, p, p, p, p, None, None, p, p, p, p, 1 << 30, None) == code


def test_null_descriptor_and_pointers(lib):
    p = 1 << 20
    assert lib.vc_jointattn_fwd(None, p, p, p, None, None, p, p, p, 1 << 30, None) == -1
    d = good_desc()
    assert lib.vc_jointattn_fwd(ctypes.byref(d), None, p, p, None, None, p, p, p, 1 << 30, None) == -1
    assert lib.vc_jointattn_fwd(ctypes.byref(d), p, p, p, None, None, p, None, p, 1 << 30, None) == -1
    assert lib.vc_jointattn_bwd(ctypes.byref(d), p, p, p, p, p, None, None, None, p, p, p, p, 1 << 30, None) == -1
    assert lib.vc_jointattn_bwd_dkdv(ctypes.byref(d), p, p, None, p, None, None, p, p, p, 1 << 30, None) == -1
    assert lib.vc_jointattn_bwd_dq(ctypes.byref(d), p, p, p, p, None, None, None, p, 1 << 30, None) == -1
    assert lib.vc_jointattn_bwd_fused(ctypes.byref(d), p, p, p, p, None, None, p, None, p, 1 << 30, None) == -1
    assert lib.vc_jointattn_bwd_fused(None, p, p, p, p, None, None, p, p, p, 1 << 30, None) == -1


def test_fused_dq_keys():
    """Keys whose dQ share the fused pass carries: head_dim 128, the leading 65% of the
    256-key blocks, rounded to whole blocks, never more than N; head_dim 64 every key; an
    invalid descriptor gives its status."""
    long720p = vc.make_desc(1, 24, 128, 256, 16, 45, 80)  # 57,856 tokens, 226 blocks
    assert vc.vc_jointattn_fused_dq_keys(long720p) == 147 * 256
    tiny = vc.make_desc(1, 1, 128, 0, 1, 1, 5)  # 5 tokens, one block
    assert vc.vc_jointattn_fused_dq_keys(tiny) == 5
    for n_blocks in (1, 2, 3, 7, 100):
        d = vc.make_desc(1, 1, 128, 0, 1, 1, 256 * n_blocks)
        k = vc.vc_jointattn_fused_dq_keys(d)
        assert k % 256 == 0 and 0 <= k <= 256 * n_blocks
        assert k == 256 * ((n_blocks * 65 + 50) // 100)
        assert vc.vc_jointattn_fused_dq_keys(vc.make_desc(1, 1, 64, 0, 1, 1, 256 * n_blocks)) == 256 * n_blocks
        assert vc.vc_jointattn_fused_dq_keys(vc.make_desc(1, 1, 64, 0, 1, 1, 256 * n_blocks - 3)) == 256 * n_blocks - 3
    assert vc.vc_jointattn_fused_dq_keys(vc.make_desc(1, 1, 96, 0, 1, 1, 5)) == -3  # head_dim
    # The fused pass addresses a sample's dQ accumulator with 32-bit offsets: none of it
    # once N*H*D reaches 2^32 (here 1,166,656 tokens, 144 frames of 8,100 like the paper's
    # 1.16M-token clip, at 32 heads; at 8 heads it stays below)
    big = vc.make_desc(1, 32, 128, 256, 144, 90, 90)
    n = vc.vc_jointattn_tokens(big)
    assert n * 32 * 128 >= 1 << 32 and vc.vc_jointattn_fused_dq_keys(big) == 0
    below = vc.make_desc(1, 8, 128, 256, 144, 90, 90)
    assert vc.vc_jointattn_tokens(below) * 8 * 128 < 1 << 32
    assert vc.vc_jointattn_fused_dq_keys(below) > 0


def test_misaligned_pointers(lib):
    d = good_desc()
    p = 1 << 20
    assert lib.vc_jointattn_fwd(ctypes.byref(d), p + 2, p, p, None, None, p, p, p, 1 << 30, None) == -4
    assert lib.vc_jointattn_fwd(ctypes.byref(d), p, p, p, p + 2, None, p, p, p, 1 << 30, None) == -4  # text_len
    assert lib.vc_jointattn_fwd(ctypes.byref(d), p, p, p, None, None, p, p, p + 16, 1 << 30, None) == -4  # ws 256
    assert lib.vc_jointattn_bwd_prepare(ctypes.byref(d), p, p, p, p, p, p + 16, 1 << 30, None) == -4
    assert lib.vc_jointattn_bwd_dq(ctypes.byref(d), p, p, p, p, None, None, p + 8, p, 1 << 30, None) == -4
    assert lib.vc_jointattn_bwd_fused(ctypes.byref(d), p, p, p, p, None, None, p + 8, p, p, 1 << 30, None) == -4
    assert lib.vc_jointattn_bwd_fused(ctypes.byref(d), p, p, p, p, None, None, p, p, p + 64, 1 << 30, None) == -4


def test_workspace_checks(lib):
    d = good_desc()
    p = 1 << 20
    need = vc.vc_jointattn_bwd_workspace_bytes(d)
    assert lib.vc_jointattn_bwd_prepare(ctypes.byref(d), p, p, p, p, p, None, need, None) == -5
    assert lib.vc_jointattn_bwd_prepare(ctypes.byref(d), p, p, p, p, p, p, need - 1, None) == -5
    assert lib.vc_jointattn_bwd(ctypes.byref(d), p, p, p, p, p, p, None, None, p, p, p, p, need - 4, None) == -5
    fneed = vc.vc_jointattn_fwd_workspace_bytes(d)
    assert lib.vc_jointattn_fwd(ctypes.byref(d), p, p, p, None, None, p, p, None, fneed, None) == -5
    assert lib.vc_jointattn_fwd(ctypes.byref(d), p, p, p, None, None, p, p, p, fneed - 1, None) == -5
    # the spatial backward needs more than the joint workspace when its text keys are split
    # (long video: 16 chunks); rejected before anything runs
    d3 = vc.make_desc(1, 24, 128, 256, 16, 45, 80)
    joint, spatial = vc.vc_jointattn_bwd_workspace_bytes(d3), vc.vc_spatialattn_bwd_workspace_bytes(d3)
    assert spatial > joint
    assert lib.vc_spatialattn_bwd(ctypes.byref(d3), p, p, p, p, p, p, None, None, p, p, p, p, joint, None) == -5
    assert lib.vc_spatialattn_bwd(ctypes.byref(d3), p, p, p, p, p, p, None, None, p, p, p, p, spatial - 1,
                                  None) == -5


def test_no_device_is_reported():
    torch = pytest.importorskip("torch")
    if torch.cuda.is_available():
        pytest.skip("a GPU is present; this case checks the error path without one")
    lib = vc._lib()
    d = good_desc()
    p = 1 << 20
    assert lib.vc_jointattn_fwd(ctypes.byref(d), p, p, p, None, None, p, p, p, 1 << 30, None) == -6


def test_binding_fails_loudly_without_library(monkeypatch):
    monkeypatch.setattr(vc, "_LIB", None)
    monkeypatch.setattr(vc, "LIB_PATH", "/nonexistent/libvc_jointattn.so")
    with pytest.raises(RuntimeError, match="not built"):
        vc.vc_jointattn_abi_version()


def test_temporal_argument_errors(lib):
    p = 1 << 20
    d = good_desc()
    # more than 144 frames is outside what the long-clip kernel stages in LDS
    big = good_desc(frames=145, grid_h=2, grid_w=2)
    assert lib.vc_temporalattn_fwd(ctypes.byref(big), p, p, p, None, p, p, None) == -2
    assert lib.vc_temporalattn_bwd(ctypes.byref(big), p, p, p, p, p, p, None, p, p, p, p, 1 << 30, None) == -2
    assert lib.vc_temporalattn_fwd(ctypes.byref(good_desc(head_dim=48)), p, p, p, None, p, p, None) == -3
    assert lib.vc_temporalattn_fwd(ctypes.byref(d), p, None, p, None, p, p, None) == -1
    assert lib.vc_temporalattn_fwd(ctypes.byref(d), p, p, p, None, p + 4, p, None) == -4
    need = vc.vc_temporalattn_bwd_workspace_bytes(d)
    npad = (16 + 2 * 64 + 63) // 64 * 64
    assert need == 2 * ((2 * npad * 4 + 255) // 256 * 256)
    assert vc.vc_temporalattn_bwd_workspace_bytes(good_desc(batch=0)) == 0
    # the backward reads no workspace at any clip length: NULL and a short size are not
    # refused, so with a missing pointer the call stops at that pointer (only refusal
    # paths are exercised: with every pointer set and a GPU present the call would run)
    longc = good_desc(frames=144, grid_h=1, grid_w=3)
    assert lib.vc_temporalattn_fwd(ctypes.byref(longc), p, p, p, None, p, p + 4, None) == -4
    for desc in (d, longc):
        assert lib.vc_temporalattn_bwd(ctypes.byref(desc), p, p, p, p, p, p, None, p, p, None, None, 0, None) == -1
        assert lib.vc_temporalattn_bwd(ctypes.byref(desc), p, p, p, p, p, None, None, p, p, p, None, 0, None) == -1


def test_branch_sum_argument_errors(lib):
    d = good_desc()
    p = 1 << 20
    # nothing to sum, or no output
    assert lib.vc_branchsum(ctypes.byref(d), None, None, None, p, None) == -1
    assert lib.vc_branchsum(ctypes.byref(d), p, p, p, None, None) == -1
    assert lib.vc_branchsum(ctypes.byref(d), p, p + 8, None, p, None) == -4
    assert lib.vc_branchsum(ctypes.byref(good_desc(heads=0)), p, p, p, p, None) == -2
    # fused temporal forward + sum: out required, must not be this branch's o
    assert lib.vc_temporalattn_fwd_sum(ctypes.byref(d), p, p, p, None, p, p, p, p, None, None) == -1
    assert lib.vc_temporalattn_fwd_sum(ctypes.byref(d), p, p, p, None, p, p, p, p, p, None) == -9
    assert lib.vc_temporalattn_fwd_sum(ctypes.byref(d), p, p, p, None, p + 2, None, p, p, p * 2, None) == -4
    assert vc.vc_status_string(-9) == "an output is the same buffer as another output"


def test_offload_argument_errors(lib):
    p = 1 << 20
    assert lib.vc_offload_create(None) == -1
    assert lib.vc_offload_destroy(None) == -1
    assert lib.vc_offload_wait(None, None) == -1
    assert lib.vc_offload_store(None, p, p, 16, None) == -1
    assert lib.vc_offload_load(None, p, p, 16, None) == -1
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        h = ctypes.c_void_p(123)
        assert lib.vc_offload_create(ctypes.byref(h)) == -6
        assert h.value is None


def _header_define(name):
    import re
    with open(vc.HEADER) as f:
        m = re.search(r"#define\s+%s\s+(.+)" % name, f.read())
    return m.group(1).strip()


def test_binding_constants_match_header():
    assert int(_header_define("VC_JOINTATTN_ABI_VERSION")) == vc.ABI_VERSION
    assert _header_define("VC_JOINTATTN_NOALLOC_SCRATCH_BYTES") == "((size_t)256 << 20)"
    assert vc.NOALLOC_SCRATCH_BYTES == 256 << 20


def test_binding_refuses_other_abi_version(tmp_path, monkeypatch):
    """A library reporting another ABI version is refused before any other symbol is bound
    (a binding passing a newer argument list to an older entry point would hand it a device
    pointer where it expects the stream)."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc") or shutil.which("cc")
    if gcc is None:
        pytest.skip("no host C compiler")
    src = tmp_path / "old.c"
    src.write_text("int vc_jointattn_abi_version(void) { return %d; }\n" % (vc.ABI_VERSION - 1))
    so = tmp_path / "libold.so"
    subprocess.run([gcc, "-shared", "-fPIC", str(src), "-o", str(so)], check=True)
    monkeypatch.setattr(vc, "_LIB", None)
    monkeypatch.setattr(vc, "LIB_PATH", str(so))
    with pytest.raises(RuntimeError, match="C ABI version %d, this binding version %d"
                       % (vc.ABI_VERSION - 1, vc.ABI_VERSION)):
        vc.vc_jointattn_tokens(good_desc())
    assert vc._LIB is None


def test_noalloc_forward_argument_errors(lib):
    """The no-allocation forward validates the descriptor, then refuses problems whose
    workspace exceeds its fixed scratch array (before touching a device), then checks the
    device and the pointers."""
    p = 1 << 20
    assert lib.vc_jointattn_fwd_noalloc(None, p, p, p, None, None, p, p, None) == -1
    assert lib.vc_jointattn_fwd_noalloc(ctypes.byref(good_desc(head_dim=96)), p, p, p, None, None, p, p,
                                        None) == -3
    long720p = vc.make_desc(1, 24, 128, 256, 16, 45, 80)  # 400 MB of V^T tiles
    assert vc.vc_jointattn_fwd_workspace_bytes(long720p) > vc.NOALLOC_SCRATCH_BYTES
    assert lib.vc_jointattn_fwd_noalloc(ctypes.byref(long720p), p, p, p, None, None, p, p, None) == -10
    assert "no-allocation" in vc.vc_status_string(-10)
    # one GPU's share of it under 8-way head sharding (3 heads) fits
    share = vc.make_desc(1, 3, 128, 256, 16, 45, 80)
    assert vc.vc_jointattn_fwd_workspace_bytes(share) <= vc.NOALLOC_SCRATCH_BYTES
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        assert lib.vc_jointattn_fwd_noalloc(ctypes.byref(share), p, p, p, None, None, p, p, None) == -6


def test_binding_validates_before_calling():
    """fwd()/bwd() check the tensors against each other and the descriptor before the
    library sees them: a descriptor larger than the tensors, a wrong dtype for text_len or
    key_mask, or a wrong LSE shape raise ValueError; shapes are checked before placement."""
    torch = pytest.importorskip("torch")
    B, N, H, D = 1, 16 + 2 * 64, 2, 64
    t = lambda: torch.zeros((B, N, H, D), dtype=torch.bfloat16)  # noqa: E731
    q, k, v, o, do = t(), t(), t(), t(), t()
    lse = torch.zeros((B, H, N), dtype=torch.float32)
    d = good_desc()
    big = good_desc(frames=3)
    with pytest.raises(ValueError, match="descriptor gives N"):
        vc.bwd(q, k, v, o, lse, do, big)
    with pytest.raises(ValueError, match="descriptor gives N"):
        vc.fwd(q, k, v, big)
    with pytest.raises(ValueError, match="descriptor gives B=1, H=3"):
        vc.bwd(q, k, v, o, lse, do, good_desc(heads=3))
    with pytest.raises(ValueError, match="text_len must be torch.int32"):
        vc.bwd(q, k, v, o, lse, do, d, text_len=torch.zeros(B, dtype=torch.int64))
    with pytest.raises(ValueError, match="key_mask has shape"):
        vc.bwd(q, k, v, o, lse, do, d, key_mask=torch.zeros((B, N + 1), dtype=torch.uint8))
    with pytest.raises(ValueError, match="lse has shape"):
        vc.bwd(q, k, v, o, lse[:, :, :-1], do, d)
    with pytest.raises(ValueError, match="dout must be torch.bfloat16"):
        vc.bwd(q, k, v, o, lse, do.float(), d)
    with pytest.raises(ValueError, match="must be on a GPU"):
        vc.bwd(q, k, v, o, lse, do, d)
    with pytest.raises(ValueError, match="descriptor gives N"):
        vc.spatial_bwd(q, k, v, o, lse, do, big)
    with pytest.raises(ValueError, match="text_len must be torch.int32"):
        vc.spatial_fwd(q, k, v, d, text_len=torch.zeros(B, dtype=torch.int64))
    with pytest.raises(ValueError, match="descriptor gives N"):
        vc.temporal_bwd(q, k, v, o, lse, do, big)
