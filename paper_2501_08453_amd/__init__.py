"""Joint text-video attention for MI355X (gfx950): Python binding.

Thin ctypes binding over libvc_jointattn.so (include/vc_jointattn.h). It only
marshals arguments: every step of the computation runs in the library's HIP
kernels. PyTorch supplies device memory and the stream. If the library is
not built, every call raises; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
import re

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG_DIR, "libvc_jointattn.so")
HEADER = os.path.join(os.path.dirname(PKG_DIR), "include", "vc_jointattn.h")

# The ABI the signatures below describe (VC_JOINTATTN_ABI_VERSION of include/vc_jointattn.h);
# a library reporting another version is refused, so that no call can reach an entry point
# whose arguments differ from what this binding passes.
ABI_VERSION = 10
# Bytes of the no-allocation forward's fixed scratch array (VC_JOINTATTN_NOALLOC_SCRATCH_BYTES).
NOALLOC_SCRATCH_BYTES = 256 << 20

VC_OK = 0
STATUS = {
    0: "VC_OK", -1: "VC_ERR_NULL", -2: "VC_ERR_SHAPE", -3: "VC_ERR_HEAD_DIM", -4: "VC_ERR_ALIGN",
    -5: "VC_ERR_WORKSPACE", -6: "VC_ERR_DEVICE", -7: "VC_ERR_HIP", -8: "VC_ERR_UNSUPPORTED",
    -9: "VC_ERR_ALIAS", -10: "VC_ERR_SCRATCH",
}


class JointAttnError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = _lib().vc_status_string(status).decode() if _LIB is not None else STATUS.get(status, "?")
        super().__init__("%s failed: %s (%s)" % (where, STATUS.get(status, status), msg))


class vc_jointattn_desc(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("text_slot", ctypes.c_int32),
        ("frames", ctypes.c_int32),
        ("grid_h", ctypes.c_int32),
        ("grid_w", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float),
        ("deterministic", ctypes.c_int32),
    ]


_LIB = None
_P = ctypes.c_void_p
_DP = ctypes.POINTER(vc_jointattn_desc)
_SIGS = {
    "vc_jointattn_abi_version": (ctypes.c_int, []),
    "vc_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "vc_jointattn_tokens": (ctypes.c_int64, [_DP]),
    "vc_jointattn_fwd_workspace_bytes": (ctypes.c_size_t, [_DP]),
    "vc_jointattn_fwd": (ctypes.c_int, [_DP, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "vc_jointattn_fwd_noalloc": (ctypes.c_int, [_DP, _P, _P, _P, _P, _P, _P, _P, _P]),
    "vc_jointattn_bwd_workspace_bytes": (ctypes.c_size_t, [_DP]),
    "vc_jointattn_bwd": (ctypes.c_int, [_DP, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "vc_jointattn_bwd_prepare": (ctypes.c_int, [_DP, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "vc_jointattn_bwd_dkdv": (ctypes.c_int, [_DP, _P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "vc_jointattn_bwd_dq": (ctypes.c_int, [_DP, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "vc_jointattn_fused_dq_keys": (ctypes.c_int64, [_DP]),
    "vc_jointattn_bwd_fused": (ctypes.c_int, [_DP, _P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "vc_spatialattn_fwd": (ctypes.c_int, [_DP, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "vc_spatialattn_bwd_workspace_bytes": (ctypes.c_size_t, [_DP]),
    "vc_spatialattn_bwd": (ctypes.c_int, [_DP, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "vc_temporalattn_fwd": (ctypes.c_int, [_DP, _P, _P, _P, _P, _P, _P, _P]),
    "vc_temporalattn_fwd_sum": (ctypes.c_int, [_DP, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "vc_branchsum": (ctypes.c_int, [_DP, _P, _P, _P, _P, _P]),
    "vc_offload_create": (ctypes.c_int, [ctypes.POINTER(ctypes.c_void_p)]),
    "vc_offload_destroy": (ctypes.c_int, [ctypes.c_void_p]),
    "vc_offload_store": (ctypes.c_int, [ctypes.c_void_p, _P, _P, ctypes.c_size_t, _P]),
    "vc_offload_load": (ctypes.c_int, [ctypes.c_void_p, _P, _P, ctypes.c_size_t, _P]),
    "vc_offload_wait": (ctypes.c_int, [ctypes.c_void_p, _P]),
    "vc_temporalattn_bwd_workspace_bytes": (ctypes.c_size_t, [_DP]),
    "vc_temporalattn_bwd": (ctypes.c_int, [_DP, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
}


def library_path() -> str:
    return LIB_PATH


def _lib() -> ctypes.CDLL:
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libvc_jointattn.so is not built (%s); run __graft_entry__.build()" % LIB_PATH)
        lib = ctypes.CDLL(LIB_PATH)
        # The version first, through the one signature every version shares; nothing else is
        # bound unless it matches.
        ver = lib.vc_jointattn_abi_version
        ver.restype, ver.argtypes = ctypes.c_int, []
        got = ver()
        if got != ABI_VERSION:
            raise RuntimeError("%s implements C ABI version %d, this binding version %d; rebuild the library "
                               "(__graft_entry__.build())" % (LIB_PATH, got, ABI_VERSION))
        for name, (res, args) in _SIGS.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = lib
    return _LIB


def header_functions() -> list:
    """Names of the functions include/vc_jointattn.h declares."""
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\**\s+\**(vc_[a-z_0-9]+)\s*\(", text, re.M)))


def make_desc(batch, heads, head_dim, text_slot, frames, grid_h, grid_w, scale=None, deterministic=False):
    return vc_jointattn_desc(int(batch), int(heads), int(head_dim), int(text_slot), int(frames), int(grid_h),
                             int(grid_w), float(scale) if scale else 0.0, 1 if deterministic else 0)


def desc_for(workload, scale=None, deterministic=False):
    w = workload
    return make_desc(w.batch, w.heads, w.head_dim, w.text_slot, w.frames, w.grid_h, w.grid_w, scale, deterministic)


# --------------------------------------------------------------------------
# Raw entry points with the C names (pointers are ints or torch tensors).
# --------------------------------------------------------------------------

def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _call(name, *args):
    st = getattr(_lib(), name)(*args)
    if st != VC_OK:
        raise JointAttnError(st, name)


def vc_jointattn_abi_version() -> int:
    return _lib().vc_jointattn_abi_version()


def vc_status_string(status: int) -> str:
    return _lib().vc_status_string(status).decode()


def vc_jointattn_tokens(desc) -> int:
    return _lib().vc_jointattn_tokens(ctypes.byref(desc))


def vc_jointattn_fwd_workspace_bytes(desc) -> int:
    return _lib().vc_jointattn_fwd_workspace_bytes(ctypes.byref(desc))


def vc_jointattn_bwd_workspace_bytes(desc) -> int:
    return _lib().vc_jointattn_bwd_workspace_bytes(ctypes.byref(desc))


def vc_jointattn_fwd(desc, q, k, v, text_len, key_mask, o, lse, workspace, workspace_bytes, stream=None):
    _call("vc_jointattn_fwd", ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(text_len), _ptr(key_mask),
          _ptr(o), _ptr(lse), _ptr(workspace), int(workspace_bytes), _stream(stream))


def vc_jointattn_fwd_noalloc(desc, q, k, v, text_len, key_mask, o, lse, stream=None):
    _call("vc_jointattn_fwd_noalloc", ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(text_len),
          _ptr(key_mask), _ptr(o), _ptr(lse), _stream(stream))


def vc_jointattn_bwd(desc, q, k, v, o, lse, dout, text_len, key_mask, dq, dk, dv, workspace, workspace_bytes,
                     stream=None):
    _call("vc_jointattn_bwd", ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), _ptr(dout),
          _ptr(text_len), _ptr(key_mask), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(workspace), int(workspace_bytes),
          _stream(stream))


def vc_jointattn_bwd_prepare(desc, q, k, o, lse, dout, workspace, workspace_bytes, stream=None):
    _call("vc_jointattn_bwd_prepare", ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(o), _ptr(lse), _ptr(dout),
          _ptr(workspace), int(workspace_bytes), _stream(stream))


def vc_jointattn_bwd_dkdv(desc, q, k, v, dout, text_len, key_mask, dk, dv, workspace, workspace_bytes,
                          stream=None):
    _call("vc_jointattn_bwd_dkdv", ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(dout),
          _ptr(text_len), _ptr(key_mask), _ptr(dk), _ptr(dv), _ptr(workspace), int(workspace_bytes),
          _stream(stream))


def vc_jointattn_bwd_dq(desc, q, k, v, dout, text_len, key_mask, dq, workspace, workspace_bytes, stream=None):
    _call("vc_jointattn_bwd_dq", ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(dout),
          _ptr(text_len), _ptr(key_mask), _ptr(dq), _ptr(workspace), int(workspace_bytes), _stream(stream))


def vc_jointattn_fused_dq_keys(desc) -> int:
    return _lib().vc_jointattn_fused_dq_keys(ctypes.byref(desc))


def vc_jointattn_bwd_fused(desc, q, k, v, dout, text_len, key_mask, dk, dv, workspace, workspace_bytes,
                           stream=None):
    _call("vc_jointattn_bwd_fused", ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(dout),
          _ptr(text_len), _ptr(key_mask), _ptr(dk), _ptr(dv), _ptr(workspace), int(workspace_bytes),
          _stream(stream))


def vc_spatialattn_fwd(desc, q, k, v, text_len, key_mask, o, lse, workspace, workspace_bytes, stream=None):
    _call("vc_spatialattn_fwd", ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(text_len), _ptr(key_mask),
          _ptr(o), _ptr(lse), _ptr(workspace), int(workspace_bytes), _stream(stream))


def vc_spatialattn_bwd_workspace_bytes(desc) -> int:
    return _lib().vc_spatialattn_bwd_workspace_bytes(ctypes.byref(desc))


def vc_spatialattn_bwd(desc, q, k, v, o, lse, dout, text_len, key_mask, dq, dk, dv, workspace, workspace_bytes,
                       stream=None):
    _call("vc_spatialattn_bwd", ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), _ptr(dout),
          _ptr(text_len), _ptr(key_mask), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(workspace), int(workspace_bytes),
          _stream(stream))


def vc_temporalattn_fwd(desc, q, k, v, key_mask, o, lse, stream=None):
    _call("vc_temporalattn_fwd", ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(key_mask), _ptr(o), _ptr(lse),
          _stream(stream))


def vc_temporalattn_fwd_sum(desc, q, k, v, key_mask, o_joint, o_spatial, o, lse, out, stream=None):
    _call("vc_temporalattn_fwd_sum", ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(key_mask), _ptr(o_joint),
          _ptr(o_spatial), _ptr(o), _ptr(lse), _ptr(out), _stream(stream))


def vc_branchsum(desc, o_joint, o_spatial, o_temporal, out, stream=None):
    _call("vc_branchsum", ctypes.byref(desc), _ptr(o_joint), _ptr(o_spatial), _ptr(o_temporal), _ptr(out),
          _stream(stream))


def vc_temporalattn_bwd_workspace_bytes(desc) -> int:
    return _lib().vc_temporalattn_bwd_workspace_bytes(ctypes.byref(desc))


def vc_temporalattn_bwd(desc, q, k, v, o, lse, dout, key_mask, dq, dk, dv, workspace, workspace_bytes, stream=None):
    _call("vc_temporalattn_bwd", ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), _ptr(dout),
          _ptr(key_mask), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(workspace), int(workspace_bytes), _stream(stream))


# --------------------------------------------------------------------------
# Tensor-level helpers: allocate outputs with torch, then call the library.
# --------------------------------------------------------------------------

def _check_shape(name, t, shape, dtype):
    if t.dtype != dtype:
        raise ValueError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))


def _check_placed(name, t):
    if t.device.type != "cuda":
        raise ValueError("%s must be on a GPU" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)


def _check_tensor(name, t, shape, dtype):
    _check_shape(name, t, shape, dtype)
    _check_placed(name, t)


def _workspace(nbytes, device):
    import torch
    if nbytes == 0:
        raise ValueError("invalid descriptor")
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def fwd_workspace(desc, device):
    return _workspace(vc_jointattn_fwd_workspace_bytes(desc), device)


def workspace(desc, device):
    """Backward workspace for a descriptor."""
    return _workspace(vc_jointattn_bwd_workspace_bytes(desc), device)


def spatial_workspace(desc, device):
    """Backward workspace of the spatial branch for a descriptor."""
    return _workspace(vc_spatialattn_bwd_workspace_bytes(desc), device)


def _check_joint_inputs(desc, tensors, text_len=None, key_mask=None, lse=None):
    """Shapes, dtypes and layout of the tensors of one call against each other and the
    descriptor (the library reads and writes [B, N, H, D] as the descriptor says, so a
    descriptor larger than the tensors must never reach it). Shapes and dtypes are checked
    before placement. Returns (B, N, H, D)."""
    import torch
    q = tensors[0][1]
    if q.dim() != 4:
        raise ValueError("q must have shape [B, N, H, D], got %s" % (tuple(q.shape),))
    B, N, H, D = q.shape
    every = [(n, t, (B, N, H, D), torch.bfloat16) for n, t in tensors]
    if text_len is not None:
        every.append(("text_len", text_len, (B,), torch.int32))
    if key_mask is not None:
        every.append(("key_mask", key_mask, (B, N), torch.uint8))
    if lse is not None:
        every.append(("lse", lse, (B, H, N), torch.float32))
    for n, t, shape, dtype in every:
        _check_shape(n, t, shape, dtype)
    if (desc.batch, desc.heads, desc.head_dim) != (B, H, D):
        raise ValueError("descriptor gives B=%d, H=%d, D=%d, tensors have B=%d, H=%d, D=%d"
                         % (desc.batch, desc.heads, desc.head_dim, B, H, D))
    if vc_jointattn_tokens(desc) != N:
        raise ValueError("descriptor gives N=%d, tensors have N=%d" % (vc_jointattn_tokens(desc), N))
    for n, t, _, _ in every:
        _check_placed(n, t)
    return B, N, H, D


def fwd(q, k, v, desc, text_len=None, key_mask=None, out=None, lse=None, ws=None):
    """(o, lse) for bf16 q, k, v of shape [B, N, H, D]."""
    import torch
    B, N, H, D = _check_joint_inputs(desc, (("q", q), ("k", k), ("v", v)), text_len, key_mask)
    o = torch.empty_like(q) if out is None else out
    lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device) if lse is None else lse
    _check_joint_inputs(desc, (("q", q), ("o", o)), lse=lse)
    ws = fwd_workspace(desc, q.device) if ws is None else ws
    vc_jointattn_fwd(desc, q, k, v, text_len, key_mask, o, lse, ws, ws.numel())
    return o, lse


def bwd(q, k, v, o, lse, dout, desc, text_len=None, key_mask=None, ws=None, dq=None, dk=None, dv=None):
    """(dq, dk, dv) for bf16 tensors of shape [B, N, H, D]."""
    import torch
    _check_joint_inputs(desc, (("q", q), ("k", k), ("v", v), ("o", o), ("dout", dout)), text_len, key_mask, lse)
    ws = workspace(desc, q.device) if ws is None else ws
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(q) if dk is None else dk
    dv = torch.empty_like(q) if dv is None else dv
    _check_joint_inputs(desc, (("q", q), ("dq", dq), ("dk", dk), ("dv", dv)))
    vc_jointattn_bwd(desc, q, k, v, o, lse, dout, text_len, key_mask, dq, dk, dv, ws, ws.numel())
    return dq, dk, dv


def _check_branch_inputs(desc, tensors, key_mask=None):
    return _check_joint_inputs(desc, tensors, None, key_mask)


def spatial_fwd(q, k, v, desc, text_len=None, key_mask=None, out=None, lse=None, ws=None):
    """Spatial branch (o, lse) for bf16 q, k, v of shape [B, N, H, D] (joint layout)."""
    import torch
    B, N, H, D = _check_joint_inputs(desc, (("q", q), ("k", k), ("v", v)), text_len, key_mask)
    o = torch.empty_like(q) if out is None else out
    lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device) if lse is None else lse
    _check_joint_inputs(desc, (("q", q), ("o", o)), lse=lse)
    ws = fwd_workspace(desc, q.device) if ws is None else ws
    vc_spatialattn_fwd(desc, q, k, v, text_len, key_mask, o, lse, ws, ws.numel())
    return o, lse


def spatial_bwd(q, k, v, o, lse, dout, desc, text_len=None, key_mask=None, ws=None):
    """Spatial branch (dq, dk, dv)."""
    import torch
    _check_joint_inputs(desc, (("q", q), ("k", k), ("v", v), ("o", o), ("dout", dout)), text_len, key_mask, lse)
    ws = spatial_workspace(desc, q.device) if ws is None else ws
    dq, dk, dv = (torch.empty_like(q) for _ in range(3))
    vc_spatialattn_bwd(desc, q, k, v, o, lse, dout, text_len, key_mask, dq, dk, dv, ws, ws.numel())
    return dq, dk, dv


def temporal_fwd(q, k, v, desc, key_mask=None, out=None, lse=None):
    """Temporal branch (o, lse) for bf16 q, k, v of shape [B, N, H, D] (joint layout)."""
    import torch
    B, N, H, D = _check_branch_inputs(desc, (("q", q), ("k", k), ("v", v)), key_mask)
    o = torch.empty_like(q) if out is None else out
    lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device) if lse is None else lse
    _check_joint_inputs(desc, (("q", q), ("o", o)), lse=lse)
    vc_temporalattn_fwd(desc, q, k, v, key_mask, o, lse)
    return o, lse


def temporal_fwd_sum(q, k, v, desc, o_joint=None, o_spatial=None, key_mask=None, out=None):
    """Temporal branch (o, lse) and the block sum o_joint + o_spatial + o in one pass."""
    import torch
    B, N, H, D = _check_branch_inputs(desc, (("q", q), ("k", k), ("v", v)), key_mask)
    for name, t in (("o_joint", o_joint), ("o_spatial", o_spatial)):
        if t is not None:
            _check_tensor(name, t, (B, N, H, D), torch.bfloat16)
    o = torch.empty_like(q)
    lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
    out = torch.empty_like(q) if out is None else out
    _check_joint_inputs(desc, (("q", q), ("out", out)))
    vc_temporalattn_fwd_sum(desc, q, k, v, key_mask, o_joint, o_spatial, o, lse, out)
    return o, lse, out


def branch_sum(desc, o_joint=None, o_spatial=None, o_temporal=None, out=None):
    """Block output o_joint + o_spatial + o_temporal (bf16, summed in fp32, one rounding)."""
    import torch
    given = [(n, t) for n, t in (("o_joint", o_joint), ("o_spatial", o_spatial), ("o_temporal", o_temporal))
             if t is not None]
    if not given:
        raise ValueError("branch_sum needs at least one branch output")
    out = torch.empty_like(given[0][1]) if out is None else out
    _check_joint_inputs(desc, given + [("out", out)])
    vc_branchsum(desc, o_joint, o_spatial, o_temporal, out)
    return out


class Offload:
    """Activation offload engine (C ABI vc_offload_*): device <-> pinned host copies on a
    copy stream of its own, ordered after the caller's stream; `wait` makes the caller's
    stream wait for them."""

    def __init__(self):
        h = ctypes.c_void_p()
        _call("vc_offload_create", ctypes.byref(h))
        self._h = h

    @staticmethod
    def _bytes(a, b):
        n = a.numel() * a.element_size()
        if b.numel() * b.element_size() != n:
            raise ValueError("offload copy between tensors of different sizes")
        return n

    def store(self, host, dev, stream=None):
        """host (pinned CPU tensor) <- dev (GPU tensor), after the stream's queued work."""
        _call("vc_offload_store", self._h, _ptr(host), _ptr(dev), self._bytes(host, dev), _stream(stream))

    def load(self, dev, host, stream=None):
        """dev (GPU tensor) <- host (pinned CPU tensor), after the stream's queued work."""
        _call("vc_offload_load", self._h, _ptr(dev), _ptr(host), self._bytes(dev, host), _stream(stream))

    def wait(self, stream=None):
        _call("vc_offload_wait", self._h, _stream(stream))

    def close(self):
        if self._h is not None and self._h.value:
            _call("vc_offload_destroy", self._h)
        self._h = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def temporal_bwd(q, k, v, o, lse, dout, desc, key_mask=None, ws=None):
    """Temporal branch (dq, dk, dv)."""
    import torch
    _check_joint_inputs(desc, (("q", q), ("k", k), ("v", v), ("o", o), ("dout", dout)), None, key_mask, lse)
    dq, dk, dv = (torch.empty_like(q) for _ in range(3))
    # the library reads no workspace for this branch; one passed in is handed through unused
    vc_temporalattn_bwd(desc, q, k, v, o, lse, dout, key_mask, dq, dk, dv, ws, 0 if ws is None else ws.numel())
    return dq, dk, dv


_AUTOGRAD = {}


def _autograd_functions():
    """The autograd wrappers (made once, on first use, so that importing the package does
    not need torch)."""
    if _AUTOGRAD:
        return _AUTOGRAD
    import torch

    def branch_fwd(branch, q, k, v, desc, text_len, key_mask):
        if branch == "joint":
            return fwd(q, k, v, desc, text_len, key_mask)
        if branch == "spatial":
            return spatial_fwd(q, k, v, desc, text_len, key_mask)
        return temporal_fwd(q, k, v, desc, key_mask)  # no text keys in this branch

    def branch_bwd(branch, q, k, v, o, lse, do, desc, text_len, key_mask):
        if branch == "joint":
            return bwd(q, k, v, o, lse, do, desc, text_len, key_mask)
        if branch == "spatial":
            return spatial_bwd(q, k, v, o, lse, do, desc, text_len, key_mask)
        return temporal_bwd(q, k, v, o, lse, do, desc, key_mask)

    class BranchAttention(torch.autograd.Function):
        """One attention branch ("joint", "spatial" or "temporal"): forward returns O;
        LSE is kept for backward."""

        @staticmethod
        def forward(ctx, q, k, v, desc, branch, text_len=None, key_mask=None):
            o, lse = branch_fwd(branch, q, k, v, desc, text_len, key_mask)
            ctx.save_for_backward(q, k, v, o, lse)
            ctx.desc, ctx.branch, ctx.text_len, ctx.key_mask = desc, branch, text_len, key_mask
            return o

        @staticmethod
        def backward(ctx, do):
            q, k, v, o, lse = ctx.saved_tensors
            dq, dk, dv = branch_bwd(ctx.branch, q, k, v, o, lse, do.contiguous(), ctx.desc, ctx.text_len,
                                    ctx.key_mask)
            return dq, dk, dv, None, None, None, None

    class ParallelBlockAttention(torch.autograd.Function):
        """The three branches of the parallel block (Sec. III-B) on one set of q, k, v,
        summed: forward returns joint + spatial + temporal (the sum fused into the temporal
        forward); backward hands the same output gradient to every branch and adds their
        input gradients with the branch-sum kernel (fp32, one rounding)."""

        @staticmethod
        def forward(ctx, q, k, v, desc, text_len=None, key_mask=None):
            o_j, l_j = fwd(q, k, v, desc, text_len, key_mask)
            o_s, l_s = spatial_fwd(q, k, v, desc, text_len, key_mask)
            o_t, l_t, out = temporal_fwd_sum(q, k, v, desc, o_joint=o_j, o_spatial=o_s, key_mask=key_mask)
            ctx.save_for_backward(q, k, v, o_j, l_j, o_s, l_s, o_t, l_t)
            ctx.desc, ctx.text_len, ctx.key_mask = desc, text_len, key_mask
            return out

        @staticmethod
        def backward(ctx, do):
            q, k, v, o_j, l_j, o_s, l_s, o_t, l_t = ctx.saved_tensors
            do = do.contiguous()
            desc, tl, km = ctx.desc, ctx.text_len, ctx.key_mask
            gj = bwd(q, k, v, o_j, l_j, do, desc, tl, km)
            gs = spatial_bwd(q, k, v, o_s, l_s, do, desc, tl, km)
            gt = temporal_bwd(q, k, v, o_t, l_t, do, desc, km)
            grads = tuple(branch_sum(desc, gj[i], gs[i], gt[i], out=gj[i]) for i in range(3))
            return grads + (None, None, None)

    _AUTOGRAD.update(branch=BranchAttention, block=ParallelBlockAttention)
    return _AUTOGRAD


def joint_attention(q, k, v, desc, text_len=None, key_mask=None):
    """Differentiable joint attention (bf16 in, bf16 out)."""
    return _autograd_functions()["branch"].apply(q, k, v, desc, "joint", text_len, key_mask)


def spatial_attention(q, k, v, desc, text_len=None, key_mask=None):
    """Differentiable spatial-branch attention (bf16 in, bf16 out; text rows of O are 0)."""
    return _autograd_functions()["branch"].apply(q, k, v, desc, "spatial", text_len, key_mask)


def temporal_attention(q, k, v, desc, key_mask=None):
    """Differentiable temporal-branch attention (bf16 in, bf16 out; text rows of O are 0)."""
    return _autograd_functions()["branch"].apply(q, k, v, desc, "temporal", None, key_mask)


def parallel_block_attention(q, k, v, desc, text_len=None, key_mask=None):
    """Differentiable sum of the joint, spatial and temporal branches on shared q, k, v."""
    return _autograd_functions()["block"].apply(q, k, v, desc, text_len, key_mask)
