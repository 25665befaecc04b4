"""Oracle for joint text-video attention: plain, slow, exact, fp64, CPU.

TEST INFRASTRUCTURE ONLY. Nothing on the product path imports this module:
only the test suite, the smoke check and the benchmark's CPU-baseline leg
may call it. It shares no code with the HIP kernels.

What it computes (Vchitect-2.0, Sec. III-B "Parallel Transformer
Architecture" and the method-overview figure caption; Sec. V-A "Features of
Video Training", paragraph "3D and multi-modal nature"): the full-sequence
branch of the multimodal diffusion block attends across the concatenation of
text tokens and spatio-temporal video tokens. Every token of the joint
sequence is a query and every valid token is a key. The paper writes no
formula, so this is standard scaled dot-product softmax attention, evaluated
exactly (two passes: maximum first, then exponentials), per (sample, head):

    s_ij  = c * <q_i, k_j>                      for valid keys j
    LSE_i = log sum_j exp(s_ij)                 (natural log, scale included)
    P_ij  = exp(s_ij - LSE_i), 0 for invalid j
    O_i   = sum_j P_ij v_j

and its analytic gradient for an upstream gradient dO:

    dV_j  = sum_i P_ij dO_i
    dP_ij = <dO_i, v_j>
    D_i   = sum_j P_ij dP_ij
    dS_ij = P_ij (dP_ij - D_i)
    dQ_i  = c sum_j dS_ij k_j
    dK_j  = c sum_i dS_ij q_i

Readings of points the paper leaves open (each is listed in the design notes):
  * the joint sequence is [text slot of T tokens | video tokens, frame-major];
    text appears once; the order does not change any result because the
    operation is equivariant in queries and invariant under a joint
    permutation of keys and values;
  * padded text keys (position j in [text_len_b, T)) and keys with
    key_mask == 0 are invalid: their probability is exactly zero, so their
    values have no effect and their dK, dV are exactly zero;
  * padded text *queries* are ordinary queries;
  * a query with no valid key gets O = 0, LSE = -inf, dQ = 0;
  * c defaults to 1/sqrt(head_dim); no positional term, causal mask or
    dropout inside the operation.

Layouts follow the library boundary: q, k, v, o, do, dq, dk, dv are
[B, N, H, D]; lse is [B, H, N]. All arithmetic is float64.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

try:  # keep BLAS single-threaded inside the worker threads
    from threadpoolctl import threadpool_limits
except Exception:  # pragma: no cover - threadpoolctl is optional
    threadpool_limits = None

__all__ = [
    "key_validity",
    "default_scale",
    "attention_forward",
    "attention_backward",
    "head_probabilities",
    "forward_rows",
    "backward_rows",
    "backward_cols",
    "rowblock_fwd_bwd",
    "host_threads",
]


def host_threads() -> int:
    """Number of host cores this process may run on."""
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def default_scale(head_dim: int) -> float:
    """Softmax scale c = 1/sqrt(D) (the paper states none; standard choice)."""
    return 1.0 / math.sqrt(head_dim)


def key_validity(batch: int, n_tokens: int, text_slot: int, text_len=None, key_mask=None) -> np.ndarray:
    """Boolean [B, N]: is token j of sample b a valid key.

    Text tokens occupy positions [0, text_slot); sample b uses the first
    clamp(text_len[b], 0, text_slot) of them (captions vary in length,
    Sec. IV "Video Captioning"); the rest of the slot is padding. Video
    tokens are always valid unless key_mask clears them.
    """
    valid = np.ones((batch, n_tokens), dtype=bool)
    if text_len is not None:
        tl = np.asarray(text_len).reshape(-1)
        assert tl.shape[0] == batch
        for b in range(batch):
            used = int(min(max(int(tl[b]), 0), text_slot))
            valid[b, used:text_slot] = False
    if key_mask is not None:
        km = np.asarray(key_mask).reshape(batch, n_tokens)
        valid &= km != 0
    return valid


# ---------------------------------------------------------------------------
# Per (sample, head) building blocks.  q, k, v, do: [N, D] float64.
# ---------------------------------------------------------------------------

def _scores(q_rows: np.ndarray, k: np.ndarray, valid: np.ndarray, scale: float) -> np.ndarray:
    """s_ij = c <q_i, k_j>, and -inf where key j is invalid."""
    s = scale * (q_rows @ k.T)
    s[:, ~valid] = -np.inf
    return s


def _row_lse(s: np.ndarray) -> np.ndarray:
    """Exact log-sum-exp of each row, max subtracted first (pass 1 then pass 2)."""
    m = s.max(axis=1)
    lse = np.full(s.shape[0], -np.inf)
    live = np.isfinite(m)
    if live.any():
        e = np.exp(s[live] - m[live, None])
        lse[live] = m[live] + np.log(e.sum(axis=1))
    return lse


def _probs(s: np.ndarray, lse: np.ndarray) -> np.ndarray:
    """P_ij = exp(s_ij - LSE_i); rows without a valid key are all zero."""
    p = np.zeros_like(s)
    live = np.isfinite(lse)
    if live.any():
        p[live] = np.exp(s[live] - lse[live, None])
    return p


def _block_rows(n_rows: int, n_keys: int) -> int:
    """Query rows per block, so that one [rows, keys] fp64 array stays near 128 MiB."""
    return int(max(16, min(1024, (16 << 20) // max(n_keys, 1))))


def _pool_map(fn, items, threads):
    if threads <= 1 or len(items) <= 1:
        return [fn(it) for it in items]
    with ThreadPoolExecutor(max_workers=threads) as ex:
        return list(ex.map(fn, items))


class _BlasOne:
    def __enter__(self):
        self._ctx = threadpool_limits(limits=1) if threadpool_limits is not None else None
        if self._ctx is not None:
            self._ctx.__enter__()
        return self

    def __exit__(self, *a):
        if self._ctx is not None:
            self._ctx.__exit__(*a)


def _head_forward(q, k, v, valid, scale, rows=None, threads=1):
    """O and LSE for the given query rows (all rows if None) of one head."""
    n = q.shape[0]
    rows = np.arange(n) if rows is None else np.asarray(rows)
    step = _block_rows(len(rows), k.shape[0])
    blocks = [rows[i:i + step] for i in range(0, len(rows), step)]

    def one(blk):
        s = _scores(q[blk], k, valid, scale)
        lse = _row_lse(s)
        p = _probs(s, lse)
        return p @ v, lse

    outs = _pool_map(one, blocks, threads)
    o = np.concatenate([a for a, _ in outs], axis=0) if outs else np.zeros((0, v.shape[1]))
    lse = np.concatenate([b for _, b in outs]) if outs else np.zeros(0)
    return o, lse


def _head_backward(q, k, v, do, valid, scale, lse, threads=1):
    """dQ, dK, dV of one head, recomputing P from the exact fp64 LSE."""
    n = q.shape[0]
    step = _block_rows(n, k.shape[0])
    starts = list(range(0, n, step))

    def one(i0):
        blk = slice(i0, min(n, i0 + step))
        s = _scores(q[blk], k, valid, scale)
        p = _probs(s, lse[blk])
        dp = do[blk] @ v.T
        d_i = (p * dp).sum(axis=1)
        ds = p * (dp - d_i[:, None])
        dq = scale * (ds @ k)
        dk = scale * (ds.T @ q[blk])
        dv = p.T @ do[blk]
        return dq, dk, dv

    outs = _pool_map(one, starts, threads)
    dq = np.concatenate([a for a, _, _ in outs], axis=0)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for _, pk, pv in outs:  # fixed block order: deterministic sum
        dk += pk
        dv += pv
    return dq, dk, dv


# ---------------------------------------------------------------------------
# Whole-tensor entry points, [B, N, H, D] layout.
# ---------------------------------------------------------------------------

def _as64(x):
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def attention_forward(q, k, v, valid, scale=None, threads=None):
    """Exact forward. Returns (o [B,N,H,D], lse [B,H,N]) in float64."""
    q, k, v = _as64(q), _as64(k), _as64(v)
    B, N, H, D = q.shape
    scale = default_scale(D) if scale is None else float(scale)
    threads = host_threads() if threads is None else threads
    o = np.zeros_like(q)
    lse = np.zeros((B, H, N))
    items = [(b, h) for b in range(B) for h in range(H)]

    def one(bh):
        b, h = bh
        return _head_forward(q[b, :, h], k[b, :, h], v[b, :, h], valid[b], scale)

    with _BlasOne():
        outs = _pool_map(one, items, threads)
    for (b, h), (oh, lh) in zip(items, outs):
        o[b, :, h] = oh
        lse[b, h] = lh
    return o, lse


def attention_backward(q, k, v, do, valid, scale=None, lse=None, threads=None):
    """Exact backward. Returns (dq, dk, dv), each [B,N,H,D] float64."""
    q, k, v, do = _as64(q), _as64(k), _as64(v), _as64(do)
    B, N, H, D = q.shape
    scale = default_scale(D) if scale is None else float(scale)
    threads = host_threads() if threads is None else threads
    if lse is None:
        _, lse = attention_forward(q, k, v, valid, scale, threads)
    dq, dk, dv = (np.zeros_like(q) for _ in range(3))
    items = [(b, h) for b in range(B) for h in range(H)]

    def one(bh):
        b, h = bh
        return _head_backward(q[b, :, h], k[b, :, h], v[b, :, h], do[b, :, h], valid[b], scale, lse[b, h])

    with _BlasOne():
        outs = _pool_map(one, items, threads)
    for (b, h), (a, bk, c) in zip(items, outs):
        dq[b, :, h] = a
        dk[b, :, h] = bk
        dv[b, :, h] = c
    return dq, dk, dv


def head_probabilities(q, k, valid_b, scale, b, h):
    """The full probability matrix P of one (sample, head): [N, N] float64 (small N only)."""
    q, k = _as64(q), _as64(k)
    s = _scores(q[b, :, h], k[b, :, h], valid_b, scale)
    return _probs(s, _row_lse(s))


# ---------------------------------------------------------------------------
# Sampled evaluation for sizes where the whole result is too costly on a CPU:
# the same definition, evaluated for chosen rows (queries) or columns (keys).
# ---------------------------------------------------------------------------

def forward_rows(q, k, v, valid_b, scale, b, h, rows, threads=None):
    """O[b, rows, h] and LSE[b, h, rows], exact."""
    threads = host_threads() if threads is None else threads
    with _BlasOne():
        return _head_forward(_as64(q[b, :, h]), _as64(k[b, :, h]), _as64(v[b, :, h]),
                             valid_b, scale, rows=rows, threads=threads)


def backward_rows(q, k, v, do, valid_b, scale, b, h, rows, threads=None):
    """dQ[b, rows, h], exact (only the rows' own probabilities are needed)."""
    threads = host_threads() if threads is None else threads
    rows = np.asarray(rows)
    qh, kh, vh, doh = (_as64(x[b, :, h]) for x in (q, k, v, do))
    with _BlasOne():
        step = _block_rows(len(rows), kh.shape[0])
        blocks = [rows[i:i + step] for i in range(0, len(rows), step)]

        def one(blk):
            s = _scores(qh[blk], kh, valid_b, scale)
            p = _probs(s, _row_lse(s))
            dp = doh[blk] @ vh.T
            d_i = (p * dp).sum(axis=1)
            ds = p * (dp - d_i[:, None])
            return scale * (ds @ kh)

        return np.concatenate(_pool_map(one, blocks, threads), axis=0)


def backward_cols(q, k, v, do, valid_b, scale, b, h, cols, threads=None):
    """dK[b, cols, h] and dV[b, cols, h], exact.

    Needs LSE_i and D_i of every query i, so it first runs the full forward of
    the head (O and LSE), then D_i = <dO_i, O_i> (equal to sum_j P_ij dP_ij),
    then sums over all query rows for the chosen key columns only.
    """
    threads = host_threads() if threads is None else threads
    cols = np.asarray(cols)
    qh, kh, vh, doh = (_as64(x[b, :, h]) for x in (q, k, v, do))
    with _BlasOne():
        o, lse = _head_forward(qh, kh, vh, valid_b, scale, threads=threads)
        d_all = (doh * o).sum(axis=1)
        n = qh.shape[0]
        kc, vc, validc = kh[cols], vh[cols], valid_b[cols]
        step = _block_rows(n, max(len(cols), 1024))
        starts = list(range(0, n, step))

        def one(i0):
            blk = slice(i0, min(n, i0 + step))
            s = _scores(qh[blk], kc, validc, scale)
            p = _probs(s, lse[blk])
            dp = doh[blk] @ vc.T
            ds = p * (dp - d_all[blk, None])
            return scale * (ds.T @ qh[blk]), p.T @ doh[blk]

        outs = _pool_map(one, starts, threads)
    dk = np.zeros((len(cols), kh.shape[1]))
    dv = np.zeros((len(cols), vh.shape[1]))
    for a, c in outs:
        dk += a
        dv += c
    return dk, dv


def rowblock_fwd_bwd(q, k, v, do, valid_b, scale, b, h, rows, threads=None):
    """Forward and backward restricted to a block of query rows of one head.

    Returns (o_rows, lse_rows, dq_rows, dk_part, dv_part): the rows' outputs,
    their dQ, and the dK, dV contributions of exactly these rows (the full
    dK, dV is the sum of such parts over a partition of the rows). Used to
    time the oracle on a bounded share of a large workload.
    """
    threads = host_threads() if threads is None else threads
    rows = np.asarray(rows)
    qh, kh, vh, doh = (_as64(x[b, :, h]) for x in (q, k, v, do))
    with _BlasOne():
        step = _block_rows(len(rows), kh.shape[0])
        blocks = [rows[i:i + step] for i in range(0, len(rows), step)]

        def one(blk):
            s = _scores(qh[blk], kh, valid_b, scale)
            lse = _row_lse(s)
            p = _probs(s, lse)
            o = p @ vh
            dp = doh[blk] @ vh.T
            d_i = (p * dp).sum(axis=1)
            ds = p * (dp - d_i[:, None])
            return o, lse, scale * (ds @ kh), scale * (ds.T @ qh[blk]), p.T @ doh[blk]

        outs = _pool_map(one, blocks, threads)
    o = np.concatenate([x[0] for x in outs])
    lse = np.concatenate([x[1] for x in outs])
    dq = np.concatenate([x[2] for x in outs])
    dk = np.zeros_like(kh)
    dv = np.zeros_like(vh)
    for x in outs:
        dk += x[3]
        dv += x[4]
    return o, lse, dq, dk, dv
