"""Pins for the fp64 oracle, independent of the oracle's own formulas.

Each check comes from somewhere other than the oracle: a hand-derived worked
example, central finite differences of the forward, an independent library
implementation of the textbook special case (torch's scaled_dot_product_attention
in float64 with autograd), brute-force deletion of masked keys, and identities
that hold for exact attention (row sums, permutation symmetry, identical keys,
a single valid key, gradient sums, shift invariance, linearity and bounds).
"""
import json
import math
import os

import numpy as np
import pytest

import oracle.ref_attention as ora
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rnd(shape, seed, scale=1.0):
    rng = np.random.Generator(np.random.PCG64(seed))
    return scale * rng.standard_normal(shape)


def loss(q, k, v, do, valid, scale):
    o, _ = ora.attention_forward(q, k, v, valid, scale, threads=1)
    return float((o * do).sum())


# --------------------------------------------------------------------------
# Hand-derived worked example (exact closed forms, one padded text key).
# --------------------------------------------------------------------------

def test_worked_example_golden():
    with open(os.path.join(GOLDEN, "worked_example.json")) as f:
        g = json.load(f)
    n = len(g["q"])
    shp = (1, n, 1, 1)
    q, k, v, do = (np.array(g[x], dtype=np.float64).reshape(shp) for x in ("q", "k", "v", "do"))
    valid = ora.key_validity(1, n, g["text_slot"], text_len=np.array(g["text_len"]))
    assert valid.tolist() == [[True, False, True, True]]
    o, lse = ora.attention_forward(q, k, v, valid, g["scale"])
    dq, dk, dv = ora.attention_backward(q, k, v, do, valid, g["scale"])
    e = g["expected"]
    np.testing.assert_allclose(o.reshape(-1), e["o"], atol=1e-13)
    np.testing.assert_allclose(lse.reshape(-1), e["lse"], rtol=1e-14)
    np.testing.assert_allclose(dq.reshape(-1), e["dq"], atol=1e-13)
    np.testing.assert_allclose(dk.reshape(-1), e["dk"], atol=1e-13)
    np.testing.assert_allclose(dv.reshape(-1), e["dv"], atol=1e-14)
    # closed forms restated independently of the stored digits
    assert abs(lse.reshape(-1)[0] - math.log(6)) < 1e-14
    assert abs(dq.reshape(-1)[0] - ((2 / 3) * math.log(2) - 2 * math.log(3))) < 1e-13


# --------------------------------------------------------------------------
# P1: central finite differences of L = sum(dO * O).
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", [0, 1])
def test_finite_differences(seed):
    B, N, H, D, T = 2, 9, 2, 4, 3
    q, k, v, do = (rnd((B, N, H, D), seed * 10 + i) for i in range(4))
    text_len = np.array([1, 3])          # sample 0: two padded text keys
    km = np.ones((B, N), np.uint8)
    km[1, 5] = 0                          # one masked video key in sample 1
    valid = ora.key_validity(B, N, T, text_len, km)
    scale = 0.7
    dq, dk, dv = ora.attention_backward(q, k, v, do, valid, scale, threads=1)
    h = 1e-6
    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        num = np.zeros_like(x)
        it = np.nditer(x, flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            xp = x.copy(); xp[idx] += h
            xm = x.copy(); xm[idx] -= h
            args_p = dict(q=q, k=k, v=v); args_p[name] = xp
            args_m = dict(q=q, k=k, v=v); args_m[name] = xm
            num[idx] = (loss(args_p["q"], args_p["k"], args_p["v"], do, valid, scale)
                        - loss(args_m["q"], args_m["k"], args_m["v"], do, valid, scale)) / (2 * h)
        err = np.abs(num - g).max() / max(np.abs(g).max(), 1e-30)
        assert err < 1e-6, (name, err)
    # masked keys: exactly zero gradient
    assert np.all(dk[0, 1:3] == 0) and np.all(dv[0, 1:3] == 0)
    assert np.all(dk[1, 5] == 0) and np.all(dv[1, 5] == 0)


# --------------------------------------------------------------------------
# P10: torch's scaled_dot_product_attention (float64, CPU, autograd).
# --------------------------------------------------------------------------

@pytest.mark.parametrize("case", ["p1", "tiny"])
def test_against_torch_sdpa(case):
    torch = pytest.importorskip("torch")
    if case == "p1":
        B, N, H, D, T = 2, 12, 2, 4, 4
        q, k, v, do = (rnd((B, N, H, D), 40 + i) for i in range(4))
        text_len = np.array([2, 4])
    else:
        w = W.WORKLOADS[1]
        x = W.make_inputs(w)
        q, k, v, do = (x[n].astype(np.float64) for n in ("q", "k", "v", "do"))
        B, N, H, D = w.shape
        T = w.text_slot
        text_len = np.array([9])
    valid = ora.key_validity(B, N, T, text_len)
    scale = 1.0 / math.sqrt(D)
    o, lse = ora.attention_forward(q, k, v, valid, scale)
    dq, dk, dv = ora.attention_backward(q, k, v, do, valid, scale)

    tq, tk, tv = (torch.tensor(a.transpose(0, 2, 1, 3), dtype=torch.float64, requires_grad=True)
                  for a in (q, k, v))
    mask = torch.tensor(valid)[:, None, None, :]           # [B,1,1,N] broadcast over heads/queries
    to = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask, scale=scale)
    to.backward(torch.tensor(do.transpose(0, 2, 1, 3)))
    np.testing.assert_allclose(o, to.detach().numpy().transpose(0, 2, 1, 3), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dq, tq.grad.numpy().transpose(0, 2, 1, 3), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dk, tk.grad.numpy().transpose(0, 2, 1, 3), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dv, tv.grad.numpy().transpose(0, 2, 1, 3), rtol=1e-10, atol=1e-12)
    # LSE against torch.logsumexp over the masked scores
    s = torch.einsum("bhid,bhjd->bhij", tq.detach(), tk.detach()) * scale
    s = s.masked_fill(~mask, float("-inf"))
    np.testing.assert_allclose(lse, torch.logsumexp(s, dim=-1).numpy(), rtol=1e-12)


@pytest.mark.parametrize("head_dim", [4, 64, 128])
def test_default_scale_against_torch_sdpa_default(head_dim):
    """The oracle's default scale (scale=None) against torch SDPA's own default (no scale
    argument: 1/sqrt of the query's last dimension), so that a wrong default in the oracle
    cannot go unnoticed; the GPU parity tests run the library with its default scale
    (descriptor softmax_scale = 0) against this oracle default."""
    torch = pytest.importorskip("torch")
    B, N, H, D, T = 1, 10, 2, head_dim, 3
    q, k, v, do = (rnd((B, N, H, D), 90 + i) for i in range(4))
    valid = ora.key_validity(B, N, T, np.array([2]))
    o, lse = ora.attention_forward(q, k, v, valid, None, threads=1)
    dq, dk, dv = ora.attention_backward(q, k, v, do, valid, None, threads=1)
    tq, tk, tv = (torch.tensor(a.transpose(0, 2, 1, 3), dtype=torch.float64, requires_grad=True)
                  for a in (q, k, v))
    mask = torch.tensor(valid)[:, None, None, :]
    to = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask)
    to.backward(torch.tensor(do.transpose(0, 2, 1, 3)))
    np.testing.assert_allclose(o, to.detach().numpy().transpose(0, 2, 1, 3), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dq, tq.grad.numpy().transpose(0, 2, 1, 3), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dk, tk.grad.numpy().transpose(0, 2, 1, 3), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dv, tv.grad.numpy().transpose(0, 2, 1, 3), rtol=1e-10, atol=1e-12)
    # a different scale gives a different result, so the comparison above has power
    o2, _ = ora.attention_forward(q, k, v, valid, 1.1 / math.sqrt(D), threads=1)
    assert np.abs(o2 - o).max() > 1e-6


# --------------------------------------------------------------------------
# Invariants of exact attention.
# --------------------------------------------------------------------------

def _case(seed=3, B=1, N=14, H=2, D=6, T=4):
    q, k, v, do = (rnd((B, N, H, D), seed * 7 + i) for i in range(4))
    return q, k, v, do, B, N, H, D, T


def test_rows_sum_to_one_and_masked_exactly_zero():
    q, k, v, do, B, N, H, D, T = _case()
    valid = ora.key_validity(B, N, T, np.array([2]))
    p = ora.head_probabilities(q, k, valid[0], 0.5, 0, 1)
    assert np.abs(p.sum(axis=1) - 1).max() < 1e-12
    assert np.all(p[:, ~valid[0]] == 0)
    assert np.all(p[:, valid[0]] > 0)


def test_key_permutation_invariance_and_query_equivariance():
    q, k, v, do, B, N, H, D, T = _case(seed=4)
    valid = ora.key_validity(B, N, T, np.array([3]))
    o, lse = ora.attention_forward(q, k, v, valid, 0.4)
    dq, dk, dv = ora.attention_backward(q, k, v, do, valid, 0.4)
    perm = np.random.Generator(np.random.PCG64(9)).permutation(N)
    # joint permutation of keys, values and validity: but queries are tokens too,
    # so permute only the key side by building separate query and key arrays.
    kp, vp, validp = k[:, perm], v[:, perm], valid[:, perm]
    o2, lse2 = _fwd_split(q, kp, vp, validp, 0.4)
    np.testing.assert_allclose(o2, o, atol=1e-12)
    np.testing.assert_allclose(lse2, lse, atol=1e-12)
    # query permutation (whole token order): outputs permute along with it
    qp, dop = q[:, perm], do[:, perm]
    o3, lse3 = ora.attention_forward(qp, kp, vp, validp, 0.4)
    dq3, dk3, dv3 = ora.attention_backward(qp, kp, vp, dop, validp, 0.4)
    np.testing.assert_allclose(o3, o[:, perm], atol=1e-12)
    np.testing.assert_allclose(lse3, lse[:, :, perm], atol=1e-12)
    np.testing.assert_allclose(dq3, dq[:, perm], atol=1e-12)
    np.testing.assert_allclose(dk3, dk[:, perm], atol=1e-12)
    np.testing.assert_allclose(dv3, dv[:, perm], atol=1e-12)


def _fwd_split(q, k, v, valid, scale):
    """Forward with queries and keys as separate sequences, by brute force per row."""
    B, N, H, D = q.shape
    o = np.zeros_like(q)
    lse = np.zeros((B, H, N))
    for b in range(B):
        for h in range(H):
            for i in range(N):
                s = np.array([scale * q[b, i, h] @ k[b, j, h] for j in range(k.shape[1]) if valid[b, j]])
                vv = np.array([v[b, j, h] for j in range(k.shape[1]) if valid[b, j]])
                m = s.max()
                w = np.exp(s - m)
                lse[b, h, i] = m + math.log(w.sum())
                o[b, i, h] = (w[:, None] * vv).sum(0) / w.sum()
    return o, lse


def test_identical_keys_give_mean_of_values():
    q, k, v, do, B, N, H, D, T = _case(seed=5)
    text_len = np.array([1])
    valid = ora.key_validity(B, N, T, text_len)
    kk = np.broadcast_to(rnd((1, 1, H, D), 77), k.shape).copy()
    o, lse = ora.attention_forward(q, kk, v, valid, 0.9)
    dq, dk, dv = ora.attention_backward(q, kk, v, do, valid, 0.9)
    nval = valid[0].sum()
    for h in range(H):
        mean_v = v[0, valid[0], h].mean(axis=0)
        np.testing.assert_allclose(o[0, :, h], np.broadcast_to(mean_v, (N, D)), atol=1e-12)
        expect_lse = 0.9 * (q[0, :, h] @ kk[0, 0, h]) + math.log(nval)
        np.testing.assert_allclose(lse[0, h], expect_lse, atol=1e-12)
    assert np.abs(dq).max() < 1e-12


def test_masked_keys_equal_deleting_them():
    q, k, v, do, B, N, H, D, T = _case(seed=6)
    km = np.ones((B, N), np.uint8)
    km[0, [2, 7, 11]] = 0
    valid = ora.key_validity(B, N, T, np.array([3]), km)
    o, lse = ora.attention_forward(q, k, v, valid, 0.6)
    dq, dk, dv = ora.attention_backward(q, k, v, do, valid, 0.6)
    # random values at masked keys change nothing
    k2, v2 = k.copy(), v.copy()
    bad = ~valid[0]
    k2[0, bad] = rnd(k2[0, bad].shape, 99, 50.0)
    v2[0, bad] = rnd(v2[0, bad].shape, 98, 50.0)
    o2, lse2 = ora.attention_forward(q, k2, v2, valid, 0.6)
    dq2, dk2, dv2 = ora.attention_backward(q, k2, v2, do, valid, 0.6)
    assert np.array_equal(o2, o) and np.array_equal(lse2, lse) and np.array_equal(dq2, dq)
    assert np.all(dk[0, bad] == 0) and np.all(dv[0, bad] == 0)
    # deleting the masked keys from the key side (queries unchanged), by brute force
    keep = valid[0]
    o3, lse3 = _fwd_split(q, k[:, keep], v[:, keep], np.ones((1, keep.sum()), bool), 0.6)
    np.testing.assert_allclose(o3, o, atol=1e-12)
    np.testing.assert_allclose(lse3, lse, atol=1e-12)


def test_single_valid_key():
    q, k, v, do, B, N, H, D, T = _case(seed=7)
    km = np.zeros((B, N), np.uint8)
    km[0, 9] = 1
    valid = ora.key_validity(B, N, T, None, km)
    o, lse = ora.attention_forward(q, k, v, valid, 0.3)
    dq, dk, dv = ora.attention_backward(q, k, v, do, valid, 0.3)
    for h in range(H):
        np.testing.assert_allclose(o[0, :, h], np.broadcast_to(v[0, 9, h], (N, D)), atol=1e-14)
        np.testing.assert_allclose(lse[0, h], 0.3 * q[0, :, h] @ k[0, 9, h], atol=1e-13)
        np.testing.assert_allclose(dv[0, 9, h], do[0, :, h].sum(0), atol=1e-12)
    assert np.abs(dq).max() < 1e-13 and np.abs(dk).max() < 1e-13
    assert np.all(dv[0, np.arange(N) != 9] == 0)


def test_no_valid_key_rows():
    q, k, v, do, B, N, H, D, T = _case(seed=8)
    km = np.zeros((B, N), np.uint8)
    valid = ora.key_validity(B, N, T, None, km)
    o, lse = ora.attention_forward(q, k, v, valid, 0.3)
    dq, dk, dv = ora.attention_backward(q, k, v, do, valid, 0.3)
    assert np.all(o == 0) and np.all(np.isneginf(lse))
    assert np.all(dq == 0) and np.all(dk == 0) and np.all(dv == 0)


def test_gradient_sums_and_D_identity():
    q, k, v, do, B, N, H, D, T = _case(seed=9, B=2)
    valid = ora.key_validity(B, N, T, np.array([4, 1]))
    o, lse = ora.attention_forward(q, k, v, valid, 0.5)
    dq, dk, dv = ora.attention_backward(q, k, v, do, valid, 0.5)
    # sum_j dS_ij = 0 for every i  =>  sum_j dK_j = 0 ; sum_j dV_j = sum_i dO_i
    np.testing.assert_allclose(dk.sum(axis=1), 0, atol=1e-12)
    np.testing.assert_allclose(dv.sum(axis=1), do.sum(axis=1), atol=1e-12)
    # D_i = sum_j P_ij dP_ij equals <dO_i, O_i>
    for b in range(B):
        for h in range(H):
            p = ora.head_probabilities(q, k, valid[b], 0.5, b, h)
            dp = do[b, :, h] @ v[b, :, h].T
            np.testing.assert_allclose((p * dp).sum(1), (do[b, :, h] * o[b, :, h]).sum(1), atol=1e-12)


def test_shift_of_keys():
    q, k, v, do, B, N, H, D, T = _case(seed=10)
    valid = ora.key_validity(B, N, T, np.array([2]))
    o, lse = ora.attention_forward(q, k, v, valid, 1.0)
    u = rnd((1, 1, H, D), 55, 30.0)          # large shift: logits of order 100s
    o2, lse2 = ora.attention_forward(q, k + u, v, valid, 1.0)
    np.testing.assert_allclose(o2, o, atol=1e-10)
    for h in range(H):
        np.testing.assert_allclose(lse2[0, h], lse[0, h] + q[0, :, h] @ u[0, 0, h], rtol=1e-12, atol=1e-9)


def test_linearity_and_bounds_in_values():
    q, k, v, do, B, N, H, D, T = _case(seed=11)
    valid = ora.key_validity(B, N, T, np.array([4]))
    v2 = rnd(v.shape, 321)
    o1, _ = ora.attention_forward(q, k, v, valid, 0.8)
    o2, _ = ora.attention_forward(q, k, v2, valid, 0.8)
    o3, _ = ora.attention_forward(q, k, 2.0 * v - 3.0 * v2, valid, 0.8)
    np.testing.assert_allclose(o3, 2.0 * o1 - 3.0 * o2, atol=1e-12)
    lo = v[0, valid[0]].min(axis=0)
    hi = v[0, valid[0]].max(axis=0)
    assert np.all(o1[0] >= lo - 1e-12) and np.all(o1[0] <= hi + 1e-12)


def test_ragged_batch_equals_independent_runs():
    B, H, D, T, F, Hp, Wp = 3, 2, 8, 6, 2, 2, 3
    N = T + F * Hp * Wp
    q, k, v, do = (rnd((B, N, H, D), 60 + i) for i in range(4))
    text_len = np.array([6, 2, 0])
    valid = ora.key_validity(B, N, T, text_len)
    o, lse = ora.attention_forward(q, k, v, valid, 0.5)
    dq, dk, dv = ora.attention_backward(q, k, v, do, valid, 0.5)
    for b in range(B):
        tl = text_len[b]
        keep = np.r_[np.arange(tl), np.arange(T, N)]
        sl = lambda x: x[b:b + 1, keep]  # noqa: E731 - sample b on its valid tokens only
        one = np.ones((1, len(keep)), bool)
        ob, lb = ora.attention_forward(sl(q), sl(k), sl(v), one, 0.5)
        dqb, dkb, dvb = ora.attention_backward(sl(q), sl(k), sl(v), sl(do), one, 0.5)
        np.testing.assert_allclose(ob, o[b:b + 1, keep], atol=1e-12)
        np.testing.assert_allclose(lb, lse[b:b + 1][:, :, keep], atol=1e-12)
        # dQ of a row depends only on that row's probabilities and dO: it matches.
        np.testing.assert_allclose(dqb, dq[b:b + 1, keep], atol=1e-12)
        # padded text rows are still queries of the joint run, and their dO feeds
        # dK, dV of the valid keys; equality there needs dO = 0 on padded rows
        # (next test), except for the sample without padding.
        if tl == T:
            np.testing.assert_allclose(dkb, dk[b:b + 1, keep], atol=1e-12)
            np.testing.assert_allclose(dvb, dv[b:b + 1, keep], atol=1e-12)


def test_ragged_batch_zero_padded_dO():
    """With dO = 0 on padded query rows, a sample equals its run without padding."""
    B, H, D, T = 2, 2, 8, 5
    N = T + 12
    q, k, v, do = (rnd((B, N, H, D), 80 + i) for i in range(4))
    text_len = np.array([2, 4])
    for b in range(B):
        do[b, text_len[b]:T] = 0.0
    valid = ora.key_validity(B, N, T, text_len)
    dq, dk, dv = ora.attention_backward(q, k, v, do, valid, 0.5)
    for b in range(B):
        keep = np.r_[np.arange(text_len[b]), np.arange(T, N)]
        sl = lambda x: x[b:b + 1, keep]  # noqa: E731
        one = np.ones((1, len(keep)), bool)
        dqb, dkb, dvb = ora.attention_backward(sl(q), sl(k), sl(v), sl(do), one, 0.5)
        np.testing.assert_allclose(dqb, dq[b:b + 1, keep], atol=1e-12)
        np.testing.assert_allclose(dkb, dk[b:b + 1, keep], atol=1e-12)
        np.testing.assert_allclose(dvb, dv[b:b + 1, keep], atol=1e-12)


# --------------------------------------------------------------------------
# Sampled evaluation equals the whole-tensor evaluation.
# --------------------------------------------------------------------------

def test_sampled_rows_and_cols_match_full():
    B, N, H, D, T = 2, 70, 3, 16, 10
    q, k, v, do = (rnd((B, N, H, D), 90 + i) for i in range(4))
    text_len = np.array([4, 10])
    valid = ora.key_validity(B, N, T, text_len)
    o, lse = ora.attention_forward(q, k, v, valid, 0.25)
    dq, dk, dv = ora.attention_backward(q, k, v, do, valid, 0.25)
    rows = np.array([0, 3, 9, 10, 33, 69])
    for b in range(B):
        for h in range(H):
            orow, lrow = ora.forward_rows(q, k, v, valid[b], 0.25, b, h, rows)
            np.testing.assert_allclose(orow, o[b, rows, h], atol=1e-13)
            np.testing.assert_allclose(lrow, lse[b, h, rows], atol=1e-13)
            np.testing.assert_allclose(ora.backward_rows(q, k, v, do, valid[b], 0.25, b, h, rows),
                                       dq[b, rows, h], atol=1e-13)
            dkc, dvc = ora.backward_cols(q, k, v, do, valid[b], 0.25, b, h, rows)
            np.testing.assert_allclose(dkc, dk[b, rows, h], atol=1e-12)
            np.testing.assert_allclose(dvc, dv[b, rows, h], atol=1e-12)
    # a partition of the rows into blocks reproduces the whole backward
    parts = [np.arange(0, 30), np.arange(30, 70)]
    acc_dk = np.zeros((N, D)); acc_dv = np.zeros((N, D))
    for rows_p in parts:
        ob, lb, dqb, dkp, dvp = ora.rowblock_fwd_bwd(q, k, v, do, valid[1], 0.25, 1, 2, rows_p)
        np.testing.assert_allclose(ob, o[1, rows_p, 2], atol=1e-13)
        np.testing.assert_allclose(dqb, dq[1, rows_p, 2], atol=1e-13)
        acc_dk += dkp; acc_dv += dvp
    np.testing.assert_allclose(acc_dk, dk[1, :, 2], atol=1e-12)
    np.testing.assert_allclose(acc_dv, dv[1, :, 2], atol=1e-12)


def test_threaded_equals_serial():
    B, N, H, D, T = 1, 300, 4, 8, 20
    q, k, v, do = (rnd((B, N, H, D), 120 + i) for i in range(4))
    valid = ora.key_validity(B, N, T, np.array([7]))
    a = ora.attention_backward(q, k, v, do, valid, 0.3, threads=1)
    b = ora.attention_backward(q, k, v, do, valid, 0.3, threads=4)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


# --------------------------------------------------------------------------
# The pins are sensitive: plausible mistakes planted in the oracle fail them.
# --------------------------------------------------------------------------

def _golden_ok():
    try:
        test_worked_example_golden()
        test_finite_differences(0)
        test_gradient_sums_and_D_identity()
        test_identical_keys_give_mean_of_values()
        return True
    except AssertionError:
        return False


@pytest.mark.parametrize("mutant", ["drop_D", "sign_dS", "transpose_dk", "no_mask", "scale_dq", "lse_base2"])
def test_planted_mistakes_are_caught(monkeypatch, mutant):
    real_scores = ora._scores
    real_probs = ora._probs
    real_back = ora._head_backward
    real_lse = ora._row_lse
    if mutant == "no_mask":
        monkeypatch.setattr(ora, "_scores", lambda q, k, valid, scale: scale * (q @ k.T))
    elif mutant == "lse_base2":
        monkeypatch.setattr(ora, "_row_lse", lambda s: real_lse(s) / math.log(2))
    else:
        def bad_back(q, k, v, do, valid, scale, lse, threads=1):
            n = q.shape[0]
            s = real_scores(q, k, valid, scale)
            p = real_probs(s, lse)
            dp = do @ v.T
            d_i = (p * dp).sum(axis=1)
            if mutant == "drop_D":
                ds = p * dp
            elif mutant == "sign_dS":
                ds = p * (d_i[:, None] - dp)
            else:
                ds = p * (dp - d_i[:, None])
            dq = (1.0 if mutant == "scale_dq" else scale) * (ds @ k)
            dk = scale * (ds @ q if mutant == "transpose_dk" else ds.T @ q)
            dv = p.T @ do
            return dq, dk, dv
        monkeypatch.setattr(ora, "_head_backward", bad_back)
    assert not _golden_ok(), mutant
    monkeypatch.setattr(ora, "_scores", real_scores)
    monkeypatch.setattr(ora, "_head_backward", real_back)
    monkeypatch.setattr(ora, "_row_lse", real_lse)
    assert _golden_ok()
