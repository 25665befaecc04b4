"""Pins for the block oracle (oracle/ref_block.py): the element-wise sum of the three
attention branches and the bf16 rounding of the summed output.

Independent checks: torch's float32 -> bfloat16 conversion and hand-made ties for the
rounding; the one-frame block, where the temporal branch reduces to each video query
attending to itself (O = v) and the spatial branch to the joint one on the video rows,
so the block output has a closed form in the joint oracle; central finite differences
of <dout, block output> against the block backward with shared inputs; and planted
mistakes that must fail.
"""
import numpy as np
import pytest
import torch

import oracle.ref_attention as ora
import oracle.ref_block as obl


def rnd(shape, seed):
    return np.random.Generator(np.random.PCG64(seed)).standard_normal(shape)


def shared(q, k, v):
    return {n: (q, k, v) for n in obl.BRANCHES}


def test_round_bf16_matches_torch_and_ties():
    rng = np.random.Generator(np.random.PCG64(3))
    x = (rng.standard_normal(50000) * np.exp(rng.uniform(-60, 60, 50000))).astype(np.float32).astype(np.float64)
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(obl.round_bf16(x), ref)
    # exact ties between neighbouring bf16 values (spacing 2^-7 on [1, 2)) go to the even one
    u = 2.0 ** -7
    ties = np.array([1 + u / 2, 1 + 3 * u / 2, -(1 + u / 2), 2 - u / 2, 0.75 + u / 4])
    np.testing.assert_array_equal(obl.round_bf16(ties), [1.0, 1 + 2 * u, -1.0, 2.0, 0.75])
    # just above a tie rounds up; fp64 detail beyond float32 precision is honoured
    assert obl.round_bf16(1 + u / 2 + 2.0 ** -40) == 1 + u
    special = np.array([0.0, -0.0, np.inf, -np.inf])
    np.testing.assert_array_equal(obl.round_bf16(special), special)
    assert np.isnan(obl.round_bf16(np.nan))


def test_branch_sum_missing_branches_are_zero():
    a, b, c = rnd((2, 5, 3), 1), rnd((2, 5, 3), 2), rnd((2, 5, 3), 3)
    np.testing.assert_array_equal(obl.branch_sum(a, None, None), a)
    np.testing.assert_array_equal(obl.branch_sum(None, b, c), b + c)
    np.testing.assert_allclose(obl.branch_sum(a, b, c), a + b + c, rtol=0, atol=1e-15)
    with pytest.raises(ValueError):
        obl.branch_sum()


def one_frame_case(seed=5):
    B, T, L, H, D = 2, 4, 9, 2, 8
    N = T + L
    q, k, v = (rnd((B, N, H, D), seed + i) for i in range(3))
    text_len = np.array([2, 4], dtype=np.int32)
    km = np.ones((B, N), dtype=np.uint8)
    km[1, T + 3] = 0
    return q, k, v, T, text_len, km


def closed_form_one_frame(q, k, v, T, text_len, km):
    """Block output with one frame, from the joint oracle and the definition of validity."""
    B, N, H, D = q.shape
    valid = ora.key_validity(B, N, T, text_len, km)
    o_joint, _ = ora.attention_forward(q, k, v, valid)
    out = o_joint.copy()
    out[:, T:] += o_joint[:, T:]                               # spatial = joint on video rows
    out[:, T:] += v[:, T:] * valid[:, T:, None, None]          # temporal: each video query sees itself
    return out


def test_one_frame_block_closed_form():
    q, k, v, T, text_len, km = one_frame_case()
    out, br = obl.block_forward(shared(q, k, v), T, 1, text_len, km)
    np.testing.assert_allclose(out, closed_form_one_frame(q, k, v, T, text_len, km), rtol=0, atol=1e-12)
    # temporal LSE of a valid video query is its own scaled score; -inf where it is masked
    B, N, H, D = q.shape
    s_self = np.einsum("bnhd,bnhd->bhn", q, k) / np.sqrt(D)
    lse_t = br["temporal"][1]
    np.testing.assert_allclose(lse_t[0, :, T:], s_self[0, :, T:], rtol=0, atol=1e-12)
    assert np.isneginf(lse_t[1, :, T + 3]).all()


def test_planted_dropped_branch_fails_closed_form():
    q, k, v, T, text_len, km = one_frame_case()
    _, br = obl.block_forward(shared(q, k, v), T, 1, text_len, km)
    wrong = obl.branch_sum(br["joint"][0], br["spatial"][0], None)
    assert np.abs(wrong - closed_form_one_frame(q, k, v, T, text_len, km)).max() > 1e-2


def test_block_backward_matches_finite_differences():
    B, T, F, L, H, D = 1, 2, 2, 3, 1, 3
    N = T + F * L
    q, k, v, dout = (rnd((B, N, H, D), 40 + i) for i in range(4))
    text_len = np.array([1], dtype=np.int32)

    def loss(q_, k_, v_):
        out, _ = obl.block_forward(shared(q_, k_, v_), T, F, text_len, threads=1)
        return float((out * dout).sum())

    g = obl.block_backward(shared(q, k, v), dout, T, F, text_len, threads=1)
    total = [sum(g[n][i] for n in obl.BRANCHES) for i in range(3)]
    h = 1e-6
    for which, x in enumerate((q, k, v)):
        num = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            xp, xm = x.copy(), x.copy()
            xp[idx] += h
            xm[idx] -= h
            args_p = [q, k, v]
            args_m = [q, k, v]
            args_p[which], args_m[which] = xp, xm
            num[idx] = (loss(*args_p) - loss(*args_m)) / (2 * h)
        np.testing.assert_allclose(total[which], num, rtol=1e-6, atol=1e-8)
    # a backward that split dout over the branches (or dropped one) would be a third off
    third = [sum(g[n][i] for n in obl.BRANCHES) / 3 for i in range(3)]
    assert np.abs(third[0] - total[0]).max() > 1e-3


def test_block_forward_returns_each_branch():
    B, T, F, L, H, D = 1, 3, 2, 4, 2, 4
    N = T + F * L
    ins = {n: tuple(rnd((B, N, H, D), 60 + 3 * j + i) for i in range(3)) for j, n in enumerate(obl.BRANCHES)}
    out, br = obl.block_forward(ins, T, F)
    np.testing.assert_allclose(out, br["joint"][0] + br["spatial"][0] + br["temporal"][0], rtol=0, atol=1e-15)
    # separate inputs: text rows of the sum are the joint output alone
    np.testing.assert_array_equal(out[:, :T], br["joint"][0][:, :T])
