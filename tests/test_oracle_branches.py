"""Pins for the spatial and temporal branch oracles (oracle/ref_branches.py).

Each check is independent of the branch functions' own arithmetic: torch's
scaled_dot_product_attention in float64 with an explicit dense [queries, keys]
boolean mask built from the branch definition (forward and autograd
backward), central finite differences, the one-frame case that reduces the
spatial branch to the (separately pinned) joint oracle, locality and
symmetry properties that follow from the regrouping, gradient-sum identities,
and planted mistakes that must fail.
"""
import numpy as np
import pytest
import torch

import oracle.ref_attention as ora
import oracle.ref_branches as orb


def rnd(shape, seed, scale=1.0):
    rng = np.random.Generator(np.random.PCG64(seed))
    return scale * rng.standard_normal(shape)


def case(B=2, T=5, F=3, L=7, H=2, D=8, seed=0):
    N = T + F * L
    q, k, v, do = (rnd((B, N, H, D), seed + i) for i in range(4))
    return q, k, v, do, N


def token_info(N, T, F):
    """For each token: is it video, its frame, its spatial position."""
    L = (N - T) // F
    idx = np.arange(N)
    video = idx >= T
    frame = np.where(video, (idx - T) // L, -1)
    pos = np.where(video, (idx - T) % L, -1)
    return video, frame, pos


def dense_mask(kind, N, T, F, valid_b):
    """[N, N] boolean: may query i attend to key j, from the branch definition."""
    video, frame, pos = token_info(N, T, F)
    if kind == "spatial":
        m = video[:, None] & valid_b[None, :] & (~video[None, :] | (frame[:, None] == frame[None, :]))
    else:
        m = video[:, None] & video[None, :] & valid_b[None, :] & (pos[:, None] == pos[None, :])
    return m


def sdpa_reference(kind, q, k, v, do, T, F, valid, scale):
    """Dense masked attention with torch (float64, autograd) over the video query rows."""
    B, N, H, D = q.shape
    video, _, _ = token_info(N, T, F)
    o = np.zeros_like(q)
    grads = [np.zeros_like(q) for _ in range(3)]
    for b in range(B):
        m = torch.from_numpy(dense_mask(kind, N, T, F, valid[b])[video])
        for h in range(H):
            qt = torch.tensor(q[b, video, h], requires_grad=True)
            kt = torch.tensor(k[b, :, h], requires_grad=True)
            vt = torch.tensor(v[b, :, h], requires_grad=True)
            out = torch.nn.functional.scaled_dot_product_attention(qt[None], kt[None], vt[None], attn_mask=m[None],
                                                                   scale=scale)[0]
            out.backward(torch.tensor(do[b, video, h]))
            o[b, video, h] = out.detach().numpy()
            grads[0][b, video, h] = qt.grad.numpy()
            grads[1][b, :, h] = kt.grad.numpy()
            grads[2][b, :, h] = vt.grad.numpy()
    return o, grads


@pytest.mark.parametrize("kind", ["spatial", "temporal"])
def test_branch_matches_dense_masked_sdpa(kind):
    B, T, F, L, H, D = 2, 5, 3, 7, 2, 8
    q, k, v, do, N = case(B, T, F, L, H, D, seed=10)
    text_len = np.array([3, 5], dtype=np.int32)
    km = np.ones((B, N), dtype=np.uint8)
    km[0, T + 2] = 0  # one masked video key
    scale = 0.37
    if kind == "spatial":
        valid = ora.key_validity(B, N, T, text_len, km)
        o, lse = orb.spatial_forward(q, k, v, T, F, text_len, km, scale, threads=1)
        g = orb.spatial_backward(q, k, v, do, T, F, text_len, km, scale, threads=1)
    else:
        valid = ora.key_validity(B, N, T, None, km)
        o, lse = orb.temporal_forward(q, k, v, T, F, km, scale, threads=1)
        g = orb.temporal_backward(q, k, v, do, T, F, km, scale, threads=1)
    o_ref, g_ref = sdpa_reference(kind, q, k, v, do, T, F, valid, scale)
    np.testing.assert_allclose(o, o_ref, atol=1e-12)
    for a, r in zip(g, g_ref):
        np.testing.assert_allclose(a, r, atol=1e-12)
    # text rows: no output, no key, no query gradient
    assert np.all(o[:, :T] == 0) and np.all(np.isneginf(lse[:, :, :T])) and np.all(g[0][:, :T] == 0)
    # LSE against torch's logsumexp of the masked scores
    for b in range(B):
        m = torch.from_numpy(dense_mask(kind, N, T, F, valid[b]))
        for h in range(H):
            s = scale * torch.from_numpy(q[b, :, h]) @ torch.from_numpy(k[b, :, h]).T
            s = s.masked_fill(~m, float("-inf"))
            ref = torch.logsumexp(s[T:], dim=1).numpy()
            np.testing.assert_allclose(lse[b, h, T:], ref, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("kind", ["spatial", "temporal"])
def test_branch_finite_differences(kind):
    B, T, F, L, H, D = 1, 2, 3, 2, 1, 3
    q, k, v, do, N = case(B, T, F, L, H, D, seed=20)
    text_len = np.array([1], dtype=np.int32)
    c = 0.8

    def fwd(q_, k_, v_):
        if kind == "spatial":
            return orb.spatial_forward(q_, k_, v_, T, F, text_len, None, c, threads=1)[0]
        return orb.temporal_forward(q_, k_, v_, T, F, None, c, threads=1)[0]

    def lossf(q_, k_, v_):
        return float((fwd(q_, k_, v_) * do).sum())

    if kind == "spatial":
        g = orb.spatial_backward(q, k, v, do, T, F, text_len, None, c, threads=1)
    else:
        g = orb.temporal_backward(q, k, v, do, T, F, None, c, threads=1)
    h = 1e-6
    for which, grad in zip(range(3), g):
        num = np.zeros_like(q)
        for idx in np.ndindex(q.shape):
            args = [q.copy(), k.copy(), v.copy()]
            args[which][idx] += h
            lp = lossf(*args)
            args[which][idx] -= 2 * h
            lm = lossf(*args)
            num[idx] = (lp - lm) / (2 * h)
        np.testing.assert_allclose(grad, num, rtol=1e-6, atol=1e-8)


def test_spatial_one_frame_reduces_to_joint():
    B, T, F, L, H, D = 2, 6, 1, 11, 2, 8
    q, k, v, do, N = case(B, T, F, L, H, D, seed=30)
    text_len = np.array([6, 2], dtype=np.int32)
    valid = ora.key_validity(B, N, T, text_len)
    o, lse = orb.spatial_forward(q, k, v, T, F, text_len, threads=1)
    oj, lj = ora.attention_forward(q, k, v, valid, threads=1)
    np.testing.assert_allclose(o[:, T:], oj[:, T:], atol=1e-13)
    np.testing.assert_allclose(lse[:, :, T:], lj[:, :, T:], atol=1e-13)
    # with no upstream gradient on text rows the joint gradients coincide everywhere
    do_v = do.copy()
    do_v[:, :T] = 0.0
    g = orb.spatial_backward(q, k, v, do_v, T, F, text_len, threads=1)
    gj = ora.attention_backward(q, k, v, do_v, valid, threads=1)
    np.testing.assert_allclose(g[0][:, T:], gj[0][:, T:], atol=1e-12)
    np.testing.assert_allclose(g[1], gj[1], atol=1e-12)
    np.testing.assert_allclose(g[2], gj[2], atol=1e-12)


def test_spatial_frames_are_independent():
    B, T, F, L, H, D = 1, 4, 3, 5, 1, 6
    q, k, v, do, N = case(B, T, F, L, H, D, seed=40)
    o, _ = orb.spatial_forward(q, k, v, T, F, threads=1)
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    other = slice(T + 2 * L, T + 3 * L)  # perturb frame 2 only
    for x in (q2, k2, v2):
        x[:, other] += 3.0
    o2, _ = orb.spatial_forward(q2, k2, v2, T, F, threads=1)
    np.testing.assert_array_equal(o[:, T:T + 2 * L], o2[:, T:T + 2 * L])
    # perturbing the text keys changes every frame
    k3 = k.copy()
    k3[:, :T] += 1.0
    o3, _ = orb.spatial_forward(q, k3, v, T, F, threads=1)
    for f in range(F):
        assert not np.allclose(o[:, T + f * L:T + (f + 1) * L], o3[:, T + f * L:T + (f + 1) * L])


def test_temporal_equivariant_under_position_permutation():
    B, T, F, L, H, D = 1, 3, 4, 6, 2, 5
    q, k, v, do, N = case(B, T, F, L, H, D, seed=50)
    perm = np.random.Generator(np.random.PCG64(7)).permutation(L)
    tok = np.concatenate([np.arange(T)] + [T + f * L + perm for f in range(F)])
    o, lse = orb.temporal_forward(q, k, v, T, F, threads=1)
    op, lp = orb.temporal_forward(q[:, tok], k[:, tok], v[:, tok], T, F, threads=1)
    np.testing.assert_allclose(op, o[:, tok], atol=1e-13)
    np.testing.assert_allclose(lp, lse[:, :, tok], atol=1e-13)
    # text tokens play no part at all
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    for x in (q2, k2, v2):
        x[:, :T] = 9.0
    o2, _ = orb.temporal_forward(q2, k2, v2, T, F, threads=1)
    np.testing.assert_array_equal(o2, o)


@pytest.mark.parametrize("kind", ["spatial", "temporal"])
def test_branch_gradient_sums(kind):
    B, T, F, L, H, D = 2, 4, 3, 6, 2, 5
    q, k, v, do, N = case(B, T, F, L, H, D, seed=60)
    if kind == "spatial":
        dq, dk, dv = orb.spatial_backward(q, k, v, do, T, F, np.array([4, 1]), threads=1)
    else:
        dq, dk, dv = orb.temporal_backward(q, k, v, do, T, F, threads=1)
    # every video query's probabilities sum to 1; dS rows sum to 0
    np.testing.assert_allclose(dv.sum(axis=1), do[:, T:].sum(axis=1), atol=1e-12)
    np.testing.assert_allclose(dk.sum(axis=1), 0.0, atol=1e-12)


def test_planted_mistakes_fail(monkeypatch):
    B, T, F, L, H, D = 1, 3, 2, 4, 1, 4
    q, k, v, do, N = case(B, T, F, L, H, D, seed=70)
    valid = ora.key_validity(B, N, T)
    o_ref, _ = sdpa_reference("spatial", q, k, v, do, T, F, valid, 0.5)
    # dropped text keys
    monkeypatch.setattr(orb, "_frame_keys", lambda T_, L_, f: np.arange(T_ + f * L_, T_ + (f + 1) * L_))
    o_bad, _ = orb.spatial_forward(q, k, v, T, F, scale=0.5, threads=1)
    assert not np.allclose(o_bad, o_ref, atol=1e-6)
    monkeypatch.undo()
    # temporal sequence taken along the wrong axis (consecutive tokens instead of frames)
    t_ref, _ = sdpa_reference("temporal", q, k, v, do, T, F, valid, 0.5)
    monkeypatch.setattr(orb, "_temporal_tokens", lambda T_, F_, L_, l: T_ + l * F_ + np.arange(F_))
    t_bad, _ = orb.temporal_forward(q, k, v, T, F, scale=0.5, threads=1)
    assert not np.allclose(t_bad, t_ref, atol=1e-6)
