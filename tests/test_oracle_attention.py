"""Pins of the oracle's window indexing, StereoRoPE and neighbourhood attention -- CPU only.

Every check compares the oracle with something fixed independently of its
code: a brute-force characterisation of the border-clamped window, dense
masked attention in numpy, plain full attention (torch CPU, float64), special
cases with closed forms, rotation invariants, torch autograd and finite
differences."""
import itertools

import numpy as np
import pytest
import torch

import oracle


def brute_window(i, L, k):
    """The k-long run of positions inside [0, L) whose centre lies nearest to i."""
    r = (k - 1) // 2
    best = min(range(0, L - k + 1), key=lambda s: abs(s + r - i))
    return set(range(best, best + k))


@pytest.mark.parametrize("L,k", [(1, 1), (5, 1), (7, 7), (10, 7), (16, 7), (9, 3), (64, 9), (8, 5), (13, 13),
                                 (6, 6), (24, 24)])
def test_axis_index_brute_force(L, k):
    starts, qlo, qhi = oracle.axis_index(L, k)
    for i in range(L):
        assert set(range(starts[i], starts[i] + k)) == brute_window(i, L, k)
    for j in range(L):
        qs = [i for i in range(L) if j in brute_window(i, L, k)]
        assert qs == list(range(qlo[j], qhi[j] + 1))


def test_axis_index_rejects_bad_windows():
    # even windows are accepted only when they span the whole axis
    for L, k in ((5, 2), (5, 7), (0, 1), (5, 0), (8, 6), (24, 22)):
        with pytest.raises(ValueError):
            oracle.axis_index(L, k)


def dense_na(q, k, v, window, scale):
    """Dense attention over all N tokens of a tile with an explicit neighbourhood mask."""
    B, h, Z, H, W, d = q.shape
    N = Z * H * W
    pos = list(itertools.product(range(Z), range(H), range(W)))
    wins = [(brute_window(z, Z, window[0]), brute_window(y, H, window[1]), brute_window(x, W, window[2]))
            for z, y, x in pos]
    mask = np.zeros((N, N), bool)
    for i, (wz, wy, wx) in enumerate(wins):
        for j, (z, y, x) in enumerate(pos):
            mask[i, j] = z in wz and y in wy and x in wx
    Q = q.reshape(B, h, N, d)
    K = k.reshape(B, h, N, d)
    V = v.reshape(B, h, N, d)
    S = scale * np.einsum("bhid,bhjd->bhij", Q, K)
    S = np.where(mask, S, -np.inf)
    m = S.max(-1, keepdims=True)
    P = np.exp(S - m)
    l = P.sum(-1, keepdims=True)
    O = (P / l) @ V
    lse = (m + np.log(l))[..., 0]
    return O.reshape(q.shape), lse.reshape(q.shape[:-1]), mask


def rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


@pytest.mark.parametrize("shape,window", [((1, 2, 3, 6, 7, 8), (3, 3, 5)),
                                          ((2, 1, 4, 5, 9, 4), (1, 5, 3)),
                                          ((1, 1, 5, 8, 8, 16), (5, 7, 7)),
                                          ((1, 2, 6, 4, 5, 8), (6, 1, 1)),    # column-wise: all levels, even
                                          ((1, 1, 10, 9, 9, 8), (9, 9, 9))])
def test_fwd_matches_dense_masked_attention(shape, window):
    q, k, v = (rand(shape, s) for s in (1, 2, 3))
    scale = 0.37
    o, lse = oracle.na3d_fwd(q, k, v, window, scale)
    O, L, mask = dense_na(q, k, v, window, scale)
    assert mask.sum(1).min() == mask.sum(1).max() == np.prod(window)
    np.testing.assert_allclose(o, O, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, L, rtol=0, atol=1e-12)


def test_column_window_is_attention_along_each_column():
    """Window (Z, 1, 1): every query attends to all Z levels of its own column --
    plain softmax attention per column (torch SDPA, float64), even Z included."""
    shape = (2, 2, 6, 3, 4, 8)
    q, k, v = (rand(shape, s) for s in (70, 71, 72))
    out, lse = oracle.na3d_fwd(q, k, v, (6, 1, 1), 0.4)
    t = lambda a: torch.from_numpy(np.moveaxis(a, 2, 4).copy())  # [B, h, H, W, Z, d]
    ref = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), scale=0.4).numpy()
    np.testing.assert_allclose(out, np.moveaxis(ref, 4, 2), rtol=0, atol=1e-12)
    S = np.einsum("bhyxid,bhyxjd->bhyxij", t(q).numpy(), t(k).numpy()) * 0.4
    m = S.max(-1)
    rl = m + np.log(np.exp(S - m[..., None]).sum(-1))
    np.testing.assert_allclose(lse, np.moveaxis(rl, 4, 2), rtol=0, atol=1e-12)


def test_full_window_is_plain_attention():
    shape = (2, 3, 3, 5, 7, 16)
    q, k, v = (rand(shape, s) for s in (4, 5, 6))
    scale = 0.25
    o, lse = oracle.na3d_fwd(q, k, v, (3, 5, 7), scale)
    B, h, Z, H, W, d = shape
    t = lambda a: torch.from_numpy(a.reshape(B, h, Z * H * W, d))
    ref = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), scale=scale)
    np.testing.assert_allclose(o.reshape(B, h, -1, d), ref.numpy(), rtol=0, atol=1e-12)
    S = torch.einsum("bhid,bhjd->bhij", t(q), t(k)) * scale
    np.testing.assert_allclose(lse.reshape(B, h, -1), torch.logsumexp(S, -1).numpy(), atol=1e-12)


def test_unit_window_returns_v():
    shape = (1, 2, 3, 4, 5, 8)
    q, k, v = (rand(shape, s) for s in (7, 8, 9))
    o, lse = oracle.na3d_fwd(q, k, v, (1, 1, 1), 0.5)
    assert np.array_equal(o, v)
    np.testing.assert_allclose(lse, 0.5 * np.sum(q * k, -1), rtol=1e-14, atol=1e-14)


def test_zero_query_averages_window():
    shape = (1, 1, 4, 9, 8, 4)
    k, v = rand(shape, 10), rand(shape, 11)
    q = np.zeros(shape)
    window = (3, 5, 3)
    o, lse = oracle.na3d_fwd(q, k, v, window, 1.0)
    K = np.prod(window)
    np.testing.assert_allclose(lse, np.log(K), rtol=0, atol=1e-14)
    _, _, mask = dense_na(q, k, v, window, 1.0)
    ref = (mask / K) @ v.reshape(-1, 4)
    np.testing.assert_allclose(o.reshape(-1, 4), ref, rtol=0, atol=1e-14)


def test_one_hot_probe_marks_window_membership():
    # Q = K = 0, V = one-hot over tokens: O_q = 1/K exactly where the token is in q's window.
    Z, H, W = 4, 9, 10
    N = Z * H * W
    window = (3, 7, 5)
    K = np.prod(window)
    q = np.zeros((1, 1, Z, H, W, N))
    v = np.eye(N).reshape(1, 1, Z, H, W, N)
    o, _ = oracle.na3d_fwd(q, q, v, window, 1.0)
    o = o.reshape(N, N)
    _, _, mask = dense_na(np.zeros((1, 1, Z, H, W, 1)), np.zeros((1, 1, Z, H, W, 1)),
                          np.zeros((1, 1, Z, H, W, 1)), window, 1.0)
    assert np.array_equal(o > 0, mask)
    np.testing.assert_allclose(o[mask], 1.0 / K, rtol=1e-15)


def test_border_queries_share_one_window():
    # Queries 0..r along an axis see the same window: with identical q they agree bit for bit.
    shape = (1, 1, 1, 12, 3, 8)
    k, v = rand(shape, 12), rand(shape, 13)
    q = np.broadcast_to(rand((8,), 14), shape).copy()
    o, _ = oracle.na3d_fwd(q, k, v, (1, 7, 3), 0.3)
    for y in range(1, 4):
        assert np.array_equal(o[0, 0, 0, y], o[0, 0, 0, 0])
    for y in range(9, 12):
        assert np.array_equal(o[0, 0, 0, y], o[0, 0, 0, 8])
    assert not np.array_equal(o[0, 0, 0, 4], o[0, 0, 0, 0])


def test_sampled_queries_match_full():
    shape = (2, 2, 3, 6, 6, 8)
    q, k, v = (rand(shape, s) for s in (15, 16, 17))
    o, lse = oracle.na3d_fwd(q, k, v, (3, 3, 5), 0.4)
    sel = np.array([0, 5, 77, 431, 200])
    os_, ls_ = oracle.na3d_fwd(q, k, v, (3, 3, 5), 0.4, sel=sel)
    assert np.array_equal(os_, o.reshape(-1, 8)[sel])
    assert np.array_equal(ls_, lse.reshape(-1)[sel])


# ----------------------------------------------------------------------------- RoPE


def coords_rand(B, H, W, seed, amp=60.0):
    return (np.random.default_rng(seed).uniform(-amp, amp, (B, H, W, 2))).astype(np.float32)


def test_rope_zero_coords_is_identity():
    x = rand((2, 2, 3, 4, 5, 16), 20)
    y = oracle.rope_apply(x, np.zeros((2, 4, 5, 2), np.float32))
    assert np.array_equal(x, y)


def test_rope_is_a_rotation():
    x = rand((2, 3, 2, 4, 5, 32), 21)
    c = coords_rand(2, 4, 5, 22)
    y = oracle.rope_apply(x, c)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-14)
    # pairwise norms are preserved too (rotation within each (2t, 2t+1) plane)
    np.testing.assert_allclose(np.hypot(y[..., 0::2], y[..., 1::2]), np.hypot(x[..., 0::2], x[..., 1::2]),
                               rtol=1e-13)
    back = oracle.rope_apply(y, c, transpose=True)
    np.testing.assert_allclose(back, x, rtol=0, atol=1e-13)


def test_rope_composes_additively():
    x = rand((1, 1, 1, 3, 4, 16), 23)
    r = np.random.default_rng(24)
    a = r.integers(-50, 50, (1, 3, 4, 2)).astype(np.float32)
    b = r.integers(-50, 50, (1, 3, 4, 2)).astype(np.float32)
    y1 = oracle.rope_apply(oracle.rope_apply(x, a), b)
    y2 = oracle.rope_apply(x, a + b)
    np.testing.assert_allclose(y1, y2, rtol=0, atol=1e-12)


def test_rope_logits_depend_only_on_relative_position():
    # <R(p_i) q, R(p_j) k> is unchanged when every coordinate moves by one offset.
    x = rand((1, 1, 1, 4, 4, 32), 25)
    k = rand((1, 1, 1, 4, 4, 32), 26)
    c = coords_rand(1, 4, 4, 27, amp=20.0).round().astype(np.float32)
    shift = np.array([13.0, -7.0], np.float32)
    def logits(cc):
        a = oracle.rope_apply(x, cc).reshape(16, 32)
        b = oracle.rope_apply(k, cc).reshape(16, 32)
        return a @ b.T
    np.testing.assert_allclose(logits(c + shift), logits(c), rtol=0, atol=1e-11)


def test_rope_axis_split_and_quarter_turn():
    # Reading: the first d/4 pairs follow x, the rest follow y; pair 0 turns by x itself.
    d = 16
    x = rand((1, 1, 1, 1, 1, d), 28)
    c = np.array([[[[np.pi / 2, 0.0]]]], np.float32)
    y = oracle.rope_apply(x, c)
    assert np.array_equal(y[..., d // 2:], x[..., d // 2:])   # y-pairs untouched at y = 0
    np.testing.assert_allclose(y[..., 0], -x[..., 1], atol=1e-7)
    np.testing.assert_allclose(y[..., 1], x[..., 0], atol=1e-7)
    c2 = np.array([[[[0.0, np.pi / 2]]]], np.float32)
    y2 = oracle.rope_apply(x, c2)
    assert np.array_equal(y2[..., :d // 2], x[..., :d // 2])
    np.testing.assert_allclose(y2[..., d // 2], -x[..., d // 2 + 1], atol=1e-7)


def test_fused_rope_equals_rotate_then_attend():
    shape = (2, 2, 3, 6, 7, 16)
    q, k, v = (rand(shape, s) for s in (30, 31, 32))
    c = coords_rand(2, 6, 7, 33)
    o1, l1 = oracle.na3d_fwd(q, k, v, (3, 3, 5), 0.25, coords=c)
    o2, l2 = oracle.na3d_fwd(oracle.rope_apply(q, c), oracle.rope_apply(k, c), v, (3, 3, 5), 0.25)
    np.testing.assert_allclose(o1, o2, rtol=0, atol=1e-12)
    np.testing.assert_allclose(l1, l2, rtol=0, atol=1e-12)


# ----------------------------------------------------------------------------- backward


def torch_dense_grads(q, k, v, dout, window, scale):
    _, _, mask = dense_na(q, k, v, window, scale)
    B, h, Z, H, W, d = q.shape
    N = Z * H * W
    t = [torch.tensor(a.reshape(B, h, N, d), requires_grad=True) for a in (q, k, v)]
    S = torch.einsum("bhid,bhjd->bhij", t[0], t[1]) * scale
    S = S.masked_fill(~torch.from_numpy(mask), float("-inf"))
    O = torch.softmax(S, -1) @ t[2]
    O.backward(torch.from_numpy(dout.reshape(B, h, N, d)))
    return [x.grad.numpy().reshape(q.shape) for x in t]


@pytest.mark.parametrize("shape,window", [((1, 2, 3, 5, 6, 8), (3, 3, 5)), ((2, 1, 4, 7, 7, 4), (3, 5, 5))])
def test_bwd_matches_torch_autograd(shape, window):
    q, k, v, g = (rand(shape, s) for s in (40, 41, 42, 43))
    scale = 0.3
    dq, dk, dv = oracle.na3d_bwd(q, k, v, g, window, scale)
    rq, rk, rv = torch_dense_grads(q, k, v, g, window, scale)
    np.testing.assert_allclose(dq, rq, rtol=0, atol=1e-11)
    np.testing.assert_allclose(dk, rk, rtol=0, atol=1e-11)
    np.testing.assert_allclose(dv, rv, rtol=0, atol=1e-11)


def test_bwd_with_rope_is_transposed_rotation_of_rotated_grads():
    shape = (1, 2, 3, 5, 6, 8)
    q, k, v, g = (rand(shape, s) for s in (44, 45, 46, 47))
    c = coords_rand(1, 5, 6, 48)
    window, scale = (3, 3, 5), 0.3
    dq, dk, dv = oracle.na3d_bwd(q, k, v, g, window, scale, coords=c)
    rq, rk, rv = torch_dense_grads(oracle.rope_apply(q, c), oracle.rope_apply(k, c), v, g, window, scale)
    np.testing.assert_allclose(dq, oracle.rope_apply(rq, c, transpose=True), atol=1e-11)
    np.testing.assert_allclose(dk, oracle.rope_apply(rk, c, transpose=True), atol=1e-11)
    np.testing.assert_allclose(dv, rv, atol=1e-11)


def test_bwd_central_differences():
    shape = (1, 1, 2, 5, 5, 4)
    q, k, v, g = (rand(shape, s) for s in (50, 51, 52, 53))
    c = coords_rand(1, 5, 5, 54)
    window, scale = (1, 3, 3), 0.7
    dq, dk, dv = oracle.na3d_bwd(q, k, v, g, window, scale, coords=c)
    h = 1e-6
    r = np.random.default_rng(55)
    for which, grad in ((0, dq), (1, dk), (2, dv)):
        for _ in range(3):
            e = r.standard_normal(shape)
            args_p = [q, k, v]
            args_m = [q, k, v]
            args_p = [a + h * e if i == which else a for i, a in enumerate(args_p)]
            args_m = [a - h * e if i == which else a for i, a in enumerate(args_m)]
            op, _ = oracle.na3d_fwd(*args_p, window, scale, coords=c)
            om, _ = oracle.na3d_fwd(*args_m, window, scale, coords=c)
            fd = np.sum(g * (op - om)) / (2 * h)
            an = np.sum(grad * e)
            assert abs(fd - an) <= 1e-7 * max(1.0, abs(an))


def test_bwd_sampled_rows_match_full():
    shape = (1, 2, 3, 5, 6, 8)
    q, k, v, g = (rand(shape, s) for s in (60, 61, 62, 63))
    c = coords_rand(1, 5, 6, 64)
    dq, dk, dv = oracle.na3d_bwd(q, k, v, g, (3, 3, 3), 0.3, coords=c)
    sq = np.array([3, 17, 100, 179])
    sk = np.array([0, 44, 150])
    a, b, cc = oracle.na3d_bwd(q, k, v, g, (3, 3, 3), 0.3, coords=c, selq=sq, selk=sk)
    np.testing.assert_allclose(a, dq.reshape(-1, 8)[sq], atol=1e-13)
    np.testing.assert_allclose(b, dk.reshape(-1, 8)[sk], atol=1e-13)
    np.testing.assert_allclose(cc, dv.reshape(-1, 8)[sk], atol=1e-13)
