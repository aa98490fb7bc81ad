"""Pins of the oracle's QK RMSNorm and sigmoid output gate (App. B.5) -- CPU only.

Each check rests on something other than the oracle's own formulas: the plain
attention of the oracle (pinned in test_oracle_attention.py) on inputs whose
normalised form is known exactly, scale invariance, the logit bound that the
norm guarantees, closed-form sigmoid values, Euler's relation for functions
invariant under scaling, and central differences of the forward."""
import math

import numpy as np
import pytest

import oracle


def rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def coords_rand(B, H, W, seed, amp=60.0):
    return (np.random.default_rng(seed).uniform(-amp, amp, (B, H, W, 2))).astype(np.float32)


def signs(shape, seed, mag=1.0):
    """Entries +-mag with random signs: every row has mean square mag^2 exactly."""
    return mag * np.where(np.random.default_rng(seed).random(shape) < 0.5, -1.0, 1.0)


SHAPE, WINDOW = (1, 2, 3, 5, 6, 8), (3, 3, 5)


# ----------------------------------------------------------------------------- QK RMSNorm


def test_unit_rms_rows_are_left_unchanged():
    # rows of +-1 have mean square 1: with eps = 0 the norm is the identity
    q, k = signs(SHAPE, 1), signs(SHAPE, 2)
    v = rand(SHAPE, 3)
    c = coords_rand(1, 5, 6, 4)
    o0, l0 = oracle.na3d_fwd(q, k, v, WINDOW, 0.3, coords=c)
    o1, l1 = oracle.na3d_fwd(q, k, v, WINDOW, 0.3, coords=c, qk_norm=True, eps=0.0)
    np.testing.assert_allclose(o1, o0, rtol=0, atol=1e-13)
    np.testing.assert_allclose(l1, l0, rtol=0, atol=1e-13)


def test_eps_sits_under_the_root_of_the_mean_square():
    # rows of +-2 (mean square 4) with eps = 5: the norm divides by sqrt(4 + 5) = 3
    q, k = signs(SHAPE, 5, 2.0), signs(SHAPE, 6, 2.0)
    v = rand(SHAPE, 7)
    o0, l0 = oracle.na3d_fwd(q / 3.0, k / 3.0, v, WINDOW, 0.3)
    o1, l1 = oracle.na3d_fwd(q, k, v, WINDOW, 0.3, qk_norm=True, eps=5.0)
    np.testing.assert_allclose(o1, o0, rtol=0, atol=1e-13)
    np.testing.assert_allclose(l1, l0, rtol=0, atol=1e-13)


def test_norm_is_invariant_to_per_token_scaling():
    q, k, v = rand(SHAPE, 8), rand(SHAPE, 9), rand(SHAPE, 10)
    r = np.random.default_rng(11)
    cq = r.uniform(0.05, 20.0, SHAPE[:-1] + (1,))
    ck = r.uniform(0.05, 20.0, SHAPE[:-1] + (1,))
    c = coords_rand(1, 5, 6, 12)
    o0, l0 = oracle.na3d_fwd(q, k, v, WINDOW, 0.3, coords=c, qk_norm=True, eps=0.0)
    o1, l1 = oracle.na3d_fwd(q * cq, k * ck, v, WINDOW, 0.3, coords=c, qk_norm=True, eps=0.0)
    np.testing.assert_allclose(o1, o0, rtol=0, atol=1e-12)
    np.testing.assert_allclose(l1, l0, rtol=0, atol=1e-12)


def test_norm_bounds_the_logits():
    # |<q^, k^>| <= |q^| |k^| < d, so every logit lies within scale * d of 0 and
    # the lse within scale * d of ln(window size), however large the inputs are
    d, scale = SHAPE[-1], 0.3
    q, k, v = 300.0 * rand(SHAPE, 13), 300.0 * rand(SHAPE, 14), rand(SHAPE, 15)
    _, lse = oracle.na3d_fwd(q, k, v, WINDOW, scale, qk_norm=True, eps=1e-6)
    n = WINDOW[0] * WINDOW[1] * WINDOW[2]
    assert np.all(np.abs(lse - math.log(n)) <= scale * d)
    _, lse_raw = oracle.na3d_fwd(q, k, v, WINDOW, scale)
    assert np.max(np.abs(lse_raw - math.log(n))) > 100 * scale * d  # the bound is the norm's doing


def test_norm_commutes_with_the_rotation():
    # rotating first (the pinned rotary embedding) and normalising afterwards
    # gives what the oracle computes, which normalises before rotating
    q, k, v = rand(SHAPE, 16), rand(SHAPE, 17), rand(SHAPE, 18)
    c = coords_rand(1, 5, 6, 19)
    o0, l0 = oracle.na3d_fwd(oracle.rope_apply(q, c), oracle.rope_apply(k, c), v, WINDOW, 0.3,
                             qk_norm=True, eps=1e-3)
    o1, l1 = oracle.na3d_fwd(q, k, v, WINDOW, 0.3, coords=c, qk_norm=True, eps=1e-3)
    np.testing.assert_allclose(o1, o0, rtol=0, atol=1e-12)
    np.testing.assert_allclose(l1, l0, rtol=0, atol=1e-12)


# ----------------------------------------------------------------------------- gate


@pytest.mark.parametrize("g,factor", [(0.0, 0.5), (math.log(3.0), 0.75), (-math.log(3.0), 0.25),
                                      (40.0, 1.0), (-800.0, 0.0)])
def test_headwise_gate_closed_forms(g, factor):
    q, k, v = rand(SHAPE, 20), rand(SHAPE, 21), rand(SHAPE, 22)
    a, la = oracle.na3d_fwd(q, k, v, WINDOW, 0.3)
    o, lo = oracle.na3d_fwd(q, k, v, WINDOW, 0.3, gate=np.full(SHAPE[:-1], g))
    np.testing.assert_allclose(o, factor * a, rtol=1e-15, atol=0)
    np.testing.assert_array_equal(lo, la)  # the lse is the softmax's, before the gate


def test_channel_gate_closed_forms_follow_the_channel():
    # channel e of every token gets logit {0, ln 3, -ln 3}[(e + token) % 3]:
    # sigmoid 1/2, 3/4, 1/4; a transposed or shifted index changes the factor
    q, k, v = rand(SHAPE, 23), rand(SHAPE, 24), rand(SHAPE, 25)
    d = SHAPE[-1]
    logits = np.array([0.0, math.log(3.0), -math.log(3.0)])
    factors = np.array([0.5, 0.75, 0.25])
    tok = np.arange(np.prod(SHAPE[:-1])).reshape(SHAPE[:-1] + (1,))
    sel = (np.arange(d) + tok) % 3
    a, _ = oracle.na3d_fwd(q, k, v, WINDOW, 0.3)
    o, _ = oracle.na3d_fwd(q, k, v, WINDOW, 0.3, gate=logits[sel])
    np.testing.assert_allclose(o, factors[sel] * a, rtol=1e-15, atol=0)


def test_channel_gate_with_equal_logits_is_the_headwise_gate():
    q, k, v = rand(SHAPE, 26), rand(SHAPE, 27), rand(SHAPE, 28)
    g = rand(SHAPE[:-1], 29)
    o1, _ = oracle.na3d_fwd(q, k, v, WINDOW, 0.3, gate=g)
    o2, _ = oracle.na3d_fwd(q, k, v, WINDOW, 0.3, gate=np.repeat(g[..., None], SHAPE[-1], -1))
    np.testing.assert_array_equal(o1, o2)


def test_gate_shape_is_checked():
    q = rand(SHAPE, 30)
    with pytest.raises(ValueError):
        oracle.na3d_fwd(q, q, q, WINDOW, 0.3, gate=np.zeros(SHAPE[:-1] + (3,)))


# ----------------------------------------------------------------------------- backward


BWD_SHAPE, BWD_WINDOW = (1, 2, 2, 5, 5, 4), (1, 3, 3)


@pytest.mark.parametrize("qk_norm,gate_dim", [(True, 0), (False, 1), (False, 4), (True, 1), (True, 4)])
def test_bwd_central_differences(qk_norm, gate_dim):
    shape = BWD_SHAPE
    q, k, v, dout = (rand(shape, s) for s in (40, 41, 42, 43))
    c = coords_rand(1, 5, 5, 44)
    gate = None if gate_dim == 0 else rand(shape if gate_dim == 4 else shape[:-1], 45)
    kw = dict(coords=c, qk_norm=qk_norm, eps=1e-2, gate=gate)
    grads = oracle.na3d_bwd(q, k, v, dout, BWD_WINDOW, 0.7, **kw)
    h = 1e-6
    r = np.random.default_rng(46)
    args = [q, k, v] + ([gate] if gate is not None else [])
    for which, grad in enumerate(grads):
        for _ in range(3):
            e = r.standard_normal(args[which].shape)
            ap = [a + h * e if i == which else a for i, a in enumerate(args)]
            am = [a - h * e if i == which else a for i, a in enumerate(args)]
            kp, km = dict(kw), dict(kw)
            if gate is not None:
                kp["gate"], km["gate"] = ap[3], am[3]
            op, _ = oracle.na3d_fwd(*ap[:3], BWD_WINDOW, 0.7, **kp)
            om, _ = oracle.na3d_fwd(*am[:3], BWD_WINDOW, 0.7, **km)
            fd = np.sum(dout * (op - om)) / (2 * h)
            an = np.sum(grad * e)
            assert abs(fd - an) <= 1e-7 * max(1.0, abs(an)), (which, fd, an)


def test_normalised_gradients_are_orthogonal_to_their_inputs():
    # with eps = 0 the output does not change when one q or k row is scaled, so
    # (Euler) the gradient of every row is orthogonal to that row
    q, k, v, dout = (rand(SHAPE, s) for s in (50, 51, 52, 53))
    c = coords_rand(1, 5, 6, 54)
    dq, dk, dv = oracle.na3d_bwd(q, k, v, dout, WINDOW, 0.3, coords=c, qk_norm=True, eps=0.0)
    assert np.max(np.abs(np.sum(dq * q, -1))) < 1e-12
    assert np.max(np.abs(np.sum(dk * k, -1))) < 1e-12
    assert np.max(np.abs(dq)) > 1e-3 and np.max(np.abs(dk)) > 1e-3


def test_bwd_sampled_rows_match_full():
    q, k, v, dout = (rand(SHAPE, s) for s in (60, 61, 62, 63))
    c = coords_rand(1, 5, 6, 64)
    gate = rand(SHAPE, 65)
    kw = dict(coords=c, qk_norm=True, eps=1e-6, gate=gate)
    dq, dk, dv, dg = oracle.na3d_bwd(q, k, v, dout, WINDOW, 0.3, **kw)
    sq, sk = np.array([3, 17, 100, 179]), np.array([0, 44, 150])
    a, b, cc, g2 = oracle.na3d_bwd(q, k, v, dout, WINDOW, 0.3, selq=sq, selk=sk, **kw)
    d = SHAPE[-1]
    np.testing.assert_allclose(a, dq.reshape(-1, d)[sq], atol=1e-13)
    np.testing.assert_allclose(b, dk.reshape(-1, d)[sk], atol=1e-13)
    np.testing.assert_allclose(cc, dv.reshape(-1, d)[sk], atol=1e-13)
    np.testing.assert_allclose(g2, dg.reshape(-1, d)[sq], atol=1e-13)
