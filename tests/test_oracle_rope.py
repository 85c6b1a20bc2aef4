"""Pins for the oracle's rotary encodings: a complex-number formulation of the
2x2 rotation, closed-form theta values, and the invariants the paper states for
M-RoPE and FlatRoPE (Sec. 3.3, Sec. 4.2)."""
import numpy as np
import pytest

from oracle import rope as R


def _x(rng, n=5, heads=3, D=64):
    return rng.standard_normal((n, heads, D))


def test_rotation_matches_complex_multiplication():
    # Eq. rope-1d rotates pair (x_2d, x_2d+1) like the complex number x_2d + i x_2d+1
    # multiplied by exp(i phi).
    rng = np.random.default_rng(0)
    x = _x(rng)
    phi = rng.uniform(-50, 50, size=(5, 32))
    got = R.rotate_pairs(x, phi)
    zc = (x[..., 0::2] + 1j * x[..., 1::2]) * np.exp(1j * phi)[:, None, :]
    assert np.allclose(got[..., 0::2], zc.real, rtol=0, atol=1e-13)
    assert np.allclose(got[..., 1::2], zc.imag, rtol=0, atol=1e-13)


def test_theta_closed_forms():
    th = R.theta(128)
    assert th[0] == 1.0
    assert th[32] == pytest.approx(0.01, rel=1e-15)          # 10000^(-1/2)
    assert th[63] == pytest.approx(10000 ** (-126 / 128), rel=1e-15)
    assert np.all(np.diff(th) < 0)


def test_axis_assignment_blocked_and_interleaved():
    a = R.axis_assignment(64, (16, 24, 24), False)
    assert list(a[:16]) == [R.AXIS_T] * 16
    assert list(a[16:40]) == [R.AXIS_H] * 24
    assert list(a[40:]) == [R.AXIS_W] * 24
    b = R.axis_assignment(64, (16, 24, 24), True)
    assert list(b[:7]) == [0, 1, 2, 0, 1, 2, 0]
    with pytest.raises(ValueError):
        R.axis_assignment(64, (16, 24, 23), False)


def test_position_zero_is_identity():
    rng = np.random.default_rng(1)
    x = _x(rng)
    assert np.array_equal(R.rope1d(x, np.zeros(5)), x)


def test_mrope_equals_rope1d_when_axes_equal():
    # Sec. 3.3: for t = h = w = m the 3D rotation reduces to Eq. rope-1d.
    rng = np.random.default_rng(2)
    x = _x(rng, D=128)
    m = rng.integers(0, 5000, size=5)
    for sec, inter in [((16, 24, 24), False), ((16, 24, 24), True), ((32, 16, 16), False)]:
        got = R.mrope(x, np.stack([m, m, m]), sec, inter)
        assert np.array_equal(got, R.rope1d(x, m))


def test_flatrope_ignores_section_and_interleave():
    # Sec. 4.2 (i): under FlatRoPE mrope_section and interleaved are irrelevant.
    rng = np.random.default_rng(3)
    x = _x(rng, D=128)
    m = rng.integers(0, 5000, size=5)
    ref = R.flatrope(x, m)
    for sec in [(16, 24, 24), (8, 28, 28), (64, 0, 0)]:
        for inter in (False, True):
            assert np.array_equal(R.mrope(x, np.stack([m, m, m]), sec, inter), ref)


def test_rotation_preserves_norm():
    rng = np.random.default_rng(4)
    x = _x(rng, D=128)
    pos = rng.integers(0, 4000, size=(3, 5))
    y = R.mrope(x, pos)
    assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-12)


def test_scores_invariant_to_shared_shift():
    # R(a)^T R(b) = R(b - a) per pair: q.k after rotation depends on the
    # per-axis position differences only.
    rng = np.random.default_rng(5)
    q = _x(rng, n=1, heads=1, D=128)
    k = _x(rng, n=1, heads=1, D=128)
    pa = rng.integers(0, 3000, size=(3, 1))
    pb = rng.integers(0, 3000, size=(3, 1))
    s0 = np.sum(R.mrope(q, pa) * R.mrope(k, pb))
    for delta in (1, 17, 1000):
        s1 = np.sum(R.mrope(q, pa + delta) * R.mrope(k, pb + delta))
        assert s1 == pytest.approx(s0, rel=1e-9, abs=1e-9)
    # ... and not invariant when only one axis of one side moves
    pb2 = pb.copy()
    pb2[2] += 1
    assert abs(np.sum(R.mrope(q, pa) * R.mrope(k, pb2)) - s0) > 1e-6


def test_composition_adds_angles():
    rng = np.random.default_rng(6)
    x = _x(rng)
    a = rng.integers(0, 100, size=5)
    b = rng.integers(0, 100, size=5)
    assert np.allclose(R.rope1d(R.rope1d(x, a), b), R.rope1d(x, a + b), rtol=0, atol=1e-11)


@pytest.mark.parametrize("inter", [False, True])
def test_w_adjacent_patches_differ_only_in_w_pairs(inter):
    # Sec. 4.2: (t, h, w) and (t, h, w+1) differ only in the W subspace of phi.
    rng = np.random.default_rng(7)
    x = np.repeat(_x(rng, n=1, heads=2, D=128), 2, axis=0)
    p = np.array([[10, 10], [20, 20], [30, 31]])
    y = R.mrope(x, p, (16, 24, 24), inter)
    a = R.axis_assignment(64, (16, 24, 24), inter)
    diff_pairs = np.any(y[0].reshape(2, 64, 2) != y[1].reshape(2, 64, 2), axis=(0, 2))
    assert np.array_equal(diff_pairs, a == R.AXIS_W)


def test_flat_adjacent_tokens_differ_in_every_pair():
    # Sec. 4.2 (ii): under FlatRoPE tokens m and m+1 differ in every pair.
    rng = np.random.default_rng(8)
    x = np.repeat(_x(rng, n=1, heads=2, D=128), 2, axis=0)
    y = R.flatrope(x, np.array([40, 41]))
    diff_pairs = np.all(y[0].reshape(2, 64, 2) != y[1].reshape(2, 64, 2), axis=2)
    assert diff_pairs.all()


def _rotate_half_split(x, phi):
    """The half-split convention of public rotary code: pair d is
    (x_d, x_{d + D/2}), i.e. x * [cos, cos] + [-x2, x1] * [sin, sin]."""
    D = x.shape[-1]
    x1, x2 = x[..., :D // 2], x[..., D // 2:]
    c = np.concatenate([np.cos(phi), np.cos(phi)], axis=-1)[:, None, :]
    s = np.concatenate([np.sin(phi), np.sin(phi)], axis=-1)[:, None, :]
    return x * c + np.concatenate([-x2, x1], axis=-1) * s


@pytest.mark.parametrize("inter", [False, True])
def test_adjacent_pairs_equal_half_split_under_a_row_permutation(inter):
    # Reading of Eq. rope-1d: adjacent pairs (2d, 2d+1).  A half-split model is
    # the same model with the rows of W_q and W_k permuted so that half-split
    # dimension d lands on 2d and d + D/2 on 2d + 1: rotated vectors agree up
    # to that permutation and attention scores agree exactly.
    rng = np.random.default_rng(11)
    D, n = 64, 6
    perm = np.empty(D, dtype=np.int64)           # adjacent index -> half-split index
    perm[0::2] = np.arange(D // 2)
    perm[1::2] = np.arange(D // 2) + D // 2
    pos3 = rng.integers(0, 500, size=(3, n))
    phi = R.phases(pos3, D, (8, 12, 12), inter)
    q_half = rng.standard_normal((n, 2, D))
    k_half = rng.standard_normal((n, 2, D))
    rq_half = _rotate_half_split(q_half, phi)
    rk_half = _rotate_half_split(k_half, phi)
    rq_adj = R.mrope(q_half[..., perm], pos3, (8, 12, 12), inter)
    rk_adj = R.mrope(k_half[..., perm], pos3, (8, 12, 12), inter)
    assert np.allclose(rq_adj, rq_half[..., perm], rtol=0, atol=1e-12)
    s_half = np.einsum("ihd,jhd->hij", rq_half, rk_half)
    s_adj = np.einsum("ihd,jhd->hij", rq_adj, rk_adj)
    assert np.allclose(s_adj, s_half, rtol=1e-12, atol=1e-12)
    # without the permutation the two conventions differ
    assert not np.allclose(R.mrope(q_half, pos3, (8, 12, 12), inter), rq_half, atol=1e-3)
