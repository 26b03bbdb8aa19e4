"""Pins of the rotary-embedding oracle against closed forms and invariants (CPU only).

The position rule is the paper's (Section 2, "Algorithm implementation": each
token keeps its Repeated-Prefix Forward position); the rotation is the
standard rotary embedding. None of these checks re-evaluates the oracle's own
formula: they compare it with values written out by hand, with the
repeated-layout positions, and with properties any correct rotation has.
"""
import math

import numpy as np
import pytest

from oracle import grouped_positions, inv_freq, rope


def test_grouped_positions_small_example():
    # prefix of 3, members of 2 and 1 rows; a second group with prefix 2 and one member of 2 rows
    pre, suf = grouped_positions([3, 2], [2, 1], [2, 1, 2])
    assert pre.tolist() == [0, 1, 2, 0, 1]
    assert suf.tolist() == [3, 4, 3, 2, 3]


def test_grouped_positions_are_the_repeated_layout_positions():
    rng = np.random.default_rng(0)
    prefix = [5, 0, 9]
    groups = [3, 2, 0]
    suffix = list(rng.integers(0, 6, sum(groups)))
    pre, suf = grouped_positions(prefix, groups, suffix)
    cu_p = np.concatenate([[0], np.cumsum(prefix)])
    cu_s = np.concatenate([[0], np.cumsum(suffix)])
    m = 0
    for g, (p, gs) in enumerate(zip(prefix, groups)):
        for _ in range(gs):
            seq = np.concatenate([pre[cu_p[g]:cu_p[g + 1]], suf[cu_s[m]:cu_s[m + 1]]])
            assert seq.tolist() == list(range(p + suffix[m]))  # member i is [P; R_i] at 0 .. P+S_i-1
            m += 1
    assert len(pre) == sum(prefix) and len(suf) == sum(suffix)


def test_closed_form_single_pair():
    # d = 2: one pair, angle = position (base ** 0 = 1), for any base and either layout
    for interleaved in (False, True):
        out = rope(np.array([[[1.0, 0.0]], [[0.0, 1.0]]]), np.array([1, 1]), 10000.0, interleaved=interleaved)
        assert np.allclose(out[0, 0], [math.cos(1.0), math.sin(1.0)], atol=1e-15)
        assert np.allclose(out[1, 0], [-math.sin(1.0), math.cos(1.0)], atol=1e-15)


def test_closed_form_frequencies_and_layouts():
    # d = 4, base 10000: pair 0 turns 1 rad per position, pair 1 turns 10000 ** (-1/2) = 0.01 rad
    assert np.allclose(inv_freq(4, 10000.0), [1.0, 0.01], rtol=1e-15)
    x = np.zeros((1, 1, 4))
    c, s = math.cos(1.0), math.sin(1.0)
    # half-split: pair 1 is (x1, x3); at position 100 it turns by 1 rad
    x[0, 0] = [0.0, 1.0, 0.0, 0.0]
    assert np.allclose(rope(x, np.array([100]), 10000.0)[0, 0], [0.0, c, 0.0, s], atol=1e-12)
    # interleaved: pair 1 is (x2, x3)
    x[0, 0] = [0.0, 0.0, 1.0, 0.0]
    assert np.allclose(rope(x, np.array([100]), 10000.0, interleaved=True)[0, 0], [0.0, 0.0, c, s], atol=1e-12)
    # half-split pair 0 is (x0, x2): x2 -> (-sin, cos) on (x0, x2) at position 1
    x[0, 0] = [0.0, 0.0, 1.0, 0.0]
    assert np.allclose(rope(x, np.array([1]), 10000.0)[0, 0], [-s, 0.0, c, 0.0], atol=1e-12)


def test_position_zero_is_identity_and_tail_passes_through():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((3, 2, 16))
    assert np.array_equal(rope(x, np.zeros(3, np.int64), 500.0), x)
    y = rope(x, np.array([7, 300, 12345]), 10000.0, rotary_dim=8)
    assert np.array_equal(y[..., 8:], x[..., 8:])
    assert not np.allclose(y[..., :8], x[..., :8])


@pytest.mark.parametrize("interleaved", [False, True])
def test_rotation_is_orthogonal_and_inverse_undoes_it(interleaved):
    rng = np.random.default_rng(2)
    x = rng.standard_normal((50, 3, 32))
    pos = rng.integers(0, 40000, 50)
    y = rope(x, pos, 10000.0, interleaved=interleaved)
    assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)
    assert np.allclose(rope(y, pos, 10000.0, interleaved=interleaved, inverse=True), x, atol=1e-12)
    # inverse is the vector-Jacobian product: <R x, g> = <x, R^T g>
    g = rng.standard_normal(x.shape)
    assert np.isclose(np.sum(y * g), np.sum(x * rope(g, pos, 10000.0, interleaved=interleaved, inverse=True)))


@pytest.mark.parametrize("interleaved", [False, True])
def test_rotations_compose_and_scores_depend_on_relative_position(interleaved):
    rng = np.random.default_rng(3)
    q = rng.standard_normal((1, 1, 64))
    k = rng.standard_normal((1, 1, 64))
    a, b = np.array([37]), np.array([1200])
    # R(a) R(b) = R(a + b)
    two = rope(rope(q, a, 10000.0, interleaved=interleaved), b, 10000.0, interleaved=interleaved)
    assert np.allclose(two, rope(q, a + b, 10000.0, interleaved=interleaved), atol=1e-12)
    # <R(m) q, R(n) k> depends only on m - n
    def score(m, n):
        return float(np.sum(rope(q, np.array([m]), 10000.0, interleaved=interleaved) *
                            rope(k, np.array([n]), 10000.0, interleaved=interleaved)))
    assert math.isclose(score(100, 40), score(4160, 4100), rel_tol=1e-10, abs_tol=1e-12)
    assert not math.isclose(score(100, 40), score(100, 41), rel_tol=1e-6)


def test_layouts_are_a_permutation_of_each_other():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((20, 2, 16))
    pos = rng.integers(0, 5000, 20)
    perm = np.concatenate([np.arange(0, 16, 2), np.arange(1, 16, 2)])  # interleaved -> half-split order
    via_half = rope(x[..., perm], pos, 10000.0)
    inv = np.argsort(perm)
    assert np.allclose(via_half[..., inv], rope(x, pos, 10000.0, interleaved=True), atol=1e-13)


def test_grouped_rope_matches_repeated_layout_rows():
    """Rotating the grouped rows equals rotating each member's [P; R_i] at positions 0..P+S_i-1."""
    rng = np.random.default_rng(5)
    prefix, groups, suffix = [6, 3], [2, 2], [4, 0, 5, 2]
    pre_x = rng.standard_normal((sum(prefix), 2, 8))
    suf_x = rng.standard_normal((sum(suffix), 2, 8))
    pre_pos, suf_pos = grouped_positions(prefix, groups, suffix)
    got_pre = rope(pre_x, pre_pos, 10000.0)
    got_suf = rope(suf_x, suf_pos, 10000.0)
    cu_p = np.concatenate([[0], np.cumsum(prefix)])
    cu_s = np.concatenate([[0], np.cumsum(suffix)])
    m = 0
    for g, gs in enumerate(groups):
        for _ in range(gs):
            seq = np.concatenate([pre_x[cu_p[g]:cu_p[g + 1]], suf_x[cu_s[m]:cu_s[m + 1]]])
            rep = rope(seq, np.arange(len(seq)), 10000.0)
            p = prefix[g]
            assert np.array_equal(rep[:p], got_pre[cu_p[g]:cu_p[g + 1]])
            assert np.array_equal(rep[p:], got_suf[cu_s[m]:cu_s[m + 1]])
            m += 1
