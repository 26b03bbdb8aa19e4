"""Plain numpy oracle of rotary position embedding with grouped position ids.

TEST INFRASTRUCTURE ONLY: imported by the tests, never by the product path.

What the paper fixes (Section 2, "Algorithm implementation", the paragraph
after Eq. (4)): every token keeps the position id it has in the
Repeated-Prefix Forward of Eq. (1). In the repeated layout member i is the
sequence [P; R_i] at positions 0 .. P + S_i - 1, so in the grouped layout
prefix row t of a group sits at position t and row j of any member's response
sits at position P + j. Algorithm 1 takes q and k already rotary-encoded;
this module is that step.

The paper names rotary embeddings without defining them. The standard
definition is followed: the first ``rotary_dim``
dimensions of a head vector form rotary_dim / 2 pairs; pair i is rotated by
the angle pos * base ** (-2 i / rotary_dim); the remaining dimensions pass
through unchanged. Two pair layouts are in use and both are provided:
half-split, where pair i is (x[i], x[i + rotary_dim / 2]) (the layout of the
Qwen and LLaMA models), and interleaved, where pair i is (x[2 i], x[2 i + 1]).
The inverse rotation (angle negated) is the vector-Jacobian product of the
rotation, which is orthogonal, so it maps dq, dk of the rotated vectors back.
Everything is computed in float64.
"""
import numpy as np


def grouped_positions(prefix_lens, group_sizes, suffix_lens):
    """(pos_pre, pos_suf): the repeated-layout position of every packed prefix and response row."""
    pre, suf = [np.zeros(0, np.int64)], [np.zeros(0, np.int64)]
    m = 0
    for p, g in zip(prefix_lens, group_sizes):
        p, g = int(p), int(g)
        pre.append(np.arange(p, dtype=np.int64))
        for s in suffix_lens[m:m + g]:
            suf.append(p + np.arange(int(s), dtype=np.int64))
        m += g
    return np.concatenate(pre), np.concatenate(suf)


def inv_freq(rotary_dim, base):
    """Angle per unit position of pair i: base ** (-2 i / rotary_dim)."""
    i = np.arange(rotary_dim // 2, dtype=np.float64)
    return np.float64(base) ** (-2.0 * i / rotary_dim)


def pair_index(head_dim, rotary_dim, interleaved):
    """Dimension indices (first, second) of each rotated pair."""
    half = rotary_dim // 2
    if interleaved:
        return np.arange(0, rotary_dim, 2), np.arange(1, rotary_dim, 2)
    return np.arange(half), np.arange(half, rotary_dim)


def rope(x, positions, base, rotary_dim=None, interleaved=False, inverse=False):
    """Rotate x [rows, heads, head_dim] (any float type) by its rows' positions; returns float64."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    r = d if rotary_dim is None else int(rotary_dim)
    assert r % 2 == 0 and 0 < r <= d
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv_freq(r, base)[None, :]  # [rows, r/2]
    if inverse:
        ang = -ang
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    ia, ib = pair_index(d, r, interleaved)
    a, b = x[..., ia], x[..., ib]
    out = x.copy()
    out[..., ia] = a * c - b * s
    out[..., ib] = b * c + a * s
    return out
