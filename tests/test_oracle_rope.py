"""Pins of the oracle's rotary-embedding decode (the positional reading the
paper leaves open).

The rotation is pinned to RoFormer's complex form (each plane a complex
number multiplied by e^{i pos theta}), to hand-worked values, and to its two
defining properties (lengths kept; scores depend on position differences
only).  The decode is pinned by the full-rank special case (exact factors:
the latent decode must equal rotary attention over the dense keys, computed
with explicit rotation matrices and the library attention routine), by its
reduction to the plain decode at one token, and by a scalar brute force.
Planted mistakes (a wrong sign, the interleaved pairing) must fail them.
"""

import math

import numpy as np
import pytest
import torch

from oracle import attention, rope
from test_oracle_attention import _full_rank_case, _random_case


def test_frequencies_closed_form():
    np.testing.assert_allclose(rope.frequencies(4, 100.0), [1.0, 0.1], rtol=1e-15)
    th = rope.frequencies(128, 10000.0)
    assert th[0] == 1.0 and th.shape == (64,)
    np.testing.assert_allclose(th[32], 0.01, rtol=1e-14)            # 10000^(-64/128)
    np.testing.assert_allclose(th[1:] / th[:-1], 10000.0 ** (-2 / 128), rtol=1e-13)


def test_hand_worked_rotations():
    half_turn = math.pi / 2
    np.testing.assert_allclose(rope.rotate([1, 0, 0, 0], half_turn, 100.0), [0, 0, 1, 0], atol=1e-15)
    np.testing.assert_allclose(rope.rotate([0, 0, 1, 0], half_turn, 100.0), [-1, 0, 0, 0], atol=1e-15)
    # second plane (theta = 0.1): a quarter turn needs pos = 5 pi
    np.testing.assert_allclose(rope.rotate([0, 1, 0, 0], 5 * math.pi, 100.0), [0, 0, 0, 1], atol=1e-14)
    np.testing.assert_allclose(rope.rotate([0, 0, 0, 1], 5 * math.pi, 100.0), [0, -1, 0, 0], atol=1e-14)
    # position 0 is the identity
    x = np.random.default_rng(0).standard_normal(8)
    assert np.array_equal(rope.rotate(x, 0, 10000.0), x)


def _complex_form(x, pos, base):
    d = x.shape[-1]
    half = d // 2
    theta = base ** (-np.arange(half) * 2.0 / d)
    z = x[..., :half] + 1j * x[..., half:]
    z = z * np.exp(1j * np.asarray(pos, dtype=float)[..., None] * theta)
    return np.concatenate([z.real, z.imag], axis=-1)


def test_rotation_equals_complex_multiplication():
    g = np.random.default_rng(1)
    X = g.standard_normal((50, 128))
    pos = g.integers(0, 200000, size=50)
    np.testing.assert_allclose(rope.rotate(X, pos, 10000.0), _complex_form(X, pos, 10000.0),
                               rtol=1e-12, atol=1e-12)
    X = g.standard_normal((7, 6))
    np.testing.assert_allclose(rope.rotate(X, np.arange(7) * 3, 500.0),
                               _complex_form(X, np.arange(7) * 3, 500.0), atol=1e-13)


def test_lengths_kept_and_only_differences_matter():
    g = np.random.default_rng(2)
    for _ in range(20):
        q, k = g.standard_normal((2, 64))
        p, t, s = (int(v) for v in g.integers(0, 100000, size=3))
        np.testing.assert_allclose(np.linalg.norm(rope.rotate(k, t, 10000.0)), np.linalg.norm(k), rtol=1e-13)
        a = rope.rotate(q, p, 10000.0) @ rope.rotate(k, t, 10000.0)
        b = rope.rotate(q, p + s, 10000.0) @ rope.rotate(k, t + s, 10000.0)
        assert abs(a - b) < 1e-9 * (1 + abs(a))


def _rot_matrix(d, pos, base):
    # the block rotation written out as a d x d matrix: plane (i, i + d/2)
    half = d // 2
    M = np.zeros((d, d))
    for i in range(half):
        th = pos * base ** (-2.0 * i / d)
        c, s = math.cos(th), math.sin(th)
        M[i, i], M[i, i + half] = c, -s
        M[i + half, i], M[i + half, i + half] = s, c
    return M


def _reference_rope_sdpa(c, base):
    bk = c["bk"]
    H_q, H_kv, d = bk.num_q_heads, bk.num_kv_heads, bk.head_dim
    out = np.zeros(c["q"].shape)
    for b, x in enumerate(c["xs"]):
        T = x.shape[0]
        if T == 0:
            continue
        K = (x @ c["W_k"]).reshape(T, H_kv, d)
        K = np.stack([K[t] @ _rot_matrix(d, t, base).T for t in range(T)])     # rotate each key
        V = (x @ c["W_v"]).reshape(T, H_kv, d)
        qr = c["q"][b] @ _rot_matrix(d, T - 1, base).T
        Kt = torch.from_numpy(K).permute(1, 0, 2).repeat_interleave(H_q // H_kv, dim=0).contiguous()
        Vt = torch.from_numpy(V).permute(1, 0, 2).repeat_interleave(H_q // H_kv, dim=0).contiguous()
        o = torch.nn.functional.scaled_dot_product_attention(torch.from_numpy(qr).view(H_q, 1, d), Kt, Vt)
        out[b] = o.view(H_q, d).numpy()
    return out


CASES = [
    # (H_q, H_kv, d, group map, m, lengths)
    (4, 4, 4, [1, 0, 1, 1], 24, [37]),
    (8, 4, 6, [0, 1, 1, 0], 30, [70, 5]),
    (6, 6, 2, [2, 0, 1, 2, 0, 2], 16, [90, 1]),
]


@pytest.mark.parametrize("case", CASES)
def test_full_rank_equals_dense_rotary_attention(case):
    c = _full_rank_case(4321, *case)
    base = 50.0                       # large angles at these lengths: every plane turns many times
    got = rope.decode(c["q"], c["pool"], c["table"], c["lens"], c["R_blocks"], c["R_v"], c["bk"],
                      base, chunk=None)
    np.testing.assert_allclose(got, _reference_rope_sdpa(c, base), rtol=1e-9, atol=1e-10)


def test_one_token_reduces_to_plain_decode():
    bk, R_blocks, R_v, q, Zs, tbl, pool, lens = _random_case(11, d=4, lens=(1,))
    got = rope.decode(q, pool, tbl, lens, R_blocks, R_v, bk, 10000.0)
    ref = attention.decode(q, pool, tbl, lens, R_blocks, R_v, bk)
    np.testing.assert_allclose(got, ref, rtol=1e-14, atol=1e-15)


def test_shift_of_every_position_changes_nothing():
    bk, R_blocks, R_v, q, Zs, tbl, pool, lens = _random_case(12, d=6, lens=(130, 17))
    a = rope.decode(q, pool, tbl, lens, R_blocks, R_v, bk, 1000.0)
    b = rope.decode(q, pool, tbl, lens, R_blocks, R_v, bk, 1000.0, pos0=123457)
    np.testing.assert_allclose(a, b, rtol=1e-7, atol=1e-9)
    c = rope.decode(q, pool, tbl, lens, R_blocks, R_v, bk, 1000.0, chunk=64)
    np.testing.assert_allclose(c, a, rtol=1e-12, atol=1e-14)
    assert not np.allclose(a, attention.decode(q, pool, tbl, lens, R_blocks, R_v, bk), atol=1e-3)


def test_brute_force_scalar_loops():
    bk, R_blocks, R_v, q, Zs, tbl, pool, lens = _random_case(13, d=4, lens=(9, 3))
    base = 30.0
    got = rope.decode(q, pool, tbl, lens, R_blocks, R_v, bk, base, chunk=None)
    d, half = bk.head_dim, bk.head_dim // 2
    for b, (Zk, Zv) in enumerate(Zs):
        T = lens[b]
        for h in range(bk.num_q_heads):
            kv = h // (bk.num_q_heads // bk.num_kv_heads)
            grp = bk.group_of_kv[kv]
            j = sorted(i for i in range(bk.num_kv_heads) if bk.group_of_kv[i] == grp).index(kv)
            col0 = sum(bk.ranks[:grp])
            # the query turned by its position, plane by plane
            qr = [0.0] * d
            for i in range(half):
                ang = (T - 1) * base ** (-2.0 * i / d)
                qr[i] = q[b, h, i] * math.cos(ang) - q[b, h, i + half] * math.sin(ang)
                qr[i + half] = q[b, h, i + half] * math.cos(ang) + q[b, h, i] * math.sin(ang)
            s = []
            for t in range(T):
                k = [sum(Zk[t, col0 + r] * R_blocks[grp][r, j * d + c] for r in range(bk.ranks[grp]))
                     for c in range(d)]
                acc = 0.0
                for i in range(half):
                    ang = t * base ** (-2.0 * i / d)
                    ka = k[i] * math.cos(ang) - k[i + half] * math.sin(ang)
                    kb = k[i + half] * math.cos(ang) + k[i] * math.sin(ang)
                    acc += ka * qr[i] + kb * qr[i + half]
                s.append(acc / math.sqrt(d))
            mx = max(s)
            e = [math.exp(v - mx) for v in s]
            tot = sum(e)
            for c in range(d):
                o = 0.0
                for t in range(T):
                    o += e[t] / tot * sum(Zv[t, r] * R_v[r, kv * d + c] for r in range(bk.value_rank))
                assert abs(o - got[b, h, c]) < 1e-12 * (1 + abs(o))


def test_planted_mistakes_are_caught(monkeypatch):
    c = _full_rank_case(77, 4, 4, 4, [1, 0, 1, 1], 24, [37])
    base = 50.0
    ref = _reference_rope_sdpa(c, base)

    def run():
        return rope.decode(c["q"], c["pool"], c["table"], c["lens"], c["R_blocks"], c["R_v"],
                           c["bk"], base, chunk=None)
    np.testing.assert_allclose(run(), ref, rtol=1e-9, atol=1e-10)
    orig = rope.rotate

    def wrong_sign(X, pos, b):                 # turning the other way
        return orig(X, -np.asarray(pos), b)

    def interleaved(X, pos, b):                # planes (2i, 2i+1) instead of (i, i + d/2)
        X = np.asarray(X, dtype=np.float64)
        d = X.shape[-1]
        idx = np.concatenate([np.arange(0, d, 2), np.arange(1, d, 2)])
        inv = np.argsort(idx)
        return orig(X[..., idx], pos, b)[..., inv]

    def key_only(X, pos, b):                   # the query left unrotated
        return orig(X, pos, b) if np.ndim(pos) > 0 else np.asarray(X, dtype=np.float64)

    for mutant in (wrong_sign, interleaved, key_only):
        monkeypatch.setattr(rope, "rotate", mutant)
        assert not np.allclose(run(), ref, rtol=1e-6, atol=1e-6), mutant.__name__
        monkeypatch.undo()
    # and the rotation pins themselves reject the first two
    x = np.random.default_rng(3).standard_normal((5, 8))
    for mutant in (wrong_sign, interleaved):
        assert not np.allclose(mutant(x, np.arange(5) + 1, 100.0), _complex_form(x, np.arange(5) + 1, 100.0))
