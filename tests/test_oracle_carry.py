"""Pins of the oracle's rolling-image KV-state carryover (Section 3.4): a
retained span's keys move from positions m to m' as R(m') R(m)^-1 K, values
move unchanged, spans apply in order.

The reference rotation here is complex multiplication (numpy's complex
exponential): the rotary embedding pairs dimension i with i + d/2 and turns
the pair (a, b) = a + ib by the angle pos * theta^(-2i/d)."""
import numpy as np

import oracle

THETA = 1e6


def _rot(v, pos, theta=THETA):
    d = v.shape[-1]
    h = d // 2
    ang = pos * theta ** (-2.0 * np.arange(h) / d)
    z = (v[..., :h] + 1j * v[..., h:]) * np.exp(1j * ang)
    return np.concatenate([z.real, z.imag], axis=-1)


def _cache(L, nkv, T, hd, seed):
    """A cache whose key at slot t is a raw vector rotated to position t."""
    rng = np.random.default_rng(seed)
    raw = rng.standard_normal((L, nkv, T, hd))
    kv = np.zeros((L, 2, nkv, T, hd))
    for t in range(T):
        kv[:, 0, :, t, :] = _rot(raw[:, :, t, :], t)
    kv[:, 1] = rng.standard_normal((L, nkv, T, hd))
    return kv, raw


def test_carried_key_equals_direct_rotation_at_new_position():
    kv, raw = _cache(2, 2, 40, 16, 1)
    out = oracle.kv_carry(kv, [(20, 5, 12)], THETA)
    for i in range(12):
        want = _rot(raw[:, :, 20 + i, :], 5 + i)
        assert np.abs(out[:, 0, :, 5 + i, :] - want).max() < 1e-12
    # values move unchanged, the sources and every other slot stay as they were
    assert np.array_equal(out[:, 1, :, 5:17], kv[:, 1, :, 20:32])
    keep = [t for t in range(40) if not 5 <= t < 17]
    assert np.array_equal(out[:, :, :, keep], kv[:, :, :, keep])


def test_zero_shift_and_round_trip():
    kv, _ = _cache(1, 2, 30, 32, 2)
    same = oracle.kv_carry(kv, [(3, 3, 20)], THETA)
    assert np.abs(same - kv).max() < 1e-13
    there = oracle.kv_carry(kv, [(0, 7, 10)], THETA)
    back = oracle.kv_carry(there, [(7, 0, 10)], THETA)
    assert np.abs(back[:, :, :, 0:10] - kv[:, :, :, 0:10]).max() < 1e-12


def test_rotation_keeps_pair_norms_and_relative_scores():
    kv, raw = _cache(1, 1, 64, 64, 3)
    out = oracle.kv_carry(kv, [(40, 9, 20)], THETA)
    h = 32
    a, b = kv[0, 0, 0, 40:60], out[0, 0, 0, 9:29]
    assert np.allclose(a[:, :h] ** 2 + a[:, h:] ** 2, b[:, :h] ** 2 + b[:, h:] ** 2, atol=1e-12)
    # a query rotated to position p scores a key at m as a function of p - m:
    # shifting both by the same amount keeps every score
    q = np.random.default_rng(4).standard_normal(64)
    s_old = _rot(q, 70) @ a.T
    s_new = _rot(q, 70 - 31) @ b.T
    assert np.abs(s_old - s_new).max() < 1e-10


def test_overlapping_spans_apply_in_order():
    kv, raw = _cache(1, 2, 50, 16, 5)
    # a right shift by 2 over its own source (memmove semantics) ...
    out = oracle.kv_carry(kv, [(4, 6, 8)], THETA)
    for i in range(8):
        assert np.abs(out[0, 0, :, 6 + i] - _rot(raw[0, :, 4 + i], 6 + i)).max() < 1e-12
        assert np.array_equal(out[0, 1, :, 6 + i], kv[0, 1, :, 4 + i])
    # ... and the rolling window: [img1 | img2 | img3] -> [img2 | img3], each
    # span reading the cache as the previous span left it
    roll = oracle.kv_carry(kv, [(20, 10, 10), (30, 20, 10)], THETA)
    for i in range(10):
        assert np.abs(roll[0, 0, :, 10 + i] - _rot(raw[0, :, 20 + i], 10 + i)).max() < 1e-12
        assert np.abs(roll[0, 0, :, 20 + i] - _rot(raw[0, :, 30 + i], 20 + i)).max() < 1e-12
    # reversed order reads img2's slots after img3 landed there: a different cache
    wrong = oracle.kv_carry(kv, [(30, 20, 10), (20, 10, 10)], THETA)
    assert np.abs(wrong[0, 0, :, 10:20] - roll[0, 0, :, 10:20]).max() > 0.1
