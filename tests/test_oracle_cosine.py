"""Pins of the oracle's retrieval keys and cosine lookup (Section 3.2,
"Decoding experience memory" and "Context-compatible retrieval"; Section 4,
"Memory and retrieval": 256-dimensional int8 keys from a fixed random
projection of the final-layer state).

Each check ties the oracle to something other than itself: hand-computed
codes, exact invariances of the definition, an independent exact-rational
evaluation of the projection, brute-force float cosines, and the paper's own
boundary example."""
from fractions import Fraction

import numpy as np
import pytest

import oracle
import synth
import keycheck


def _eye(n):
    return np.eye(n, dtype=np.float64)


# ---------------------------------------------------------------- key encode

def test_encode_hand_values():
    # R = I: v = h, scale 127 / max|h|, round half to even
    assert oracle.key_encode(_eye(4), np.array([1.0, 0.5, -1.0, 0.25])).tolist() == \
        [[127, 64, -127, 32]]          # 63.5 -> 64, 31.75 -> 32
    assert oracle.key_encode(_eye(4), np.array([2.0, 1.0, -0.5, 0.0])).tolist() == \
        [[127, 64, -32, 0]]            # 63.5 -> 64, -31.75 -> -32
    # exact halves: 62.5 -> 62 and -62.5 -> -62 (to even), 63.5 -> 64
    assert oracle.key_encode(_eye(4), np.array([127.0, 62.5, -62.5, 63.5])).tolist() == \
        [[127, 62, -62, 64]]


def test_encode_zero_and_range():
    R = synth.key_projection(48, 3).astype(np.float64)
    assert (oracle.key_encode(R, np.zeros(48)) == 0).all()
    h = synth.hidden_states(20, 48, 4).astype(np.float64)
    k = oracle.key_encode(R, h).astype(np.int32)
    assert (np.abs(k).max(axis=1) == 127).all()


def test_encode_scale_and_sign_invariance():
    # a power-of-two scale multiplies every product and partial sum exactly,
    # so the codes cannot change; negating h negates them (rounding is symmetric)
    R = synth.key_projection(96, 5).astype(np.float64)
    h = synth.hidden_states(6, 96, 6).astype(np.float64)
    k = oracle.key_encode(R, h)
    for e in (-7, -1, 1, 6):
        assert (oracle.key_encode(R, h * 2.0 ** e) == k).all()
    assert (oracle.key_encode(R, -h) == -k.astype(np.int16)).all()


def test_encode_matches_float_projection():
    # numpy's float64 R @ h (another summation order) quantised the same way:
    # the codes agree except where the scaled value sits within 1e-9 of a half
    R = synth.key_projection(256, 7).astype(np.float64)
    h = synth.hidden_states(30, 256, 8).astype(np.float64)
    k = oracle.key_encode(R, h).astype(np.int64)
    v = h @ R.T
    x = v * 127.0 / np.abs(v).max(axis=1, keepdims=True)
    near_half = np.abs(np.abs(x - np.floor(x)) - 0.5) < 1e-9
    assert (np.abs(k - x) <= 0.5 + 1e-9).all()
    assert ((k == np.rint(x)) | near_half).all()


def _exact_codes(R, h):
    """The encode definition in exact rationals: v_j = sum_k R_jk h_k with no
    rounding at all (so no summation order enters), then code_j =
    round-half-even(v_j * 127 / max |v|), also exact. Returns the codes and
    the exact scaled values."""
    kd, H = R.shape
    hf = [Fraction(float(t)) for t in h]
    v = [sum((Fraction(float(R[j, k])) * hf[k] for k in range(H)), Fraction(0)) for j in range(kd)]
    m = max(abs(t) for t in v)
    if m == 0:
        return [0] * kd, [Fraction(0)] * kd
    x = [t * 127 / m for t in v]
    codes = []
    for t in x:
        f = t.numerator // t.denominator            # floor
        r = t - f
        c = f + 1 if (r > Fraction(1, 2) or (r == Fraction(1, 2) and f % 2 == 1)) else f
        codes.append(int(c))
    return codes, x


@pytest.mark.parametrize("kd,H,n,seed", [(5, 40, 3, 9), (24, 512, 2, 11), (256, 64, 2, 13)])
def test_encode_exact_rational_reference(kd, H, n, seed):
    """The oracle's fp64 codes equal the exact rational codes, except where the
    exact scaled value lies within the fp64 summation bound of a half-integer
    (then either neighbour is a correct rounding of an fp64 evaluation)."""
    R = synth.key_projection(H, seed)[:kd].astype(np.float64)
    h = synth.hidden_states(n, H, seed + 1).astype(np.float64)
    k = oracle.key_encode(R, h)
    v = oracle.key_project(R, h)
    _, d = keycheck.scaled_bounds(R, h, v)
    band = 0
    for r in range(n):
        want, x = _exact_codes(R, h[r])
        for j in range(kd):
            if int(k[r, j]) == want[j]:
                continue
            frac = abs(float(x[j] - (x[j].numerator // x[j].denominator)) - 0.5)
            assert frac <= d[r, j] and abs(int(k[r, j]) - want[j]) == 1, (r, j, int(k[r, j]), want[j])
            band += 1
    assert band == 0  # with these seeds no exact value sits that close to a half


def test_encode_projection_is_the_exact_sum_to_fp64_accuracy():
    """or_key_project against the exact rational sum: within the summation
    bound of every component (a dropped term, a transposed R or a wrong
    stride misses it by orders of magnitude)."""
    R = synth.key_projection(96, 17)[:12].astype(np.float64)
    h = synth.hidden_states(2, 96, 18).astype(np.float64)
    v = oracle.key_project(R, h)
    for r in range(2):
        for j in range(12):
            exact = sum(Fraction(float(R[j, k])) * Fraction(float(h[r, k])) for k in range(96))
            s = float(np.abs(R[j]) @ np.abs(h[r]))
            assert abs(v[r, j] - float(exact)) <= 96 * 2.0 ** -53 * s * 1.01


def test_a_different_summation_order_is_valid_under_the_band_check():
    """keycheck accepts codes from another fp64 order (16 interleaved chains,
    as a blocked kernel would sum) and rejects a planted wrong code."""
    H = 2048
    R = synth.key_projection(H, 31).astype(np.float64)
    h = synth.hidden_states(8, H, 32).astype(np.float64)
    v = oracle.key_project(R, h)
    chains = np.zeros((8, 256))
    for c in range(16):
        chains += h[:, c::16] @ R[:, c::16].T
    m = np.abs(chains).max(axis=1, keepdims=True)
    other = np.clip(np.rint(chains * 127.0 / m), -127, 127).astype(np.int8)
    keycheck.check_codes(other, R, h, v)
    keycheck.check_codes(oracle.key_encode(R, h), R, h, v)
    bad = other.astype(np.int64).copy()
    bad[3, 7] += 1 if bad[3, 7] < 127 else -1
    with pytest.raises(AssertionError):
        keycheck.check_codes(bad, R, h, v)


# ---------------------------------------------------------- cosine retrieval

def test_paper_boundary_example():
    # [A, B, C | D, E]: the entry at B has its boundary at C, so its proposal
    # may include C but not D; C itself and E are last positions (p = b) and
    # are not entries
    A, B, C, D, E = 10, 11, 12, 13, 14
    tokens = np.array([A, B, C, D, E], np.int32)
    offs = np.array([0, 3, 5], np.int64)
    keys = synth.random_keys(5, 11)
    q = keys[1]
    d = oracle.cos_lookup(tokens, offs, keys, B, q, k_max=4)
    assert d["token"].tolist() == [B, C]
    assert d["cand_pos"].tolist() == [1] and d["cand_len"].tolist() == [1]
    assert oracle.cos_lookup(tokens, offs, keys, C, keys[2], k_max=4)["n_nodes"] == 1
    assert oracle.cos_lookup(tokens, offs, keys, E, keys[4], k_max=4)["n_nodes"] == 1
    d = oracle.cos_lookup(tokens, offs, keys, A, keys[0], k_max=4)
    assert d["token"].tolist() == [A, B, C]
    d = oracle.cos_lookup(tokens, offs, keys, D, keys[3], k_max=4)
    assert d["token"].tolist() == [D, E]


def _brute(tokens, offs, keys, y, q, k_max):
    """(cos, len, p) of every eligible entry by float arithmetic."""
    out = []
    qf = q.astype(np.float64)
    for s in range(len(offs) - 1):
        a, b = int(offs[s]), int(offs[s + 1]) - 1
        for p in range(a, b):
            if tokens[p] != y:
                continue
            kf = keys[p].astype(np.float64)
            nq, nk = np.linalg.norm(qf), np.linalg.norm(kf)
            cos = float(qf @ kf / (nq * nk)) if nq > 0 and nk > 0 else 0.0
            out.append((cos, min(k_max, b - p), p))
    return sorted(out, key=lambda t: (t[0], t[1], t[2]), reverse=True)


@pytest.mark.parametrize("case", range(6))
def test_cosine_argmax_brute_force(case):
    rng = np.random.default_rng(100 + case)
    T = 400
    tokens = rng.integers(0, 6, T).astype(np.int32)
    cuts = np.sort(rng.choice(np.arange(1, T), 30, replace=False))
    offs = np.concatenate([[0], cuts, [T]]).astype(np.int64)
    keys = synth.random_keys(T, 200 + case)
    for y in range(6):
        q = synth.perturb_key(keys[int(rng.integers(0, T))], 300 + case * 10 + y)
        ref = _brute(tokens, offs, keys, y, q, 16)
        d = oracle.cos_lookup(tokens, offs, keys, y, q, k_max=16, n_cand=4, tree=True)
        assert d["n_found"] == min(4, len(ref))
        for c in range(d["n_found"]):
            cos, ln, p = ref[c]
            if c + 1 < len(ref):
                assert ref[c][0] - ref[c + 1][0] > 1e-12 or ref[c][0] == ref[c + 1][0]
            assert int(d["cand_pos"][c]) == p and int(d["cand_len"][c]) == ln
            assert abs(float(d["cand_cos"][c]) - cos) < 1e-12


def test_ties_prefer_longer_then_later():
    tokens = np.array([5, 7, 7, 7, 5, 7, 7, 5, 7, 8], np.int32)
    offs = np.array([0, 4, 7, 10], np.int64)   # b = 3, 6, 9
    keys = np.zeros((10, 256), np.int8)
    keys[:] = synth.random_keys(1, 12)[0]      # every key identical: cosine ties
    q = keys[0]
    d = oracle.cos_lookup(tokens, offs, keys, 5, q, k_max=2, n_cand=4, tree=True)
    # entries with token 5: p = 0 (len 2), 4 (len 2), 7 (len 2) -> later first
    assert d["cand_pos"].tolist() == [7, 4, 0]
    d = oracle.cos_lookup(tokens, offs, keys, 5, q, k_max=8, n_cand=4, tree=True)
    # lengths 3, 2, 2: the longest first, then later p
    assert d["cand_pos"].tolist() == [0, 7, 4] and d["cand_len"].tolist() == [3, 2, 2]


def test_sign_classes():
    tokens = np.array([1, 1, 1, 1, 9], np.int32)
    offs = np.array([0, 5], np.int64)
    q = synth.random_keys(1, 13)[0]
    keys = np.zeros((5, 256), np.int8)
    keys[0] = -q                  # cos = -1
    keys[1] = 0                   # zero key: cos taken as 0
    keys[2] = q                   # cos = +1
    keys[3] = np.where(np.arange(256) < 128, q, -q)  # a smaller positive or negative
    d = oracle.cos_lookup(tokens, offs, keys, 1, q, k_max=1, n_cand=4, tree=True)
    order = d["cand_pos"].tolist()
    assert order[0] == 2 and order[-1] == 0
    assert order.index(1) < order.index(0)


def test_zero_query_ranks_by_length_then_position():
    rng = np.random.default_rng(14)
    tokens = rng.integers(0, 3, 200).astype(np.int32)
    offs = np.array([0, 50, 120, 200], np.int64)
    keys = synth.random_keys(200, 15)
    d = oracle.cos_lookup(tokens, offs, keys, 1, np.zeros(256, np.int8), k_max=16, n_cand=4,
                          tree=True)
    ref = []
    for s in range(3):
        a, b = int(offs[s]), int(offs[s + 1]) - 1
        ref += [(min(16, b - p), p) for p in range(a, b) if tokens[p] == 1]
    ref.sort(reverse=True)
    assert list(zip(d["cand_len"].tolist(), d["cand_pos"].tolist())) == ref[:4]


def test_only_matching_tokens_and_greedy_fallback():
    tokens = np.array([3, 4, 5, 6, 7], np.int32)
    offs = np.array([0, 5], np.int64)
    keys = synth.random_keys(5, 16)
    # the identical key sits at a different token: never chosen
    d = oracle.cos_lookup(tokens, offs, keys, 9, keys[1], k_max=4)
    assert d["n_nodes"] == 1 and d["token"].tolist() == [9] and d["n_found"] == 0
    d = oracle.cos_lookup(tokens, offs, keys, 4, keys[1], k_max=2)
    assert d["token"].tolist() == [4, 5, 6]


def test_tree_merges_top_candidates():
    # two near-equal contexts after token 1 that share the first next token
    tokens = np.array([1, 2, 3, 0, 1, 2, 4, 0, 1, 5, 6, 0], np.int32)
    offs = np.array([0, 4, 8, 12], np.int64)
    q = synth.random_keys(1, 17)[0]
    keys = np.zeros((12, 256), np.int8)
    keys[0] = q
    keys[4] = synth.perturb_key(q, 18, changes=4)
    keys[8] = -q
    d = oracle.cos_lookup(tokens, offs, keys, 1, q, k_max=3, n_cand=3, tree=True)
    assert d["cand_pos"].tolist() == [0, 4, 8]
    # proposals (each ends at its sequence's last position, which it may
    # include): [2, 3, 0], [2, 4, 0], [5, 6, 0], merged in rank order
    assert d["token"].tolist() == [1, 2, 3, 0, 4, 0, 5, 6, 0]
    assert d["parent"].tolist() == [-1, 0, 1, 2, 1, 4, 0, 6, 7]
    assert d["depth"].tolist() == [0, 1, 2, 3, 2, 3, 1, 2, 3]
