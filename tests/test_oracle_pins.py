"""Pins of the CPU oracle against things other than itself.

Each test checks the oracle against a value the paper prints, a closed form,
an invariant the method guarantees, a library routine the computation reduces
to, or brute force on tiny inputs, chosen so that a plausible slip (a dropped
term, a wrong sign or index, a transposed operand) fails at least one.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------------------
# number format
# ----------------------------------------------------------------------------

def test_bf16_round_ties_to_even():
    # 8 significant bits: the spacing just above 1.0 is 2^-7.
    assert oracle.round_bf16(1.0 + 2 ** -8) == 1.0                # tie -> even
    assert oracle.round_bf16(1.0 + 3 * 2 ** -8) == 1.0 + 2 ** -6  # tie -> even (up)
    assert oracle.round_bf16(1.0 + 2 ** -8 + 2 ** -30) == 1.0 + 2 ** -7
    assert oracle.round_bf16(-(1.0 + 2 ** -8)) == -1.0
    assert oracle.round_bf16(0.0) == 0.0


def test_bf16_round_matches_torch_on_fp32_values():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(20000) * np.exp(rng.uniform(-20, 20, 20000))).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    ours = np.array([oracle.round_bf16(float(v)) for v in x])
    assert np.array_equal(ours, ref)


# ----------------------------------------------------------------------------
# building blocks
# ----------------------------------------------------------------------------

def test_rmsnorm_closed_forms():
    eps = 1e-6
    g = np.ones(8, np.float32)
    # constant vector c: every output is c / sqrt(c^2 + eps)
    for c in (3.0, -0.5, 1e-3):
        y = oracle.rmsnorm(np.full(8, c), g, eps)
        assert np.allclose(y, c / math.sqrt(c * c + eps), rtol=1e-15, atol=0)
    # (3, 4) pattern: mean square 12.5
    x = np.array([3.0, 4.0] * 4)
    y = oracle.rmsnorm(x, g, 0.0)
    assert np.allclose(y, x / math.sqrt(12.5), rtol=1e-15)
    # gains multiply elementwise after normalisation
    gg = np.arange(1, 9).astype(np.float32)
    y2 = oracle.rmsnorm(x, gg, 0.0)
    assert np.allclose(y2, x / math.sqrt(12.5) * gg, rtol=1e-15)
    # unit gains give unit RMS
    z = np.random.default_rng(1).standard_normal(256)
    assert abs(np.sqrt(np.mean(oracle.rmsnorm(z, np.ones(256, np.float32), 0.0) ** 2)) - 1) < 1e-14


@pytest.mark.parametrize("d", [4, 64, 128])
def test_rope_basis_closed_form(d):
    theta, pos = 1e4, 37.0
    h = d // 2
    for i in (0, 1, h - 1):
        ang = pos * theta ** (-2.0 * i / d)
        e = np.zeros(d); e[i] = 1.0
        r = oracle.rope(e, pos, theta)
        want = np.zeros(d); want[i] = math.cos(ang); want[i + h] = math.sin(ang)
        assert np.allclose(r, want, atol=1e-15)
        e2 = np.zeros(d); e2[i + h] = 1.0
        r2 = oracle.rope(e2, pos, theta)
        want2 = np.zeros(d); want2[i] = -math.sin(ang); want2[i + h] = math.cos(ang)
        assert np.allclose(r2, want2, atol=1e-15)


def test_rope_relative_position_and_norm():
    rng = np.random.default_rng(2)
    q, k = rng.standard_normal(128), rng.standard_normal(128)
    theta = 1e6
    base = oracle.rope(q, 100, theta) @ oracle.rope(k, 60, theta)
    for shift in (1, 17, 5000):
        s = oracle.rope(q, 100 + shift, theta) @ oracle.rope(k, 60 + shift, theta)
        assert abs(s - base) < 1e-9 * (1 + abs(base))
    assert abs(np.linalg.norm(oracle.rope(q, 1234, theta)) - np.linalg.norm(q)) < 1e-12
    assert np.allclose(oracle.rope(q, 0, theta), q, atol=0)


def test_attention_closed_forms():
    rng = np.random.default_rng(3)
    d = 16
    q = rng.standard_normal(d)
    # one key: the output is its value
    v = rng.standard_normal((1, d))
    assert np.allclose(oracle.attend(q, rng.standard_normal((1, d)), v, 0.25), v[0], atol=1e-15)
    # equal keys: the output is the mean value
    k = np.repeat(rng.standard_normal((1, d)), 5, axis=0)
    vs = rng.standard_normal((5, d))
    assert np.allclose(oracle.attend(q, k, vs, 0.3), vs.mean(0), atol=1e-14)
    # two keys: weight of the first is the logistic of the scaled score gap
    k2 = rng.standard_normal((2, d))
    v2 = np.stack([np.ones(d), np.zeros(d)])
    scale = 1 / math.sqrt(d)
    gap = (q @ k2[0] - q @ k2[1]) * scale
    assert np.allclose(oracle.attend(q, k2, v2, scale), 1 / (1 + math.exp(-gap)), atol=1e-14)


def test_swiglu_properties():
    # silu(g) * u: zero when either factor path is zero
    assert oracle.swiglu(0.0, 5.0) == 0.0
    assert oracle.swiglu(3.0, 0.0) == 0.0
    # silu(x) - silu(-x) = x (with u = 1), silu(x) -> x, silu(-x) -> 0
    for x in (0.3, 1.7, 4.0):
        assert abs(oracle.swiglu(x, 1.0) - oracle.swiglu(-x, 1.0) - x) < 1e-14
    assert abs(oracle.swiglu(40.0, 2.0) - 80.0) < 1e-12
    assert abs(oracle.swiglu(-40.0, 2.0)) < 1e-12
    # the gate is the first argument: large negative gate silences a large up
    assert abs(oracle.swiglu(-40.0, 1e6)) < 1e-5


@pytest.mark.parametrize("bf16", [False, True])
def test_linear_matches_numpy_matmul(bf16):
    rng = np.random.default_rng(4)
    W = rng.standard_normal((37, 53)).astype(np.float32)
    x = rng.standard_normal((5, 53))
    if bf16:
        Wb = torch.from_numpy(W).to(torch.bfloat16)
        Wstored = Wb.view(torch.int16).numpy().view(np.uint16)
        Wf = Wb.to(torch.float64).numpy()
    else:
        Wstored, Wf = W, W.astype(np.float64)
    y = oracle.linear(Wstored, x)
    assert np.allclose(y, x @ Wf.T, rtol=1e-13, atol=1e-13)


def test_argmax_ties_and_nan():
    assert oracle.argmax(np.array([1, 3, 3, 2], np.float32)) == 1
    assert oracle.argmax(np.array([np.nan, 1, np.nan, 1], np.float32)) == 1
    assert oracle.argmax(np.array([-np.inf, -5], np.float32)) == 1
    assert oracle.argmax(np.array([np.nan, np.nan], np.float32)) == -1


# ----------------------------------------------------------------------------
# retrieval
# ----------------------------------------------------------------------------

def test_paper_boundary_example():
    with open(os.path.join(GOLDEN, "paper_boundary_example.json")) as f:
        g = json.load(f)
    ids = g["tokens"]
    seqs = [[ids[t] for t in s] for s in g["sequences"]]
    tokens = np.array(sum(seqs, []), np.int32)
    offs = np.cumsum([0] + [len(s) for s in seqs]).astype(np.int64)
    for c in g["cases"]:
        ctx = np.array([ids[c["current"]]], np.int32)
        d = oracle.lookup(tokens, offs, g["ngram"], ctx, g["k_max"])
        assert list(d["token"][1:]) == [ids[t] for t in c["draft"]], c
        if c["match_pos"] is None:
            assert d["n_found"] == 0
        else:
            assert d["n_found"] == 1 and int(d["cand_pos"][0]) == c["match_pos"]


def _brute_candidates(tokens, offs, n, ctx, k_max):
    """All eligible (len, pos) pairs by plain enumeration over sequences."""
    out = []
    q = tuple(ctx[-n:])
    for s in range(len(offs) - 1):
        seq = list(tokens[offs[s]:offs[s + 1]])
        for i in range(n - 1, len(seq) - 1):   # i < last index
            if tuple(seq[i - n + 1:i + 1]) == q:
                out.append((min(k_max, len(seq) - 1 - i), int(offs[s]) + i))
    return sorted(out, reverse=True)


@pytest.mark.parametrize("seed", range(12))
def test_lookup_matches_brute_force(seed):
    rng = np.random.default_rng(100 + seed)
    vocab = 3 + seed % 4
    n_seqs = rng.integers(1, 9)
    lens = rng.integers(1, 14, n_seqs)
    tokens = rng.integers(0, vocab, lens.sum()).astype(np.int32)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    for n in (1, 2, 3):
        for k_max in (0, 1, 4, 64):
            ctx = rng.integers(0, vocab, rng.integers(0, 6)).astype(np.int32)
            want = _brute_candidates(tokens, offs, n, ctx, k_max) if len(ctx) >= n else []
            for n_cand in (1, 4):
                d = oracle.lookup(tokens, offs, n, ctx, k_max, n_cand=n_cand, tree=n_cand > 1,
                                  max_nodes=48)
                got = list(zip(d["cand_len"].tolist(), d["cand_pos"].tolist()))
                assert got == want[:n_cand]
                if n_cand == 1 and want:
                    L, p = want[0]
                    assert list(d["token"][1:]) == list(tokens[p + 1:p + 1 + L])


def test_planted_grams_give_their_continuation():
    wl = synth.WORKLOADS["tiny"]
    st = synth.make_store(wl, 7)
    assert len(st.planted) == 8
    for gram in st.planted:
        ctx = np.concatenate([[1, 2, 3], gram[:wl.ngram]]).astype(np.int32)
        d = oracle.lookup(st.tokens, st.seq_offsets, wl.ngram, ctx, wl.k_max)
        assert list(d["token"][1:]) == list(gram[wl.ngram:wl.ngram + wl.k_max])


def _trie_paths(d):
    paths = {}
    for u in range(d["n_nodes"]):
        seq, v = [], u
        while v > 0:
            seq.append(int(d["token"][v]))
            v = int(d["parent"][v])
        paths[u] = tuple(reversed(seq))
    return paths


@pytest.mark.parametrize("seed", range(8))
def test_tree_matches_prefix_enumeration(seed):
    rng = np.random.default_rng(200 + seed)
    vocab = 2 + seed % 3
    lens = rng.integers(4, 20, 12)
    tokens = rng.integers(0, vocab, lens.sum()).astype(np.int32)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    ctx = rng.integers(0, vocab, 4).astype(np.int32)
    for max_nodes in (48, 5):
        d = oracle.lookup(tokens, offs, 2, ctx, 6, n_cand=4, tree=True, max_nodes=max_nodes)
        # brute force: the node list is every distinct proposal prefix in order
        # of first appearance (candidates in rank order), capped at max_nodes
        want, seen, full = [()], {()}, False
        for L, p in _brute_candidates(tokens, offs, 2, ctx, 6)[:4]:
            draft = tuple(tokens[p + 1:p + 1 + L])
            for i in range(1, L + 1):
                if draft[:i] not in seen:
                    if len(want) - 1 >= max_nodes:
                        full = True
                        break
                    seen.add(draft[:i])
                    want.append(draft[:i])
            if full:
                break
        paths = _trie_paths(d)
        assert [paths[u] for u in range(d["n_nodes"])] == want
        for u in range(d["n_nodes"]):
            assert d["depth"][u] == len(paths[u])
            anc = {v for v in range(d["n_nodes"]) if paths[u][:len(paths[v])] == paths[v]}
            assert int(d["anc"][u]) == sum(1 << v for v in anc)


def test_single_candidate_tree_is_the_linear_chain():
    wl = synth.WORKLOADS["tiny"]
    st = synth.make_store(wl, 11)
    for c in range(6):
        ctx, _ = synth.make_context(wl, 11 + c, st, hit=True)
        a = oracle.lookup(st.tokens, st.seq_offsets, 3, ctx, 8)
        b = oracle.lookup(st.tokens, st.seq_offsets, 3, ctx, 8, n_cand=1, tree=True, max_nodes=63)
        for k in ("n_nodes", "token", "parent", "depth", "anc"):
            assert np.array_equal(a[k], b[k])


# ----------------------------------------------------------------------------
# forward and verification
# ----------------------------------------------------------------------------

SMALL = synth.ModelShape(2, 64, 4, 2, 16, 96, 97, 1e4, 1e-6, "f32")
SMALL_BF16 = synth.ModelShape(2, 64, 4, 2, 16, 96, 97, 1e4, 1e-6, "bf16")


def _small(shape, seed, P=23):
    w = synth.make_weights(shape, seed)
    kv = synth.make_kv_prefix(shape, seed, P)
    return oracle.Model(shape, w), w, kv


def test_no_sublayer_output_reduces_to_norm_and_head():
    m, w, kv = _small(SMALL, 5)
    w = dict(w)
    w["wo"] = np.zeros_like(w["wo"])
    w["wd"] = np.zeros_like(w["wd"])
    m = oracle.Model(SMALL, w)
    tok = [3, 50, 96]
    lg, _ = m.forward(kv, tok, [23, 24, 25], np.tril(np.ones((3, 3))))
    for r, t in enumerate(tok):
        xn = oracle.rmsnorm(w["embed"][t].astype(np.float64), w["final_norm"], SMALL.rms_eps)
        want = w["lm_head"].astype(np.float64) @ xn
        assert np.allclose(lg[r], want, rtol=1e-6, atol=1e-7)


@pytest.mark.parametrize("shape", [SMALL, SMALL_BF16], ids=["f32", "bf16"])
def test_causality_later_rows_do_not_change_earlier(shape):
    m, w, kv = _small(shape, 6)
    tok = np.array([5, 9, 13, 17, 21], np.int32)
    vis = np.tril(np.ones((5, 5)))
    a, _ = m.forward(kv, tok, 23 + np.arange(5), vis)
    tok2 = tok.copy(); tok2[3] = 60
    b, _ = m.forward(kv, tok2, 23 + np.arange(5), vis)
    assert np.array_equal(a[:3], b[:3])
    assert not np.array_equal(a[3], b[3])


@pytest.mark.parametrize("shape", [SMALL, SMALL_BF16], ids=["f32", "bf16"])
def test_prefix_slot_permutation_invariance(shape):
    m, w, kv = _small(shape, 7)
    perm = np.random.default_rng(0).permutation(kv.shape[3])
    tok = [1, 2, 3]
    vis = np.tril(np.ones((3, 3)))
    a, ka = m.forward(kv, tok, [23, 24, 25], vis)
    b, kb = m.forward(kv[:, :, :, perm, :], tok, [23, 24, 25], vis)
    assert np.allclose(a, b, rtol=1e-9, atol=1e-9)


def test_gqa_head_mapping_is_equivariant_under_group_swap():
    """Swap the two KV groups (prefix K/V and their projection rows) and the
    matching query heads (projection rows and output-projection columns):
    with query head h reading KV head h // (n_heads / n_kv_heads) the logits
    are unchanged."""
    shape = SMALL
    m, w, kv = _small(shape, 8)
    hd, nq, nkv = shape.head_dim, shape.n_heads, shape.n_kv_heads
    G = nq // nkv
    qperm = np.concatenate([np.arange(hd) + hd * ((h + G) % nq) for h in range(nq)])
    kperm = np.concatenate([np.arange(hd) + hd * ((g + 1) % nkv) for g in range(nkv)])
    w2 = dict(w)
    qkv = w["wqkv"]
    qd, kvd = nq * hd, nkv * hd
    w2["wqkv"] = np.concatenate([qkv[:, qperm], qkv[:, qd + kperm], qkv[:, qd + kvd + kperm]],
                                axis=1)
    w2["wo"] = w["wo"][:, :, qperm]
    kv2 = kv[:, :, [(g + 1) % nkv for g in range(nkv)]]
    m2 = oracle.Model(shape, w2)
    tok, pos, vis = [4, 8], [23, 24], np.tril(np.ones((2, 2)))
    a, _ = m.forward(kv, tok, pos, vis)
    b, _ = m2.forward(kv2, tok, pos, vis)
    assert np.allclose(a, b, rtol=1e-9, atol=1e-9)


def _splice_draft(wl, m, kv, st, seed, j, tree=False):
    """Store with an extra sequence [query | greedy continuation of length j |
    random], so the draft's first j tokens are the model's greedy choice."""
    ctx, _ = synth.make_context(wl, seed, st, hit=True)
    g = oracle.greedy_decode(m, kv, int(ctx[-1]), j)["tokens"] if j else np.zeros(0, np.int32)
    seq = synth.splice_sequence(wl, seed, ctx[-wl.ngram:], g, wl.k_max + 2)
    st2 = st.append(seq)
    return st2, ctx, g


@pytest.mark.parametrize("shape", [SMALL, SMALL_BF16], ids=["f32", "bf16"])
@pytest.mark.parametrize("j", [0, 1, 3, 6])
def test_batched_verify_equals_sequential_greedy(shape, j):
    wl = synth.Workload("t", 9, shape, 23, 6, 2, False, 1, 6, 20, (8, 24), "uniform", 0)
    m, w, kv = _small(shape, 9 + j)
    st = synth.make_store(wl, 9)
    st2, ctx, g = _splice_draft(wl, m, kv, st, 90 + j, j)
    d = oracle.lookup(st2.tokens, st2.seq_offsets, wl.ngram, ctx, wl.k_max)
    assert d["n_nodes"] == wl.k_max + 1
    assert list(d["token"][1:j + 1]) == list(g)
    b = oracle.verify_batched(m, kv, d, wl.rows, False)
    s = oracle.verify_sequential(m, kv, d, False)
    assert b["accept_len"] == s["accept_len"] >= j
    assert b["bonus"] == s["bonus"]
    assert b["path"] == s["path"]
    # accepted rows' KV agree with the sequential decode's
    kept = oracle.commit(b["kv_new"], b["path"])
    assert np.allclose(kept, s["kv_path"], rtol=1e-9, atol=1e-9)


@pytest.mark.parametrize("seed", range(4))
def test_tree_verify_equals_sequential_walk(seed):
    shape = SMALL
    wl = synth.Workload("t", 9, shape, 23, 5, 1, True, 4, 12, 30, (6, 20), "uniform", 0)
    m, w, kv = _small(shape, 30 + seed)
    st = synth.make_store(wl, 30 + seed)
    # put the greedy continuation behind one of several candidates
    ctx, _ = synth.make_context(wl, 300 + seed, st, hit=True)
    g = oracle.greedy_decode(m, kv, int(ctx[-1]), 3)["tokens"]
    st2 = st.append(synth.splice_sequence(wl, 300 + seed, ctx[-1:], g[:2 + seed % 2], 8))
    d = oracle.lookup(st2.tokens, st2.seq_offsets, 1, ctx, wl.k_max, n_cand=4, tree=True,
                      max_nodes=wl.max_nodes)
    b = oracle.verify_batched(m, kv, d, wl.rows, True)
    s = oracle.verify_sequential(m, kv, d, True)
    assert (b["accept_len"], b["bonus"], b["path"]) == (s["accept_len"], s["bonus"], s["path"])
    assert b["accept_len"] >= 2
    assert np.allclose(oracle.commit(b["kv_new"], b["path"]), s["kv_path"], rtol=1e-9, atol=1e-9)


def test_chain_tree_verify_equals_linear():
    shape = SMALL
    m, w, kv = _small(shape, 40)
    wl = synth.Workload("t", 9, shape, 23, 6, 2, False, 1, 6, 20, (8, 24), "uniform", 0)
    st = synth.make_store(wl, 40)
    ctx, _ = synth.make_context(wl, 41, st, hit=True)
    lin = oracle.lookup(st.tokens, st.seq_offsets, 2, ctx, 6)
    tre = oracle.lookup(st.tokens, st.seq_offsets, 2, ctx, 6, n_cand=1, tree=True, max_nodes=6)
    a = oracle.verify_batched(m, kv, lin, 7, False)
    b = oracle.verify_batched(m, kv, tre, 7, True)
    n = lin["n_nodes"]
    assert np.array_equal(a["logits"][:n], b["logits"][:n])
    assert (a["accept_len"], a["bonus"], a["path"]) == (b["accept_len"], b["bonus"], b["path"])


def test_empty_draft_is_a_greedy_step():
    m, w, kv = _small(SMALL, 50)
    d = oracle.lookup(np.zeros(0, np.int32), np.zeros(1, np.int64), 2, np.array([7, 8], np.int32), 6)
    assert d["n_nodes"] == 1
    b = oracle.verify_batched(m, kv, d, 7, False)
    g = oracle.greedy_decode(m, kv, 8, 1)["tokens"]
    assert b["accept_len"] == 0 and b["bonus"] == int(g[0])


@pytest.mark.parametrize("shape", [SMALL, SMALL_BF16], ids=["f32", "bf16"])
def test_chunked_prefill_equals_unchunked(shape):
    m, w, kv = _small(shape, 60)
    toks = np.random.default_rng(0).integers(0, shape.vocab, 29)
    a = oracle.prefill(m, kv, toks, 29)
    b = oracle.prefill(m, kv, toks, 8)
    assert np.array_equal(a["kv_new"], b["kv_new"])
    assert np.array_equal(a["logits_last"], b["logits_last"])
    # and the last row's greedy token equals a plain one-row decode after the
    # prefix extended by every earlier new token
    kv_ext = a["kv_new"][:, :, :, :-1, :]
    lg, _ = m.forward(kv, [int(toks[-1])], [23 + 28], np.ones((1, 1)), kv_extra=kv_ext)
    assert np.array_equal(lg[0], a["logits_last"])


def test_synth_numpy_stream_matches_c_stream():
    lib = synth._load()
    k = synth.key(123, 7)
    assert lib.sy_key(123, 7) == k
    assert [lib.sy_draw(k, i) for i in range(5)] == synth.draws(k, 5).tolist()


@pytest.mark.parametrize("seed", range(3))
def test_tree_rows_equal_their_root_to_node_chains(seed):
    """Each tree row must compute what a linear pass over its own root-to-node
    path computes at that path's last row (tree attention = per-path causal
    attention)."""
    shape = SMALL
    m, w, kv = _small(shape, 70 + seed)
    wl = synth.Workload("t", 9, shape, 23, 5, 1, True, 4, 12, 30, (6, 20), "uniform", 0)
    st = synth.make_store(wl, 70 + seed)
    ctx, _ = synth.make_context(wl, 700 + seed, st, hit=True)
    d = oracle.lookup(st.tokens, st.seq_offsets, 1, ctx, 5, n_cand=4, tree=True, max_nodes=12)
    n = d["n_nodes"]
    assert n > int(d["depth"].max()) + 1, "need a branching tree"
    b = oracle.verify_batched(m, kv, d, 13, True)
    for u in range(n):
        chain, v = [], u
        while v >= 0:
            chain.append(v)
            v = int(d["parent"][v])
        chain.reverse()
        toks = [int(d["token"][c]) for c in chain]
        k = len(chain)
        lg, _ = m.forward(kv, toks, 23 + np.arange(k), np.tril(np.ones((k, k))))
        assert np.array_equal(lg[-1], b["logits"][u])


def test_ffn_gate_is_the_silu_argument():
    """One layer, no attention output. Gate projections are set to -100 for
    this token, so silu(gate) ~ 0 and the feed-forward adds nothing whatever
    the up and down projections are; swapping gate and up would add a large
    term."""
    shape = synth.ModelShape(1, 64, 4, 2, 16, 96, 97, 1e4, 1e-6, "f32")
    w = dict(synth.make_weights(shape, 80))
    kv = synth.make_kv_prefix(shape, 80, 5)
    w["wo"] = np.zeros_like(w["wo"])
    t = 11
    xn = oracle.rmsnorm(w["embed"][t].astype(np.float64), w["ffn_norm"][0], shape.rms_eps)
    wgu = w["wgu"].copy()
    wgu[0, :shape.ffn, :] = (-100.0 * xn / (xn @ xn)).astype(np.float32)[None, :]
    w["wgu"] = wgu
    a, _ = oracle.Model(shape, w).forward(kv, [t], [5], np.ones((1, 1)))
    w0 = dict(w)
    w0["wd"] = np.zeros_like(w["wd"])
    b, _ = oracle.Model(shape, w0).forward(kv, [t], [5], np.ones((1, 1)))
    assert np.allclose(a, b, rtol=1e-12, atol=1e-12)
    # and with a +100 gate the feed-forward term is clearly present
    wgu[0, :shape.ffn, :] *= -1
    c, _ = oracle.Model(shape, w).forward(kv, [t], [5], np.ones((1, 1)))
    assert np.abs(c - b).max() > 1e-2


# ----------------------------------------------------------------------------
# the attention sub-layer inside the decoder forward, in closed form
# ----------------------------------------------------------------------------
# One layer, FFN output zeroed (down projection 0) and the output projection a
# cyclic permutation of the q = H features, so the layer's change of the
# residual stream is exactly the permuted (rounded) attention output. The
# expected values below come from the definitions (RMSNorm of a row, a dense
# product, a rotation of a basis pair, softmax over the visible keys) written
# with numpy and torch's bf16 rounding, not from the oracle's code.

def _fmt(x, shape):
    """fp64 values -> the model's storage format (fp32, or bf16 bits RNE)."""
    t = torch.from_numpy(np.ascontiguousarray(x, np.float64)).to(torch.float32)
    if shape.dtype == "f32":
        return t.numpy()
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _val(a, shape):
    """storage format -> fp64 values."""
    if shape.dtype == "f32":
        return np.asarray(a, np.float64)
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(
        torch.float64).numpy()


def _rnd(x, shape):
    if shape.dtype == "f32":
        return np.asarray(x, np.float64)
    return torch.from_numpy(np.asarray(x, np.float64)).to(torch.bfloat16).to(torch.float64).numpy()


def _one_layer(shape, seed):
    s1 = shape.with_layers(1)
    w = dict(synth.make_weights(s1, seed))
    H, q = s1.hidden, s1.q_dim
    assert q == H
    shift = np.roll(np.eye(H), 1, axis=1)          # (P x)[n] = x[n + 1]
    w["wo"] = _fmt(shift[None], s1).reshape(1, H, q)
    w["wd"] = np.zeros_like(w["wd"])
    return s1, w, shift


@pytest.mark.parametrize("shape", [SMALL, SMALL_BF16], ids=["f32", "bf16"])
def test_zero_queries_attend_uniformly_to_unrotated_values(shape):
    """Query projection 0: every visible key scores 0, so each head's output
    is the mean of the visible value rows of its KV group (prefix values as
    cached, new rows' values as projected, no rotation), rounded to the
    model's format, and the output projection maps it into the stream."""
    s1, w, shift = _one_layer(shape, 41)
    H, hd, nq, nkv = s1.hidden, s1.head_dim, s1.n_heads, s1.n_kv_heads
    q, kvd, grp = s1.q_dim, s1.kv_dim, nq // nkv
    wqkv = w["wqkv"].copy()
    wqkv[0, :q] = 0
    w["wqkv"] = wqkv
    m = oracle.Model(s1, w)
    P, M = 5, 3
    kv = synth.make_kv_prefix(s1, 41, P)
    tok = [7, 19, 88]
    pos = P + np.arange(M)
    resid = np.zeros((2, M, H))
    m.forward(kv, tok, pos, np.tril(np.ones((M, M))), resid=resid)
    emb = _val(w["embed"], s1)
    g = np.asarray(w["attn_norm"][0], np.float64)
    Wv = _val(w["wqkv"][0, q + kvd:], s1)                   # [kvd][H]
    vpre = _val(kv[0, 1], s1)                              # [nkv][P][hd]
    vnew = []
    for t in tok:
        x = emb[t]
        xn = _rnd(x / np.sqrt(np.mean(x * x) + s1.rms_eps) * g, s1)
        vnew.append(_rnd(Wv @ xn, s1).reshape(nkv, hd))
    for r in range(M):
        att = np.zeros(q)
        for h in range(nq):
            gk = h // grp
            rows = list(vpre[gk]) + [vnew[i][gk] for i in range(r + 1)]
            att[h * hd:(h + 1) * hd] = _rnd(np.mean(rows, axis=0), s1)
        got = resid[1, r] - resid[0, r]
        assert np.allclose(got, shift @ att, rtol=0, atol=1e-14), np.abs(got - shift @ att).max()


@pytest.mark.parametrize("shape", [SMALL, SMALL_BF16], ids=["f32", "bf16"])
def test_two_prefix_keys_weight_is_logistic_at_inverse_sqrt_head_dim(shape):
    """One new row at position P = 2 whose query is a * e_0 in head 0 (a
    one-hot embedding row, one nonzero projection weight); its own key and
    value are 0. Prefix key 1 is 0 with value 0; prefix key 2 is k * R(P) e_0
    (the query's direction after the rotation) with value e_0. Head 0's first
    output is then e^s / (2 + e^s) with s = (q_rot . k_2) / sqrt(head_dim);
    head 1 (zero query, same group) averages the three values: 1/3."""
    s1, w, shift = _one_layer(shape, 43)
    H, hd, nq, nkv = s1.hidden, s1.head_dim, s1.n_heads, s1.n_kv_heads
    q, kvd = s1.q_dim, s1.kv_dim
    P, tok, i0, c, a, kk = 2, 5, 9, 1.0, 0.75, 1.5
    emb = np.zeros((s1.vocab, H)); emb[tok, i0] = c
    w["embed"] = _fmt(emb, s1)
    wqkv = np.zeros((1, q + 2 * kvd, H)); wqkv[0, 0, i0] = a
    w["wqkv"] = _fmt(wqkv, s1)
    kv = np.zeros((1, 2, nkv, P, hd))
    half = hd // 2
    kv[0, 0, 0, 1, 0] = kk * np.cos(P)        # angle P * theta^0 on the pair (0, half)
    kv[0, 0, 0, 1, half] = kk * np.sin(P)
    kv[0, 1, 0, 1, 0] = 1.0
    kv = _fmt(kv, s1).reshape(kv.shape)
    m = oracle.Model(s1, w)
    resid = np.zeros((2, 1, H))
    m.forward(kv, [tok], [P], np.ones((1, 1)), resid=resid)
    g = float(w["attn_norm"][0, i0])
    xn = _rnd(c / np.sqrt(c * c / H + s1.rms_eps) * g, s1)
    qa = a * xn
    q_rot = np.array([_rnd(qa * np.cos(P), s1), _rnd(qa * np.sin(P), s1)])
    k2 = _val(kv[0, 0, 0, 1], s1)[[0, half]]
    s = float(q_rot @ k2) / np.sqrt(hd)
    att = np.zeros(q)
    att[0] = _rnd(np.exp(s) / (2.0 + np.exp(s)), s1)
    att[hd] = _rnd(1.0 / 3.0, s1)
    got = resid[1, 0] - resid[0, 0]
    assert abs(s - 1.5 * 0.75 * 8 / 4) < 0.2       # the construction gives s near 2.25
    assert np.allclose(got, shift @ att, rtol=0, atol=1e-14), (got[H - 1], att[0])
