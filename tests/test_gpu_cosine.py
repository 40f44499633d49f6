"""GPU parity of the paper's retrieval (Section 3.2, "Context-compatible
retrieval"; Section 4, "Memory and retrieval"): int8 keys from a fixed random
projection of final-layer states, and the exact cosine lookup over the
entries whose stored token matches the query token. Drafts are integer work
and must match the oracle bit for bit. Keys are integers decided by an fp64
projection that the device sums in another order than the oracle: they must
equal the oracle's codes except where the scaled value lies within the two
orders' rounding bound of a half-integer, where either neighbour is valid
(keycheck). Keys of the verify step's own states are compared with keys of
the oracle's states (the states themselves agree only to rounding)."""
import numpy as np
import pytest

import oracle
import synth
from pfharness import Gpu, assert_same_draft
import keycheck

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pf():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_32166_amd as pf
    pf.lib()
    return pf


def _encode_gpu(pf, kp, h, dtype):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(h, np.float32)).cuda()
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
    keys = torch.zeros(h.shape[0], pf.KEY_DIM, dtype=torch.int8, device="cuda")
    pf.pf_key_encode(kp, t, keys)
    torch.cuda.synchronize()
    return keys.cpu().numpy(), t.to(torch.float64).cpu().numpy()


@pytest.mark.parametrize("H,n,dtype", [(64, 3, "f32"), (256, 70, "f32"), (2048, 17, "bf16"),
                                       (3584, 33, "bf16"), (272, 5, "bf16"), (16, 1, "f32")])
def test_key_encode_valid(pf, H, n, dtype):
    R = synth.key_projection(H, 21)
    h = synth.hidden_states(n, H, 22 + n)
    kp = pf.pf_keyproj_create(R)
    got, hv = _encode_gpu(pf, kp, h, dtype)
    R64 = R.astype(np.float64)
    ref = oracle.key_encode(R64, hv)
    band = keycheck.check_codes(got, R64, hv, oracle.key_project(R64, hv))
    exact = (got == ref).mean()
    print(f"H={H} n={n} {dtype}: {exact:.6f} of the codes equal the oracle's, {band} in the half band")
    assert band > 0 or (got == ref).all()


def test_key_encode_zero_and_scaled_rows(pf):
    H = 128
    R = synth.key_projection(H, 23)
    h = synth.hidden_states(4, H, 24)
    h[1] = 0.0
    h[2] = h[0] * 8.0
    kp = pf.pf_keyproj_create(R)
    got, hv = _encode_gpu(pf, kp, h, "f32")
    assert (got[1] == 0).all()
    assert (got[2] == got[0]).all()
    R64 = R.astype(np.float64)
    keycheck.check_codes(got, R64, hv, oracle.key_project(R64, hv))


def _store(T, n_seqs, vocab, seed, keys=None):
    rng = np.random.default_rng(seed)
    tokens = rng.integers(0, vocab, T).astype(np.int32)
    cuts = np.sort(rng.choice(np.arange(1, T), n_seqs - 1, replace=False))
    offs = np.concatenate([[0], cuts, [T]]).astype(np.int64)
    if keys is None:
        keys = synth.random_keys(T, seed + 1)
    return tokens, offs, keys


def _eligible(tokens, offs, y):
    last = np.zeros(len(tokens), np.int64)
    for s in range(len(offs) - 1):
        last[offs[s]:offs[s + 1]] = offs[s + 1] - 1
    p = np.arange(len(tokens))
    return int(((tokens == y) & (p < last)).sum())


def _cos_case(pf, st, tokens, offs, keys, ctx, q, k_max, tree, n_cand, max_nodes=63):
    import torch
    c = pf.Context(ctx, len(ctx) + 8)
    qd = torch.from_numpy(np.ascontiguousarray(q, np.int8)).cuda()
    draft = pf.new_draft()
    pf.pf_draft_lookup_cosine(st, c, qd, k_max, tree, n_cand, max_nodes if tree else 64, draft)
    torch.cuda.synchronize()
    d = pf.read_draft(draft)
    od = oracle.cos_lookup(tokens, offs, keys, int(ctx[-1]), q, k_max, n_cand=n_cand, tree=tree,
                           max_nodes=max_nodes if tree else 64)
    assert_same_draft(d, od, tree)
    assert int(d["n_eligible"]) == _eligible(tokens, offs, int(ctx[-1]))
    f = od["n_found"]
    assert np.allclose(d["cand_score"][:f], od["cand_cos"], atol=1e-6)
    return d, od


@pytest.mark.parametrize("T,n_seqs,vocab", [(300, 20, 5), (5000, 100, 40), (200000, 800, 3)])
def test_cosine_lookup_bit_exact(pf, T, n_seqs, vocab):
    # vocab 3 over 200k positions gives ~66k entries per token: the scan runs
    # across every block of the grid
    tokens, offs, keys = _store(T, n_seqs, vocab, 31 + T)
    st = pf.pf_store_build(tokens, offs, 2)
    pf.pf_store_attach_keys(st, keys)
    rng = np.random.default_rng(T)
    for case in range(6):
        p = int(rng.integers(0, T))
        y = int(tokens[p])
        q = synth.perturb_key(keys[p], 40 + case) if case % 3 else synth.random_keys(1, 50 + case)[0]
        ctx = np.array([7, 8, y], np.int32)
        tree = case >= 3
        _cos_case(pf, st, tokens, offs, keys, ctx, q, k_max=[16, 4, 64, 8, 16, 63][case], tree=tree,
                  n_cand=[1, 1, 1, 4, 2, 3][case], max_nodes=[63, 63, 63, 48, 20, 63][case])


def test_cosine_lookup_ties_zero_query_and_misses(pf):
    tokens = np.array([5, 7, 7, 7, 5, 7, 7, 5, 7, 8, 9], np.int32)
    offs = np.array([0, 4, 7, 10, 11], np.int64)
    keys = np.repeat(synth.random_keys(1, 60), 11, axis=0)   # identical keys: ties
    st = pf.pf_store_build(tokens, offs, 1)
    pf.pf_store_attach_keys(st, keys)
    for k_max in (0, 1, 2, 8):
        _cos_case(pf, st, tokens, offs, keys, np.array([5], np.int32), keys[0], k_max, True, 4)
    _cos_case(pf, st, tokens, offs, keys, np.array([1, 5], np.int32), np.zeros(256, np.int8), 8,
              True, 4)
    # no entry for the token (9 is the last of its sequence; 3 never occurs)
    for y in (9, 3, 8):
        d, _ = _cos_case(pf, st, tokens, offs, keys, np.array([y], np.int32), keys[0], 8, False, 1)
        assert int(d["n_nodes"]) == 1
    # negative, zero and positive cosines
    k2 = keys.copy()
    k2[0] = -keys[0]
    k2[4] = 0
    st2 = pf.pf_store_build(tokens, offs, 1)
    pf.pf_store_attach_keys(st2, k2)
    _cos_case(pf, st2, tokens, offs, k2, np.array([5], np.int32), keys[0], 8, True, 4)


@pytest.mark.parametrize("lens", [[], [0, 0, 0], [1, 1, 0, 1], [0, 3, 0, 0, 4, 0]],
                         ids=["no_sequences", "only_empty", "single_tokens", "empty_between"])
def test_cosine_lookup_degenerate_stores(pf, lens):
    """Stores with no sequence, only empty ones, only one-token sequences
    (no position has a successor) and empty sequences between real ones:
    drafts bit-exact vs the oracle; nothing eligible gives the greedy draft."""
    lens = np.array(lens, np.int64)
    T = int(lens.sum())
    tokens = (np.arange(T) % 3).astype(np.int32)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    keys = synth.random_keys(T, 62) if T else np.zeros((0, 256), np.int8)
    st = pf.pf_store_build(tokens, offs, 1)
    pf.pf_store_attach_keys(st, keys)
    q = synth.random_keys(1, 63)[0]
    for y in (0, 1, 2, 5):
        for tree, n_cand in ((False, 1), (True, 4)):
            d, od = _cos_case(pf, st, tokens, offs, keys, np.array([y], np.int32), q, 8, tree, n_cand)
            if (lens < 2).all() or y == 5:
                assert int(d["n_nodes"]) == 1 and od["n_found"] == 0


def test_paper_boundary_example_gpu(pf):
    A, B, C, D, E = 10, 11, 12, 13, 14
    tokens = np.array([A, B, C, D, E], np.int32)
    offs = np.array([0, 3, 5], np.int64)
    keys = synth.random_keys(5, 61)
    st = pf.pf_store_build(tokens, offs, 1)
    pf.pf_store_attach_keys(st, keys)
    d, _ = _cos_case(pf, st, tokens, offs, keys, np.array([B], np.int32), keys[1], 4, False, 1)
    assert list(d["token"][:int(d["n_nodes"])]) == [B, C]


def test_cosine_lookup_requires_keys(pf):
    import torch
    tokens = np.arange(10, dtype=np.int32)
    st = pf.pf_store_build(tokens, np.array([0, 10], np.int64), 1)
    c = pf.Context(tokens, 16)
    q = torch.zeros(256, dtype=torch.int8, device="cuda")
    with pytest.raises(pf.PfError) as e:
        pf.pf_draft_lookup_cosine(st, c, q, 4, False, 1, 64, pf.new_draft())
    assert e.value.status == -5


@pytest.mark.parametrize("name,layers", [("tiny", None), ("3b", 2)])
def test_verify_keys_against_oracle_states(pf, name, layers):
    """Keys of the verify step's final-layer states against keys of the
    oracle's states for the same rows (the states agree only to rounding):
    the key directions agree and most codes agree exactly."""
    import torch
    wl = synth.WORKLOADS[name]
    shape = wl.model if layers is None else wl.model.with_layers(layers)
    seed = synth.case_seed(wl, 2)
    w = synth.make_weights(shape, seed)
    prefix = min(wl.prefix, 512)
    kv_host = synth.make_kv_prefix(shape, seed, prefix)
    store = synth.make_store(wl, seed)
    ctx, _ = synth.make_context(wl, seed, store, hit=True)
    gpu = Gpu(shape, w, kv_host, prefix, ((prefix + 2 * 65 + 63) // 64) * 64)
    st = pf.pf_store_build(store.tokens, store.seq_offsets, wl.ngram)
    out = gpu.step(st, ctx, wl.k_max, commit=False)
    R = synth.key_projection(shape.hidden, 70)
    kp = pf.pf_keyproj_create(R)
    rows = out["rows"]
    kd = torch.zeros(rows, 256, dtype=torch.int8, device="cuda")
    qd = torch.zeros(256, dtype=torch.int8, device="cuda")
    pf.pf_verify_row_keys(gpu.model, kp, rows, kd)
    pf.pf_verify_query_key(gpu.model, kp, gpu.res, qd)
    torch.cuda.synchronize()
    got = kd.cpu().numpy()
    od = oracle.lookup(store.tokens, store.seq_offsets, wl.ngram, ctx, wl.k_max)
    ores = oracle.verify_batched(oracle.Model(shape, w), kv_host, od, rows, False, want_hidden=True)
    ref = oracle.key_encode(R.astype(np.float64), ores["hidden"])
    # a relative state difference e moves a code by about 127 * e. fp32
    # states agree to ~1e-7 (codes identical); bf16 states agree to ~0.5%
    # after two layers (the residual stream's rounding chaos), so about a
    # quarter of the codes move by a step or two while the key direction,
    # which is what the cosine ranking sees, stays the same
    diff = np.abs(got.astype(np.int32) - ref.astype(np.int32))
    gf, rf = got.astype(np.float64), ref.astype(np.float64)
    cos = (gf * rf).sum(1) / np.sqrt((gf * gf).sum(1) * (rf * rf).sum(1))
    print(f"[{name}] codes: max diff {diff.max()}, exact {(diff == 0).mean():.4f}, "
          f"min row cosine {cos.min():.6f}")
    assert diff.max() <= 3
    assert cos.min() > 0.999
    if shape.dtype == "f32":
        assert diff.max() == 0
    res = out["res"]
    q_row = int(res["path"][int(res["accept_len"])])
    assert (qd.cpu().numpy() == got[q_row]).all()
