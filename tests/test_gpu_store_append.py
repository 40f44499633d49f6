"""GPU parity of the online memory update (Section 3.2, step 6) and the
decoding-memory budget (Section 5.6): appended output sequences are ranked
by the cosine lookup exactly like built ones (drafts bit-exact against the
oracle's exhaustive lookup over the same sequences and against a store
built from scratch); compaction keeps the sequences in order and evicts the
oldest first; a decoding loop that appends every iteration's tokens with the
keys of the states that produced them retrieves its own earlier outputs."""
import numpy as np
import pytest

import oracle
import synth
from pfharness import assert_same_draft

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pf():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_32166_amd as pf
    pf.lib()
    return pf


class Mirror:
    """Host view of a store's sequences (built, then appended) for the oracle."""

    def __init__(self, tokens, offs, keys):
        self.seqs = [(tokens[offs[i]:offs[i + 1]].copy(), keys[offs[i]:offs[i + 1]].copy())
                     for i in range(len(offs) - 1)]
        self.T = int(offs[-1])
        self.log = []          # appended sequences as [tokens list, keys list]

    def begin(self):
        self.log.append([[], []])

    def append(self, toks, keys):
        self.log[-1][0].extend(int(t) for t in toks)
        self.log[-1][1].extend(np.asarray(keys, np.int8))

    def arrays(self, drop=0):
        parts = self.seqs + [(np.array(t, np.int32), np.array(k, np.int8).reshape(-1, 256))
                             for t, k in self.log]
        parts = [p for p in parts if len(p[0])][drop:]
        tok = np.concatenate([p[0] for p in parts]).astype(np.int32)
        keys = np.concatenate([p[1] for p in parts]).astype(np.int8)
        offs = np.cumsum([0] + [len(p[0]) for p in parts]).astype(np.int64)
        return tok, offs, keys


def _lookup(pf, st, y, q, k_max, tree, n_cand):
    import torch
    c = pf.Context(np.array([3, y], np.int32), 8)
    qd = torch.from_numpy(np.ascontiguousarray(q, np.int8)).cuda()
    d = pf.new_draft()
    pf.pf_draft_lookup_cosine(st, c, qd, k_max, tree, n_cand, 63 if tree else 64, d)
    torch.cuda.synchronize()
    return pf.read_draft(d)


def _compare(pf, st, mirror, rng, n_queries=12, drop=0, extra=None):
    tok, offs, keys = mirror.arrays(drop)
    for case in range(n_queries):
        p = int(rng.integers(0, len(tok)))
        y = int(tok[p])
        q = synth.perturb_key(keys[p], 500 + case) if case % 2 else synth.random_keys(1, 600 + case)[0]
        tree = case % 3 == 2
        n_cand = 3 if tree else 1
        k_max = [8, 16, 64][case % 3]
        d = _lookup(pf, st, y, q, k_max, tree, n_cand)
        od = oracle.cos_lookup(tok, offs, keys, y, q, k_max, n_cand=n_cand, tree=tree, max_nodes=63)
        assert_same_draft(d, od, tree)
        if extra is not None:
            assert_same_draft(_lookup(pf, extra, y, q, k_max, tree, n_cand), od, tree)


def _dev(x, dtype):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype)).cuda()


def test_appends_rank_like_built_sequences(pf):
    import torch
    rng = np.random.default_rng(1)
    T, V = 3000, 20
    tok = rng.integers(0, V, T).astype(np.int32)
    cuts = np.sort(rng.choice(np.arange(1, T), 49, replace=False))
    offs = np.concatenate([[0], cuts, [T]]).astype(np.int64)
    keys = synth.random_keys(T, 2)
    st = pf.pf_store_build(tok, offs, 2)
    pf.pf_store_attach_keys(st, keys)
    pf.pf_store_reserve(st, 2000, 8)
    mirror = Mirror(tok, offs, keys)
    # nothing appended yet: the built store
    _compare(pf, st, mirror, rng, 6)
    batches = [("begin",), (37,), (1,), (0,), ("begin",), (50,), ("begin",), ("begin",), (12,),
               (64,)]
    for b in batches:
        if b[0] == "begin":
            pf.pf_store_begin_sequence(st)
            mirror.begin()
            continue
        n = b[0]
        t = rng.integers(0, V, max(n, 1)).astype(np.int32)
        k = synth.random_keys(max(n, 1), int(rng.integers(1 << 20)))
        # near copies of earlier keys so that appended entries win some queries
        for i in range(max(n, 1) // 2):
            k[i] = synth.perturb_key(keys[int(rng.integers(0, T))], 7 + i)
        pf.pf_store_append(st, _dev(t, np.int32), _dev(k, np.int8), _dev([n], np.int32), 64)
        mirror.append(t[:n], k[:n])
        ft, fo, fk = mirror.arrays()
        fresh = pf.pf_store_build(ft, fo, 2)
        pf.pf_store_attach_keys(fresh, fk)
        _compare(pf, st, mirror, rng, 8, extra=fresh)
    assert pf.pf_store_appended(st) == 37 + 1 + 50 + 12 + 64
    # compaction without a budget keeps every sequence at its position
    pf.pf_store_compact(st, 0)
    assert pf.pf_store_size(st) == T + 164
    _compare(pf, st, mirror, rng, 8)
    # with a budget the oldest sequences go first
    budget = 2500
    pf.pf_store_compact(st, budget)
    lens = [len(s[0]) for s in mirror.seqs] + [len(t) for t, _ in mirror.log if len(t)]
    drop, total = 0, sum(lens)
    while total > budget:
        total -= lens[drop]
        drop += 1
    assert pf.pf_store_size(st) == total
    _compare(pf, st, mirror, rng, 10, drop=drop)
    # the rebuilt store has an empty append region again
    with pytest.raises(pf.PfError) as e:
        pf.pf_store_append(st, _dev([1], np.int32), _dev(keys[:1], np.int8), _dev([1], np.int32), 1)
    assert e.value.status == -5
    pf.pf_store_begin_sequence(st)
    pf.pf_store_append(st, _dev([5, 6], np.int32), _dev(keys[:2], np.int8), _dev([2], np.int32), 2)
    assert pf.pf_store_appended(st) == 2


def test_append_errors(pf):
    rng = np.random.default_rng(3)
    tok = rng.integers(0, 5, 100).astype(np.int32)
    offs = np.array([0, 100], np.int64)
    keys = synth.random_keys(100, 4)
    st = pf.pf_store_build(tok, offs, 1)
    with pytest.raises(pf.PfError) as e:           # keys first
        pf.pf_store_reserve(st, 10, 2)
    assert e.value.status == -5
    pf.pf_store_attach_keys(st, keys)
    pf.pf_store_reserve(st, 10, 2)
    t, k = _dev(tok[:8], np.int32), _dev(keys[:8], np.int8)
    with pytest.raises(pf.PfError) as e:           # no open sequence
        pf.pf_store_append(st, t, k, _dev([4], np.int32), 4)
    assert e.value.status == -5
    pf.pf_store_begin_sequence(st)
    pf.pf_store_append(st, t, k, _dev([8], np.int32), 8)
    with pytest.raises(pf.PfError) as e:           # capacity (host bound)
        pf.pf_store_append(st, t, k, _dev([1], np.int32), 8)
    assert e.value.status == -4
    pf.pf_store_begin_sequence(st)
    with pytest.raises(pf.PfError) as e:           # sequence table
        pf.pf_store_begin_sequence(st)
    assert e.value.status == -4
    with pytest.raises(pf.PfError) as e:           # keys cannot be replaced now
        pf.pf_store_attach_keys(st, keys)
    assert e.value.status == -5


def test_decoding_appends_its_own_outputs(pf):
    """Tiny fp32 model, greedy decoding with the memory update on: every
    iteration's tokens land in the open sequence with the keys of the states
    that produced them (equal to the oracle's keys of its own states, fp32),
    so a query with the oracle's key of an output token's context finds that
    token's entry, and a second decode of the same task accepts proposals
    from the first."""
    import torch
    wl = synth.WORKLOADS["tiny"]
    shape = wl.model
    seed = synth.case_seed(wl, 60)
    w = synth.make_weights(shape, seed)
    kv_host = synth.make_kv_prefix(shape, seed, wl.prefix)
    store = synth.make_store(wl, seed)
    ctx, _ = synth.make_context(wl, seed, store, hit=False)
    G = 40
    om = oracle.Model(shape, w)
    g = oracle.greedy_decode(om, kv_host, int(ctx[-1]), G + 70, want_hidden=True)
    R = synth.key_projection(shape.hidden, seed)
    okeys = oracle.key_encode(R.astype(np.float64), g["hidden"])
    low = np.nonzero(g["margin"] <= 1e-4)[0]
    n_cmp = int(low[0]) if len(low) else G
    assert n_cmp >= 16

    model = pf.pf_model_create(pf.model_config(shape), pf.weights_to_device(w, shape.dtype))
    P = wl.prefix
    kv = pf.KVCache(model, ((P + 3 * G + 200) // 64) * 64)
    base_keys = synth.random_keys(len(store.tokens), seed)
    st = pf.pf_store_build(store.tokens, store.seq_offsets, wl.ngram)
    pf.pf_store_attach_keys(st, base_keys)
    pf.pf_store_reserve(st, 4 * G + 200, 4)
    kp = pf.pf_keyproj_create(R)
    q = torch.zeros(pf.KEY_DIM, dtype=torch.int8, device="cuda")
    draft, res = pf.new_draft(), pf.new_result()

    def run(l_fixed):
        pf.pf_kv_import(kv, pf.array_to_device(kv_host), P)
        c = pf.Context(ctx, len(ctx) + G + 140)
        q.zero_()
        pf.pf_store_begin_sequence(st)
        its, produced = [], 0
        while produced < G:
            it = pf.pf_decode_iteration(model, kv, c, st, kp, None, l_fixed, q, draft, res,
                                        append=True)
            its.append(it)
            produced += it["accepted"] + 1
        torch.cuda.synchronize()
        return c.tokens()[len(ctx):], its, produced

    out1, its1, n1 = run(0)                  # greedy: builds the memory online
    m1 = min(n_cmp, len(out1))
    assert (out1[:m1] == g["tokens"][:m1]).all()
    assert pf.pf_store_appended(st) == n1
    T = len(store.tokens)
    # appended entry j (token out1[j], key of the state that produced it)
    for j in range(0, m1 - 1, 5):
        d = _lookup(pf, st, int(out1[j]), okeys[j], 8, False, 1)
        assert int(d["cand_pos"][0]) == T + j, (j, d["cand_pos"][0], d["cand_score"][0])
        assert d["cand_score"][0] > 0.999
    out2, its2, n2 = run(16)                 # the same task again, from memory
    m = min(n_cmp, len(out2))
    assert (out2[:m] == g["tokens"][:m]).all()
    assert sum(it["accepted"] for it in its2) >= G // 2, [it["accepted"] for it in its2]
    assert pf.pf_store_appended(st) == n1 + n2
