"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded inputs. Integer results (drafts, accept lengths, paths, KV
indices) must match exactly; logits within the dtype's tolerance (max over a
row of |gpu - ref| / max|ref| <= 1e-4 fp32, 2e-2 bf16), with acceptance
compared exactly wherever the oracle's top-2 margin clears the tolerance."""
import json
import os

import numpy as np
import pytest

import oracle
import synth
from pfharness import (Gpu, assert_same_draft, check_accept_against_oracle, clear_rows,
                       rel_err_rows, splice, tol_of)

pytestmark = pytest.mark.gpu

TINY = synth.WORKLOADS["tiny"]
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module")
def pf():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_32166_amd as pf
    pf.lib()
    return pf


# ----------------------------------------------------------------------------
# draft lookup: bit-exact against the exhaustive scan
# ----------------------------------------------------------------------------

def _gpu_lookup(pf, store, ctx, k_max, tree, n_cand, max_nodes):
    import torch
    st = pf.pf_store_build(store.tokens, store.seq_offsets, store_ngram[0])
    c = pf.Context(ctx, len(ctx) + 8)
    d = pf.new_draft()
    pf.pf_draft_lookup(st, c, k_max, tree, n_cand, max_nodes, d)
    torch.cuda.synchronize()
    return pf.read_draft(d)


store_ngram = [3]


def test_lookup_paper_boundary_example(pf):
    with open(os.path.join(GOLDEN, "paper_boundary_example.json")) as f:
        g = json.load(f)
    ids = g["tokens"]
    seqs = [[ids[t] for t in s] for s in g["sequences"]]
    store = synth.Store(np.array(sum(seqs, []), np.int32),
                        np.cumsum([0] + [len(s) for s in seqs]).astype(np.int64))
    store_ngram[0] = g["ngram"]
    for c in g["cases"]:
        ctx = np.array([ids[c["current"]]], np.int32)
        d = _gpu_lookup(pf, store, ctx, g["k_max"], False, 1, 64)
        assert list(d["token"][1:int(d["n_nodes"])]) == [ids[t] for t in c["draft"]]
        od = oracle.lookup(store.tokens, store.seq_offsets, g["ngram"], ctx, g["k_max"])
        assert_same_draft(d, od, False)


@pytest.mark.parametrize("seed", range(10))
def test_lookup_random_small_stores(pf, seed):
    rng = np.random.default_rng(500 + seed)
    vocab = 2 + seed % 4
    lens = rng.integers(1, 40, rng.integers(1, 30))
    store = synth.Store(rng.integers(0, vocab, lens.sum()).astype(np.int32),
                        np.concatenate([[0], np.cumsum(lens)]).astype(np.int64))
    for n in (1, 2, 3):
        store_ngram[0] = n
        for k_max in (0, 1, 5, 64):
            for tree, n_cand, max_nodes in ((False, 1, 64), (True, 4, 48), (True, 3, 5)):
                ctx = rng.integers(0, vocab, rng.integers(1, 6)).astype(np.int32)
                d = _gpu_lookup(pf, store, ctx, k_max, tree, n_cand, max_nodes)
                od = oracle.lookup(store.tokens, store.seq_offsets, n, ctx, k_max, n_cand=n_cand,
                                   tree=tree, max_nodes=max_nodes)
                assert_same_draft(d, od, tree)


@pytest.mark.parametrize("case", ["no_sequences", "only_empty", "shorter_than_n", "empty_between"])
def test_lookup_degenerate_stores(pf, case):
    """Stores with nothing to retrieve, or with empty sequences among real
    ones: drafts bit-exact vs the oracle; a store without an eligible entry
    gives the greedy step's draft (the current token alone)."""
    rng = np.random.default_rng(900)
    if case == "no_sequences":
        lens = np.zeros(0, np.int64)
    elif case == "only_empty":
        lens = np.zeros(5, np.int64)
    elif case == "shorter_than_n":
        lens = np.array([1, 2, 0, 2, 1], np.int64)
    else:
        lens = np.array([0, 9, 0, 0, 12, 0, 7, 0], np.int64)
    toks = rng.integers(0, 3, int(lens.sum())).astype(np.int32)
    store = synth.Store(toks, np.concatenate([[0], np.cumsum(lens)]).astype(np.int64))
    store_ngram[0] = 3
    for k_max in (0, 4, 64):
        for tree, n_cand, max_nodes in ((False, 1, 64), (True, 4, 48)):
            for ctx in (np.array([1], np.int32), np.array([0, 1, 2, 0, 1], np.int32),
                        toks[:5] if len(toks) >= 5 else np.array([2, 2, 2], np.int32)):
                d = _gpu_lookup(pf, store, ctx, k_max, tree, n_cand, max_nodes)
                od = oracle.lookup(store.tokens, store.seq_offsets, 3, ctx, k_max, n_cand=n_cand,
                                   tree=tree, max_nodes=max_nodes)
                assert_same_draft(d, od, tree)
                if case != "empty_between":
                    assert od["n_found"] == 0 and int(d["n_nodes"]) == 1


@pytest.mark.parametrize("name", ["tiny", "3b", "3b_tree", "7b"])
def test_lookup_workload_stores(pf, name):
    wl = synth.WORKLOADS[name]
    store = synth.make_store(wl, synth.case_seed(wl, 0))
    store_ngram[0] = wl.ngram
    st = pf.pf_store_build(store.tokens, store.seq_offsets, wl.ngram)
    import torch
    for c in range(12):
        ctx, info = synth.make_context(wl, synth.case_seed(wl, c), store, length=64)
        cc = pf.Context(ctx, 128)
        d = pf.new_draft()
        pf.pf_draft_lookup(st, cc, wl.k_max, wl.tree, wl.n_cand, wl.max_nodes if wl.tree else 64, d)
        torch.cuda.synchronize()
        dd = pf.read_draft(d)
        od = oracle.lookup(store.tokens, store.seq_offsets, wl.ngram, ctx, wl.k_max,
                           n_cand=wl.n_cand, tree=wl.tree, max_nodes=wl.max_nodes)
        assert_same_draft(dd, od, wl.tree)
        if info["hit"]:
            assert od["n_found"] >= 1


# ----------------------------------------------------------------------------
# verify + commit on the tiny fp32 decoder (64 cases, half spliced)
# ----------------------------------------------------------------------------

def _verify_case(pf, wl, shape, seed, j, tree=False, gpu=None, w=None, kv_host=None):
    w = w if w is not None else synth.make_weights(shape, seed)
    kv_host = kv_host if kv_host is not None else synth.make_kv_prefix(shape, seed, wl.prefix)
    om = oracle.Model(shape, w)
    store = synth.make_store(wl, seed)
    ctx, _ = synth.make_context(wl, seed, store, hit=True)
    g_cont = None
    if j is not None:
        store, g_cont = splice(wl, om, kv_host, store, ctx, seed, j)
    if gpu is None:
        cap = ((wl.prefix + 4 * 65 + 63) // 64) * 64
        gpu = Gpu(shape, w, kv_host, wl.prefix, cap)
    st = pf.pf_store_build(store.tokens, store.seq_offsets, wl.ngram)
    max_nodes = wl.max_nodes if tree else 64
    out = gpu.step(st, ctx, wl.k_max, tree=tree, n_cand=wl.n_cand if tree else 1,
                   max_nodes=max_nodes)
    od = oracle.lookup(store.tokens, store.seq_offsets, wl.ngram, ctx, wl.k_max,
                       n_cand=wl.n_cand if tree else 1, tree=tree, max_nodes=wl.max_nodes)
    assert_same_draft(out["draft"], od, tree)
    ores = oracle.verify_batched(om, kv_host, od, out["rows"], tree)
    return out, od, ores, gpu, g_cont


def _compare_step(out, od, ores, shape, P, tree=False):
    tol = tol_of(shape)
    n = od["n_nodes"]
    res = out["res"]
    lg = out["logits"]
    err = rel_err_rows(lg[:n], ores["logits"][:n])
    assert err.max() <= tol, (err.max(), tol)
    # the device's greedy choice is the argmax of its own logits
    for r in range(n):
        assert int(res["pred"][r]) == oracle.argmax(lg[r])
    # acceptance is a function of the device's own predictions
    mine = oracle.accept(od, res["pred"][:out["rows"]], tree)
    assert int(res["accept_len"]) == mine["accept_len"]
    assert int(res["bonus"]) == mine["bonus"]
    assert [int(x) for x in res["path"][:mine["accept_len"] + 1]] == mine["path"]
    assert int(res["kv_base"]) == P
    # and it matches the oracle wherever the margins are clear
    exact = check_accept_against_oracle(res, ores, ores["logits"], tol)
    # appended K/V of the real rows
    kv = Gpu.to_np(out["kv_rows"])[:, :, :, :n, :]
    ref = ores["kv_new"][:, :, :, :n, :]
    for l in range(shape.n_layers):
        for t in range(2):
            e = np.abs(kv[l, t] - ref[l, t]).max() / np.abs(ref[l, t]).max()
            assert e <= tol, (l, t, e)
    # commit: length and context
    L = int(res["accept_len"])
    assert out["kv_len"] == P + L + 1
    emitted = [int(x) for x in res["out_tokens"][:L + 1]]
    assert list(out["ctx_tokens"][-(L + 1):]) == emitted
    assert emitted[-1] == int(res["bonus"])
    return exact


@pytest.mark.parametrize("case", range(64))
def test_verify_tiny(pf, case):
    wl = TINY
    seed = synth.case_seed(wl, case)
    j = None if case % 2 == 0 else [0, 1, wl.k_max // 2, wl.k_max][(case // 2) % 4]
    out, od, ores, gpu, g = _verify_case(pf, wl, wl.model, seed, j)
    exact = _compare_step(out, od, ores, wl.model, wl.prefix)
    if j is not None and exact:
        assert ores["accept_len"] >= j
        assert int(out["res"]["accept_len"]) >= j


@pytest.mark.parametrize("case", range(8))
def test_verify_tiny_sequential_equivalence(pf, case):
    """The batched device verify gives what K sequential greedy decodes give."""
    wl = TINY
    seed = synth.case_seed(wl, 100 + case)
    j = [0, 2, 5, 8][case % 4]
    out, od, ores, gpu, g = _verify_case(pf, wl, wl.model, seed, j)
    sq = oracle.verify_sequential(oracle.Model(wl.model, synth.make_weights(wl.model, seed)),
                                  synth.make_kv_prefix(wl.model, seed, wl.prefix), od, False)
    res = out["res"]
    clear = clear_rows(ores["logits"], 1e-4)
    if all(clear[u] for u in sq["path"]):
        assert int(res["accept_len"]) == sq["accept_len"]
        assert int(res["bonus"]) == sq["bonus"]


TREE_TINY = synth.Workload("tiny_tree", 6, TINY.model, 512, 8, 1, True, 4, 24, 64, (128, 128),
                           "uniform", 8)


@pytest.mark.parametrize("case", range(12))
def test_verify_tiny_tree(pf, case):
    wl = TREE_TINY
    seed = synth.case_seed(wl, case)
    j = None if case % 3 == 0 else [1, 3, 8][case % 3]
    out, od, ores, gpu, g = _verify_case(pf, wl, wl.model, seed, j, tree=True)
    _compare_step_tree(out, od, ores, wl.model, wl.prefix)


def _compare_step_tree(out, od, ores, shape, P):
    tol = tol_of(shape)
    n = od["n_nodes"]
    res = out["res"]
    err = rel_err_rows(out["logits"][:n], ores["logits"][:n])
    assert err.max() <= tol
    mine = oracle.accept(od, res["pred"][:out["rows"]], True)
    assert (int(res["accept_len"]), int(res["bonus"])) == (mine["accept_len"], mine["bonus"])
    assert [int(x) for x in res["path"][:mine["accept_len"] + 1]] == mine["path"]
    check_accept_against_oracle(res, ores, ores["logits"], tol)
    L = int(res["accept_len"])
    assert out["kv_len"] == P + L + 1


@pytest.mark.parametrize("case", range(4))
def test_tree_commit_compacts_the_accepted_path(pf, case):
    wl = TREE_TINY
    seed = synth.case_seed(wl, 50 + case)
    out, od, ores, gpu, g = _verify_case(pf, wl, wl.model, seed, 3 + case, tree=True)
    res = out["res"]
    L = int(res["accept_len"])
    path = [int(x) for x in res["path"][:L + 1]]
    got = Gpu.to_np(gpu.export(wl.prefix, L + 1))
    before = Gpu.to_np(out["kv_rows"])
    want = before[:, :, :, path, :]
    assert np.array_equal(got, want)


# ----------------------------------------------------------------------------
# chained steps: lookup -> verify -> commit repeated equals greedy decoding
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("case", range(3))
def test_chained_steps_equal_greedy_decoding(pf, case):
    import torch
    wl = TINY
    seed = synth.case_seed(wl, 200 + case)
    shape = wl.model
    w = synth.make_weights(shape, seed)
    kv_host = synth.make_kv_prefix(shape, seed, wl.prefix)
    om = oracle.Model(shape, w)
    store = synth.make_store(wl, seed)
    ctx, _ = synth.make_context(wl, seed, store, hit=True)
    steps_tokens = 20
    greedy = oracle.greedy_decode(om, kv_host, int(ctx[-1]), steps_tokens)
    # make the store hold the greedy continuation in pieces so drafts hit
    gt = greedy["tokens"]
    store = store.append(np.concatenate([ctx[-3:], gt[:7]]))
    store = store.append(gt[4:16])
    gpu = Gpu(shape, w, kv_host, wl.prefix, ((wl.prefix + 20 * 9 + 63) // 64) * 64 + 64)
    st = pf.pf_store_build(store.tokens, store.seq_offsets, wl.ngram)
    c = pf.Context(ctx, len(ctx) + 400)
    rows = wl.k_max + 1
    emitted = []
    accepted = []
    for it in range(12):
        pf.pf_draft_lookup(st, c, wl.k_max, False, 1, 64, gpu.draft)
        pf.pf_verify_step(gpu.model, gpu.kv, gpu.draft, rows, False, None, gpu.res)
        pf.pf_kv_commit(gpu.kv, gpu.res, c)
        r = pf.read_result(gpu.res)
        accepted.append(int(r["accept_len"]))
        emitted += [int(x) for x in r["out_tokens"][:int(r["accept_len"]) + 1]]
        if len(emitted) >= steps_tokens:
            break
    torch.cuda.synchronize()
    n = min(len(emitted), steps_tokens)
    assert emitted[:n] == list(gt[:n])
    assert max(accepted) >= 2  # the retrieved continuation was used
    assert int(gpu.kv.len.item()) == wl.prefix + len(emitted)
    assert list(c.tokens()[len(ctx):]) == emitted


def _poison_past_len(gpu, torch):
    """Fill every cache slot at or past the committed length with NaN (keys
    and values are both [slot][head_dim] rows)."""
    s = gpu.shape
    n = int(gpu.kv.len.item())
    cap = gpu.kv.data.numel() // (s.n_layers * 2 * s.n_kv_heads * s.head_dim *
                                  (2 if s.dtype == "bf16" else 4))
    dt = torch.bfloat16 if s.dtype == "bf16" else torch.float32
    planes = gpu.kv.data.view(dt).view(s.n_layers, 2, s.n_kv_heads, cap * s.head_dim)
    planes[:, 0].view(s.n_layers, s.n_kv_heads, cap, s.head_dim)[:, :, n:, :] = float("nan")
    planes[:, 1].view(s.n_layers, s.n_kv_heads, cap, s.head_dim)[:, :, n:, :] = float("nan")


@pytest.mark.parametrize("shape_name,tree", [("tiny", False), ("tiny", True), ("ragged", False),
                                             ("ragged", True)])
def test_rejected_slots_poisoned_with_nan_do_not_leak(pf, shape_name, tree):
    """Rollback correctness: after every commit, one of two identical caches
    gets NaN in every slot past the committed length (the rejected drafts'
    K/V and everything beyond). Chained steps on both give bit-identical
    logits, accept decisions and committed K/V: no kernel reads a slot past
    the length it was given, not even as a zero-weighted value."""
    import torch
    wl = TINY if shape_name == "tiny" else RAGGED_WL
    shape = wl.model
    seed = synth.case_seed(wl, 300 + int(tree))
    w = synth.make_weights(shape, seed)
    kv_host = synth.make_kv_prefix(shape, seed, wl.prefix)
    om = oracle.Model(shape, w)
    store = synth.make_store(wl, seed)
    ctx, _ = synth.make_context(wl, seed, store, hit=True)
    greedy = oracle.greedy_decode(om, kv_host, int(ctx[-1]), 24)["tokens"]
    # the store holds pieces of the continuation (with a wrong token) so
    # drafts are partly accepted and partly rolled back
    g2 = greedy.copy()
    g2[9] = (g2[9] + 1) % shape.vocab
    store = store.append(np.concatenate([ctx[-3:], g2[:14]]))
    store = store.append(np.concatenate([g2[5:7], (g2[7:15] + 3) % shape.vocab]))
    cap = ((wl.prefix + 12 * 70 + 63) // 64) * 64 + 64
    a = Gpu(shape, w, kv_host, wl.prefix, cap)
    b = Gpu(shape, w, kv_host, wl.prefix, cap)
    st = pf.pf_store_build(store.tokens, store.seq_offsets, wl.ngram)
    ca, cb = pf.Context(ctx, len(ctx) + 1200), pf.Context(ctx, len(ctx) + 1200)
    rows = 49 if tree else wl.k_max + 1
    la = torch.zeros(rows, shape.vocab, device="cuda")
    lb = torch.zeros(rows, shape.vocab, device="cuda")
    rejected = 0
    for it in range(8):
        for g, c, lg in ((a, ca, la), (b, cb, lb)):
            pf.pf_draft_lookup(st, c, wl.k_max, tree, 4 if tree else 1, 48 if tree else 64, g.draft)
            pf.pf_verify_step(g.model, g.kv, g.draft, rows, tree, lg, g.res)
            pf.pf_kv_commit(g.kv, g.res, c)
        torch.cuda.synchronize()
        assert torch.equal(la, lb), it
        ra, rb = pf.read_result(a.res), pf.read_result(b.res)
        assert (ra["accept_len"], ra["bonus"]) == (rb["accept_len"], rb["bonus"])
        d = pf.read_draft(a.draft)
        rejected += int(d["n_nodes"]) - 1 - int(ra["accept_len"])
        _poison_past_len(b, torch)
    n = int(a.kv.len.item())
    assert n == int(b.kv.len.item())
    assert torch.equal(a.export(0, n), b.export(0, n))
    assert not torch.isnan(lb).any()
    assert rejected > 0, "no draft token was rolled back"


# ----------------------------------------------------------------------------
# bf16, several tiles and ragged tails
# ----------------------------------------------------------------------------

RAGGED = synth.ModelShape(2, 512, 8, 2, 128, 1360, 4000, 1e6, 1e-6, "bf16")
RAGGED_WL = synth.Workload("ragged", 7, RAGGED, 300, 16, 4, False, 1, 16, 200, (64, 256), "zipf", 0)


@pytest.mark.parametrize("case", range(6))
def test_verify_bf16_ragged(pf, case):
    wl = RAGGED_WL
    seed = synth.case_seed(wl, case)
    j = [None, 0, 4, 16, 1, None][case]
    out, od, ores, gpu, g = _verify_case(pf, wl, wl.model, seed, j)
    _compare_step(out, od, ores, wl.model, wl.prefix)


# Rows wider than the verify norm's eight 512-column slices: 4160 columns are
# eight slices of 520 (some threads take two four-column chunks), and the
# final norm's wide form runs past its 1024 threads.
WIDE = synth.ModelShape(2, 4160, 8, 2, 128, 1360, 4000, 1e6, 1e-6, "bf16")
WIDE_WL = synth.Workload("wide", 12, WIDE, 300, 16, 4, False, 1, 16, 200, (64, 256), "zipf", 0)


@pytest.mark.parametrize("case", range(2))
def test_verify_bf16_wide_rows(pf, case):
    wl = WIDE_WL
    seed = synth.case_seed(wl, case)
    out, od, ores, gpu, g = _verify_case(pf, wl, wl.model, seed, [None, 16][case])
    _compare_step(out, od, ores, wl.model, wl.prefix)


RAGGED_TREE = synth.Workload("ragged_tree", 8, RAGGED, 300, 16, 4, True, 4, 48, 200, (64, 256),
                             "zipf", 0)


@pytest.mark.parametrize("case", range(3))
def test_verify_bf16_ragged_tree(pf, case):
    wl = RAGGED_TREE
    seed = synth.case_seed(wl, case)
    out, od, ores, gpu, g = _verify_case(pf, wl, wl.model, seed, [None, 3, 9][case], tree=True)
    _compare_step_tree(out, od, ores, wl.model, wl.prefix)


@pytest.mark.parametrize("k_max", [0, 1, 31, 64])
def test_verify_draft_lengths(pf, k_max):
    """k_max from 0 (ordinary greedy pass) to the cap of 64 (65 rows)."""
    wl = synth.Workload("klen", 9, TINY.model, 200, k_max, 2, False, 1, k_max, 64, (100, 128),
                        "uniform", 0)
    seed = synth.case_seed(wl, k_max)
    out, od, ores, gpu, g = _verify_case(pf, wl, wl.model, seed, min(k_max, 5))
    _compare_step(out, od, ores, wl.model, wl.prefix)


def test_miss_and_short_context_are_greedy_steps(pf):
    import torch
    wl = TINY
    seed = synth.case_seed(wl, 300)
    w = synth.make_weights(wl.model, seed)
    kv_host = synth.make_kv_prefix(wl.model, seed, wl.prefix)
    om = oracle.Model(wl.model, w)
    store = synth.make_store(wl, seed)
    gpu = Gpu(wl.model, w, kv_host, wl.prefix, 1024)
    st = pf.pf_store_build(store.tokens, store.seq_offsets, wl.ngram)
    greedy = oracle.greedy_decode(om, kv_host, 77, 1)["tokens"][0]
    for ctx in (np.array([77], np.int32), np.array([5000 % 4096, 4095, 77], np.int32)):
        out = gpu.step(st, ctx, wl.k_max)
        assert int(out["draft"]["n_nodes"]) == 1
        assert int(out["res"]["accept_len"]) == 0
        assert int(out["res"]["bonus"]) == int(greedy)


def test_capacity_and_argument_errors(pf):
    import torch
    wl = TINY
    seed = synth.case_seed(wl, 301)
    w = synth.make_weights(wl.model, seed)
    kv_host = synth.make_kv_prefix(wl.model, seed, wl.prefix)
    gpu = Gpu(wl.model, w, kv_host, wl.prefix, 576)
    with pytest.raises(pf.PfError) as e:
        pf.pf_verify_step(gpu.model, gpu.kv, gpu.draft, 65, False, None, gpu.res)
    assert e.value.status == pf.PF_ECAPACITY
    with pytest.raises(pf.PfError) as e:
        pf.pf_verify_step(gpu.model, gpu.kv, gpu.draft, 66, False, None, gpu.res)
    assert e.value.status == pf.PF_EINVAL
    with pytest.raises(pf.PfError) as e:
        pf.pf_kv_commit(gpu.kv, gpu.res, None)
    assert e.value.status == pf.PF_ESTATE
    st = pf.pf_store_build(np.arange(10, dtype=np.int32), np.array([0, 10]), 2)
    c = pf.Context(np.array([1, 2], np.int32), 4)
    with pytest.raises(pf.PfError) as e:
        pf.pf_draft_lookup(st, c, 65, False, 1, 64, gpu.draft)
    assert e.value.status == pf.PF_EINVAL
    with pytest.raises(pf.PfError) as e:
        pf.pf_draft_lookup(st, c, 8, True, 5, 48, gpu.draft)
    assert e.value.status == pf.PF_EINVAL
    # a verify + commit whose context append cannot fit is refused on the host
    pf.pf_draft_lookup(st, c, 8, False, 1, 64, gpu.draft)
    pf.pf_verify_step(gpu.model, gpu.kv, gpu.draft, 9, False, None, gpu.res)
    with pytest.raises(pf.PfError) as e:
        pf.pf_kv_commit(gpu.kv, gpu.res, c)
    assert e.value.status == pf.PF_ECAPACITY
    torch.cuda.synchronize()


def test_graph_replay_matches_eager(pf):
    """The step captured into a HIP graph gives the eager step's results on
    every replay (with eager work and synchronisation between replays)."""
    import torch
    wl = TINY
    seed = synth.case_seed(wl, 400)
    w = synth.make_weights(wl.model, seed)
    kv_host = synth.make_kv_prefix(wl.model, seed, wl.prefix)
    om = oracle.Model(wl.model, w)
    store = synth.make_store(wl, seed)
    ctx, _ = synth.make_context(wl, seed, store, hit=True)
    store, _ = splice(wl, om, kv_host, store, ctx, seed, 5)
    gpu = Gpu(wl.model, w, kv_host, wl.prefix, 1024)
    st = pf.pf_store_build(store.tokens, store.seq_offsets, wl.ngram)
    c = pf.Context(ctx, len(ctx) + 64)
    logits = torch.zeros(wl.rows, wl.model.vocab, device="cuda")

    def step():
        pf.pf_kv_set_len(gpu.kv, wl.prefix)
        pf.pf_context_init(c, len(ctx))
        pf.pf_draft_lookup(st, c, wl.k_max, False, 1, 64, gpu.draft)
        pf.pf_verify_step(gpu.model, gpu.kv, gpu.draft, wl.rows, False, logits, gpu.res)
        pf.pf_kv_commit(gpu.kv, gpu.res, c)

    step()
    torch.cuda.synchronize()
    ref_res = pf.read_result(gpu.res).copy()
    ref_logits = logits.cpu().numpy().copy()
    ref_ctx = c.tokens().copy()
    assert int(ref_res["accept_len"]) >= 5
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    with torch.cuda.graph(graph):
        step()
    for rep in range(4):
        logits.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        r = pf.read_result(gpu.res)
        assert r.tobytes() == ref_res.tobytes(), rep
        assert np.array_equal(logits.cpu().numpy(), ref_logits), rep
        assert np.array_equal(c.tokens(), ref_ctx), rep
        assert int(gpu.kv.len.item()) == wl.prefix + int(ref_res["accept_len"]) + 1
