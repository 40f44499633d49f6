"""Full-size parity at the benchmark's shapes and launch configuration: the
3B- and 7B-class bf16 decoders (every layer, the full vocabulary) and the 3B
tree draft, each compared with the oracle's batched verify on the same seeded
inputs. The oracle runs every layer on the host's cores (seconds to a minute)."""
import gc

import numpy as np
import pytest

import oracle
import synth
from pfharness import (Gpu, assert_same_draft, check_accept_against_oracle, rel_err_rows, splice,
                       tol_of)

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


@pytest.fixture(scope="module")
def pf():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_32166_amd as pf
    pf.lib()
    return pf


def _full_case(pf, name, splices):
    import torch
    wl = synth.WORKLOADS[name]
    shape = wl.model
    seed = synth.case_seed(wl, 0)
    print(f"[{name}] generating inputs", flush=True)
    w = synth.make_weights(shape, seed)
    kv_host = synth.make_kv_prefix(shape, seed, wl.prefix)
    om = oracle.Model(shape, w)
    base_store = synth.make_store(wl, seed)
    cap = ((wl.prefix + 2 * 65 + 63) // 64) * 64
    gpu = Gpu(shape, w, kv_host, wl.prefix, cap)
    tol = tol_of(shape)
    worst = 0.0
    try:
        for ci, j in enumerate(splices):
            cseed = synth.case_seed(wl, ci)
            ctx, _ = synth.make_context(wl, cseed, base_store, hit=True)
            store = base_store
            if j is not None:
                print(f"[{name}] oracle greedy continuation of {j}", flush=True)
                store, _ = splice(wl, om, kv_host, base_store, ctx, cseed, j)
            st = pf.pf_store_build(store.tokens, store.seq_offsets, wl.ngram)
            max_nodes = wl.max_nodes if wl.tree else 64
            print(f"[{name}] case {ci}: gpu step", flush=True)
            out = gpu.step(st, ctx, wl.k_max, tree=wl.tree, n_cand=wl.n_cand if wl.tree else 1,
                           max_nodes=max_nodes)
            od = oracle.lookup(store.tokens, store.seq_offsets, wl.ngram, ctx, wl.k_max,
                               n_cand=wl.n_cand if wl.tree else 1, tree=wl.tree,
                               max_nodes=wl.max_nodes)
            assert_same_draft(out["draft"], od, wl.tree)
            print(f"[{name}] case {ci}: oracle batched verify ({od['n_nodes']} nodes)", flush=True)
            ores = oracle.verify_batched(om, kv_host, od, out["rows"], wl.tree)
            n = od["n_nodes"]
            err = rel_err_rows(out["logits"][:n], ores["logits"][:n])
            worst = max(worst, float(err.max()))
            print(f"[{name}] case {ci}: max rel err {err.max():.3e}", flush=True)
            assert err.max() <= tol
            res = out["res"]
            for r in range(n):
                assert int(res["pred"][r]) == oracle.argmax(out["logits"][r])
            mine = oracle.accept(od, res["pred"][:out["rows"]], wl.tree)
            assert (int(res["accept_len"]), int(res["bonus"])) == (mine["accept_len"],
                                                                  mine["bonus"])
            check_accept_against_oracle(res, ores, ores["logits"], tol)
            kv = Gpu.to_np(out["kv_rows"])[:, :, :, :n, :]
            ref = ores["kv_new"][:, :, :, :n, :]
            e = np.abs(kv - ref).max(axis=(2, 3, 4)) / np.abs(ref).max(axis=(2, 3, 4))
            assert e.max() <= tol, e.max()
            assert out["kv_len"] == wl.prefix + int(res["accept_len"]) + 1
    finally:
        del gpu
        gc.collect()
        torch.cuda.empty_cache()
    return worst


def test_full_3b_linear(pf):
    _full_case(pf, "3b", [None, 8])


def test_full_3b_tree(pf):
    _full_case(pf, "3b_tree", [5])


def test_full_7b_linear(pf):
    _full_case(pf, "7b", [None])
