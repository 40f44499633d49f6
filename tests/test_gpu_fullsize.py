"""Full-size parity at the benchmark's shapes and launch configuration: the
3B- and 7B-class bf16 decoders and the 3B tree draft, compared with the
oracle on the same seeded inputs (Section 3.2, "Single-pass token
verification"; the decoder and workload readings).

Eight cases per workload (four seeded queries and four drafts spliced with
the oracle's own greedy continuation of length 0, 1, K/2 and K), each run
twice at the benchmark's widths, vocabulary, prefix length and rows:

* two layers: logits, appended K/V and acceptance against the oracle's
  batched verify at the fixed 2e-2 bound;
* every layer, driven layer by layer: the device returns its residual stream
  after every layer (pf_verify_step_trace); the oracle runs layer l from the
  device's own input of layer l, and the device's output of that layer, its
  appended K/V, and the logits of its final stream must match at the fixed
  2e-2 bound. Greedy choices and acceptance are compared where the top-2
  margin clears that bound.

The network is chaotic at the bf16 rounding scale (one bf16 ulp on one input
element moves the oracle's own 36-layer logits by ~3%), so two valid bf16
computations of all layers in a row differ by about that much end to end;
that end-to-end figure is printed for the first case of each workload, and
the per-layer comparison is the one held to 2e-2."""
import gc

import numpy as np
import pytest

import oracle
import synth
from pfharness import Gpu, assert_same_draft, check_accept_against_oracle, rel_err_rows

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

TOL = 2e-2


@pytest.fixture(scope="module")
def pf():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_32166_amd as pf
    pf.lib()
    return pf


def _cases(wl):
    """(case index, splice length or None) of the eight cases; the spliced
    cases share one query and one greedy continuation."""
    K = wl.k_max
    return [(0, None), (1, None), (2, None), (3, None), (4, 0), (4, 1), (4, K // 2), (4, K)]


def _store_for(wl, om, kv_host, base_store, ctx, cseed, j, cont):
    if j is None:
        return base_store
    g = cont[:j]
    seq = synth.splice_sequence(wl, cseed, ctx[-wl.ngram:], g, wl.k_max + 2)
    return base_store.append(seq)


def _inputs(name, layers):
    wl = synth.WORKLOADS[name]
    shape = wl.model if layers is None else wl.model.with_layers(layers)
    seed = synth.case_seed(wl, 0)
    print(f"[{name}] generating inputs ({shape.n_layers} layers)", flush=True)
    w = synth.make_weights(shape, seed)
    kv_host = synth.make_kv_prefix(shape, seed, wl.prefix)
    return wl, shape, w, kv_host


def _continuation(wl, om, kv_host, ctx, layers_note):
    print(f"[{wl.name}] oracle greedy continuation of {wl.k_max} ({layers_note})", flush=True)
    return oracle.greedy_decode(om, kv_host, int(ctx[-1]), wl.k_max)["tokens"]


def _run_cases(pf, name, layers):
    import torch
    wl, shape, w, kv_host = _inputs(name, layers)
    om = oracle.Model(shape, w)
    base_store = synth.make_store(wl, synth.case_seed(wl, 0))
    cap = ((wl.prefix + 2 * 65 + 63) // 64) * 64
    gpu = Gpu(shape, w, kv_host, wl.prefix, cap)
    n_cand = wl.n_cand if wl.tree else 1
    max_nodes = wl.max_nodes if wl.tree else 64
    rows = (max_nodes + 1) if wl.tree else (wl.k_max + 1)
    cont = None
    accepted = []
    try:
        for ci, j in _cases(wl):
            cseed = synth.case_seed(wl, ci)
            ctx, _ = synth.make_context(wl, cseed, base_store, hit=True)
            if j is not None and cont is None:
                cont = _continuation(wl, om, kv_host, ctx,
                                     "full depth" if layers is None else f"{layers} layers")
            store = _store_for(wl, om, kv_host, base_store, ctx, cseed, j, cont)
            st = pf.pf_store_build(store.tokens, store.seq_offsets, wl.ngram)
            od = oracle.lookup(store.tokens, store.seq_offsets, wl.ngram, ctx, wl.k_max,
                               n_cand=n_cand, tree=wl.tree, max_nodes=wl.max_nodes)
            tag = f"[{name} {'L=' + str(layers) if layers else 'full'} case {ci} splice {j}]"
            if layers is not None:
                out = gpu.step(st, ctx, wl.k_max, tree=wl.tree, n_cand=n_cand,
                               max_nodes=max_nodes, rows=rows)
                assert_same_draft(out["draft"], od, wl.tree)
                _check_batched(tag, wl, out, om, kv_host, od, rows)
            else:
                out = _traced_step(pf, gpu, st, ctx, wl, n_cand, max_nodes, rows)
                assert_same_draft(out["draft"], od, wl.tree)
                _check_layerwise(tag, wl, shape, out, om, kv_host, od, rows, ci == 0)
            accepted.append(int(out["res"]["accept_len"]))
            del st
    finally:
        del gpu
        gc.collect()
        torch.cuda.empty_cache()
    print(f"[{name}] accept lengths {accepted}", flush=True)
    return accepted


def _check_common(out, od, rows, tree):
    """Device-internal consistency: greedy choices from its own logits and
    acceptance from its own choices (exact)."""
    res = out["res"]
    n = od["n_nodes"]
    for r in range(n):
        assert int(res["pred"][r]) == oracle.argmax(out["logits"][r])
    mine = oracle.accept(od, res["pred"][:rows], tree)
    assert (int(res["accept_len"]), int(res["bonus"])) == (mine["accept_len"], mine["bonus"])


def _check_batched(tag, wl, out, om, kv_host, od, rows):
    _check_common(out, od, rows, wl.tree)
    ores = oracle.verify_batched(om, kv_host, od, rows, wl.tree)
    n = od["n_nodes"]
    err = rel_err_rows(out["logits"][:n], ores["logits"][:n])
    kv = Gpu.to_np(out["kv_rows"])[:, :, :, :n, :]
    ref = ores["kv_new"][:, :, :, :n, :]
    ekv = np.abs(kv - ref).max(axis=(2, 3, 4)) / np.abs(ref).max(axis=(2, 3, 4))
    print(f"{tag} logits max rel err {err.max():.3e}, K/V {ekv.max():.3e}, accept "
          f"{int(out['res']['accept_len'])} (oracle {ores['accept_len']})", flush=True)
    assert err.max() <= TOL
    assert ekv.max() <= TOL
    check_accept_against_oracle(out["res"], ores, ores["logits"], TOL)
    assert out["kv_len"] == wl.prefix + int(out["res"]["accept_len"]) + 1


def _traced_step(pf, gpu, st, ctx_tokens, wl, n_cand, max_nodes, rows):
    import torch
    s = gpu.shape
    gpu.reset()
    ctx = pf.Context(ctx_tokens, len(ctx_tokens) + 4 * 65)
    logits = torch.zeros(rows, s.vocab, device="cuda")
    resid = torch.zeros(s.n_layers + 1, rows, s.hidden, device="cuda")
    pf.pf_draft_lookup(st, ctx, wl.k_max, wl.tree, n_cand, max_nodes, gpu.draft)
    pf.pf_verify_step_trace(gpu.model, gpu.kv, gpu.draft, rows, wl.tree, logits, gpu.res, resid)
    kv_rows = gpu.export(gpu.prefix, rows)
    pf.pf_kv_commit(gpu.kv, gpu.res, ctx)
    torch.cuda.synchronize()
    return {"draft": pf.read_draft(gpu.draft), "res": pf.read_result(gpu.res),
            "logits": logits.cpu().numpy(), "resid": resid.cpu().numpy().astype(np.float64),
            "kv_rows": Gpu.to_np(kv_rows), "kv_len": int(gpu.kv.len.item())}


def _check_layerwise(tag, wl, shape, out, om, kv_host, od, rows, end_to_end):
    _check_common(out, od, rows, wl.tree)
    tok, dep = oracle.draft_rows(od, rows, wl.tree)
    pos = wl.prefix + dep
    vis = oracle.visibility(od, rows, wl.tree)
    resid = out["resid"]
    # the embeddings are copied rows of the embedding table
    emb = synth_rows(om, tok)
    assert np.array_equal(resid[0], emb)
    worst_x, worst_d, worst_kv = 0.0, 0.0, 0.0
    for l in range(shape.n_layers):
        x_ref, kv_ref = om.layer(l, kv_host, resid[l], pos, vis, want_kv=True)
        e_x = rel_err_rows(resid[l + 1], x_ref).max()
        d_ref = x_ref - resid[l]
        e_d = rel_err_rows(resid[l + 1] - resid[l], d_ref).max()
        kv_dev = out["kv_rows"][l]
        e_kv = (np.abs(kv_dev - kv_ref).max(axis=(1, 2, 3)) / np.abs(kv_ref).max(axis=(1, 2, 3))).max()
        worst_x, worst_d, worst_kv = max(worst_x, e_x), max(worst_d, e_d), max(worst_kv, e_kv)
        assert e_x <= TOL, (l, e_x)
        assert e_kv <= TOL, (l, e_kv)
    lg_ref = om.head(resid[shape.n_layers])
    n = od["n_nodes"]
    e_lg = rel_err_rows(out["logits"][:n], lg_ref[:n]).max()
    print(f"{tag} per layer: stream {worst_x:.3e}, layer update {worst_d:.3e}, K/V "
          f"{worst_kv:.3e}; logits of the final stream {e_lg:.3e}; accept "
          f"{int(out['res']['accept_len'])}", flush=True)
    assert e_lg <= TOL
    # greedy choices where the oracle's margin on the device's final stream is clear
    pred_ref = np.array([oracle.argmax(lg_ref[r]) for r in range(rows)], np.int32)
    ref = oracle.accept(od, pred_ref, wl.tree)
    ref.update(pred=pred_ref)
    check_accept_against_oracle(out["res"], ref, lg_ref, TOL)
    assert out["kv_len"] == wl.prefix + int(out["res"]["accept_len"]) + 1
    if end_to_end:
        ores = oracle.verify_batched(om, kv_host, od, rows, wl.tree)
        e2e = rel_err_rows(out["logits"][:n], ores["logits"][:n]).max()
        print(f"{tag} end to end over all layers: logits max rel err {e2e:.3e} "
              f"(per-layer bound {TOL}; chaotic growth, see module notes)", flush=True)


def synth_rows(om, tok):
    e = om.w["embed"]
    if e.dtype == np.uint16:
        import torch
        t = torch.from_numpy(e[np.asarray(tok)].view(np.int16)).view(torch.bfloat16)
        return t.to(torch.float64).numpy()
    return e[np.asarray(tok)].astype(np.float64)


@pytest.mark.parametrize("name", ["3b", "7b", "3b_tree"])
def test_full_width_two_layers(pf, name):
    """Full widths, vocabulary and prefix, 2 layers: eight cases at 2e-2."""
    acc = _run_cases(pf, name, layers=2)
    assert max(acc) > 0   # the spliced drafts exercise partial acceptance


@pytest.mark.parametrize("name", ["3b", "7b", "3b_tree"])
def test_full_depth_layer_by_layer(pf, name):
    """Every layer at full size: eight cases, each layer at 2e-2 from the
    device's own layer input."""
    _run_cases(pf, name, layers=None)
