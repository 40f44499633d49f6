"""Prompt-prefix carryover prefill on the GPU against the oracle: the reused
prefix's KV stays, new tokens run through every layer in causal chunks, and
their K/V land after the prefix. Then a retrieval-drafted verify step runs on
the extended cache, as in the carry-forward workload."""
import gc

import numpy as np
import pytest

import oracle
import synth
from pfharness import Gpu, check_accept_against_oracle, rel_err_rows, tol_of

pytestmark = pytest.mark.gpu

RAGGED = synth.ModelShape(2, 512, 8, 2, 128, 1360, 4000, 1e6, 1e-6, "bf16")
# bf16 shapes outside the staged prefill attention (head_dim 128 with 4..8
# query heads per KV head): two heads per KV head, and head_dim 64
GROUP2 = synth.ModelShape(2, 512, 4, 2, 128, 1360, 4000, 1e6, 1e-6, "bf16")
HD64 = synth.ModelShape(2, 512, 8, 2, 64, 1360, 4000, 1e4, 1e-6, "bf16")
# ragged widths for the chunk-wide SwiGLU GEMM: hidden 528 is 17 k fragments
# of 32 (its last 64-k stage holds one), FFN 1392 is 87 gate tiles of 16
# columns (its last block of five holds two)
RAGGED_W = synth.ModelShape(2, 528, 8, 2, 128, 1392, 4000, 1e6, 1e-6, "bf16")


@pytest.fixture(scope="module")
def pf():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_32166_amd as pf
    pf.lib()
    return pf


def _to_storage(shape, kv64):
    """fp64 K/V values (already on the storage grid) -> storage format."""
    if shape.dtype == "bf16":
        import torch
        return torch.from_numpy(kv64.astype(np.float32)).to(torch.bfloat16).view(
            torch.int16).numpy().view(np.uint16)
    return kv64.astype(np.float32)


def _prefill_case(pf, shape, seed, P, n, chunk, cap_extra=128):
    import torch
    w = synth.make_weights(shape, seed)
    kv_host = synth.make_kv_prefix(shape, seed, P)
    toks = synth.make_prefill_tokens(synth.Workload("p", 10, shape, P, 16, 4, False, 1, 16, 1,
                                                    (8, 8), "zipf", 0), seed, n)
    cap = ((P + n + cap_extra + 63) // 64) * 64
    gpu = Gpu(shape, w, kv_host, P, cap)
    tdev = torch.from_numpy(toks.astype(np.int32)).cuda()
    logits = torch.zeros(shape.vocab, device="cuda")
    pf.pf_prefill(gpu.model, gpu.kv, tdev, n, chunk, logits)
    torch.cuda.synchronize()
    assert int(gpu.kv.len.item()) == P + n
    kv_new = Gpu.to_np(gpu.export(P, n))
    return w, kv_host, toks, gpu, kv_new, logits.cpu().numpy()


@pytest.mark.parametrize("shape,P,n,chunk", [
    (RAGGED, 300, 200, 64),
    (RAGGED, 130, 77, 77),
    (synth.WORKLOADS["tiny"].model, 512, 100, 32),
    (GROUP2, 200, 150, 64),
    (HD64, 200, 150, 64),
    (RAGGED, 100, 5, 1),
    (RAGGED_W, 150, 130, 130),
    (RAGGED, 100, 600, 600),
], ids=["bf16_chunks", "bf16_one_chunk", "f32_chunks", "bf16_group2", "bf16_hd64",
        "bf16_single_rows", "bf16_ragged_widths", "bf16_chunk_over_512_rows"])
def test_prefill_matches_oracle(pf, shape, P, n, chunk):
    seed = 4242 + n
    w, kv_host, toks, gpu, kv_new, logits = _prefill_case(pf, shape, seed, P, n, chunk)
    om = oracle.Model(shape, w)
    ref = oracle.prefill(om, kv_host, toks, chunk)
    tol = tol_of(shape)
    r = ref["kv_new"]
    e = np.abs(kv_new - r).max(axis=(2, 3, 4)) / np.abs(r).max(axis=(2, 3, 4))
    assert e.max() <= tol, e
    err = rel_err_rows(logits[None, :], ref["logits_last"][None, :])
    assert err.max() <= tol, err
    del gpu
    gc.collect()


def test_prefill_chunk_size_invariance(pf):
    """Chunking is an implementation choice: results agree across chunk sizes."""
    shape = RAGGED
    _, _, _, g1, kv1, lg1 = _prefill_case(pf, shape, 77, 200, 150, 150)
    del g1
    _, _, _, g2, kv2, lg2 = _prefill_case(pf, shape, 77, 200, 150, 40)
    del g2
    e = np.abs(kv1 - kv2).max() / np.abs(kv1).max()
    assert e <= 1e-2, e
    assert np.argmax(lg1) == np.argmax(lg2) or rel_err_rows(lg1[None], lg2[None]).max() < 1e-2


def test_verify_after_prefill(pf):
    """Carry-forward: reused prefix + prefilled chunk, then a verify step on the
    extended cache; compared with the oracle's verify over the oracle's own
    prefill of the same tokens."""
    import torch
    shape = RAGGED
    P, n = 256, 96
    w, kv_host, toks, gpu, kv_new, _ = _prefill_case(pf, shape, 99, P, n, 32, cap_extra=192)
    om = oracle.Model(shape, w)
    ref = oracle.prefill(om, kv_host, toks, 32)
    kv_ext = np.concatenate([kv_host, _to_storage(shape, ref["kv_new"])], axis=3)
    wl = synth.Workload("carry", 11, shape, P + n, 16, 4, False, 1, 16, 100, (64, 128), "zipf", 0)
    store = synth.make_store(wl, 99)
    ctx, _ = synth.make_context(wl, 99, store, hit=True)
    st = pf.pf_store_build(store.tokens, store.seq_offsets, wl.ngram)
    gpu.prefix = P + n  # the cache now holds the prefilled rows
    out = gpu.step(st, ctx, wl.k_max)
    od = oracle.lookup(store.tokens, store.seq_offsets, wl.ngram, ctx, wl.k_max)
    ores = oracle.verify_batched(om, kv_ext, od, out["rows"], False)
    nn = od["n_nodes"]
    err = rel_err_rows(out["logits"][:nn], ores["logits"][:nn])
    assert err.max() <= tol_of(shape), err
    assert out["kv_len"] == P + n + int(out["res"]["accept_len"]) + 1


def test_prefill_3b_widths_two_layers(pf):
    """3B-class widths (8 query heads per KV head, the widest group of the
    staged prefill attention) at 2 layers: a 1000-token prefix, 300 new
    tokens in 128-row chunks (the last one 44 rows)."""
    wl = synth.WORKLOADS["3b"]
    shape = wl.model.with_layers(2)
    w, kv_host, toks, gpu, kv_new, logits = _prefill_case(pf, shape, synth.case_seed(wl, 5), 1000,
                                                          300, 128)
    om = oracle.Model(shape, w)
    ref = oracle.prefill(om, kv_host, toks, 128)
    r = ref["kv_new"]
    e = np.abs(kv_new - r).max(axis=(2, 3, 4)) / np.abs(r).max(axis=(2, 3, 4))
    assert e.max() <= tol_of(shape), e
    assert rel_err_rows(logits[None], ref["logits_last"][None]).max() <= tol_of(shape)
    del gpu
    gc.collect()


@pytest.mark.slow
def test_carry_forward_7b_widths_two_layers(pf):
    """The carry-forward workload at 7B-class widths and lengths, 2 layers (so
    the oracle finishes in about a minute): 6144 reused positions, 2048 new
    tokens prefilled in 512-row chunks, then a K=16 retrieval-drafted verify
    step on the cache the prefill left (8192 positions), compared with the
    oracle's verify over the oracle's own prefill of the same tokens
    (Section 3.4, prompt-prefix KV-state carryover; Section 3.2, single-pass
    verification)."""
    wl = synth.WORKLOADS["7b_carry"]
    shape = wl.model.with_layers(2)
    seed = synth.case_seed(wl, 0)
    w, kv_host, toks, gpu, kv_new, logits = _prefill_case(
        pf, shape, seed, wl.prefill_reuse, wl.prefill_new, wl.prefill_chunk)
    om = oracle.Model(shape, w)
    ref = oracle.prefill(om, kv_host, toks, wl.prefill_new)
    r = ref["kv_new"]
    e = np.abs(kv_new - r).max(axis=(2, 3, 4)) / np.abs(r).max(axis=(2, 3, 4))
    print(f"prefill: K/V max rel err {e.max():.3e}", flush=True)
    assert e.max() <= tol_of(shape), e
    assert rel_err_rows(logits[None], ref["logits_last"][None]).max() <= tol_of(shape)
    # the verify step on the prefilled cache
    P = wl.prefill_reuse + wl.prefill_new
    kv_ext = np.concatenate([kv_host, _to_storage(shape, r)], axis=3)
    store = synth.make_store(wl, seed)
    ctx, _ = synth.make_context(wl, seed, store, hit=True)
    st = pf.pf_store_build(store.tokens, store.seq_offsets, wl.ngram)
    gpu.prefix = P
    out = gpu.step(st, ctx, wl.k_max)
    od = oracle.lookup(store.tokens, store.seq_offsets, wl.ngram, ctx, wl.k_max)
    assert out["rows"] == wl.k_max + 1
    ores = oracle.verify_batched(om, kv_ext, od, out["rows"], False)
    nn = od["n_nodes"]
    err = rel_err_rows(out["logits"][:nn], ores["logits"][:nn])
    kvv = Gpu.to_np(out["kv_rows"])[:, :, :, :nn, :]
    kref = ores["kv_new"][:, :, :, :nn, :]
    ekv = np.abs(kvv - kref).max(axis=(2, 3, 4)) / np.abs(kref).max(axis=(2, 3, 4))
    print(f"verify after prefill ({nn} nodes): logits max rel err {err.max():.3e}, K/V "
          f"{ekv.max():.3e}, accept {int(out['res']['accept_len'])}", flush=True)
    assert err.max() <= tol_of(shape), err
    assert ekv.max() <= tol_of(shape), ekv
    check_accept_against_oracle(out["res"], ores, ores["logits"], tol_of(shape))
    assert out["kv_len"] == P + int(out["res"]["accept_len"]) + 1
    del gpu
    gc.collect()
