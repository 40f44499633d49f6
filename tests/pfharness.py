"""Shared set-up for the GPU parity tests: the same seeded inputs go to the
HIP library (through the C ABI) and to the CPU oracle, and the results are
compared element by element."""
from __future__ import annotations

import functools
from typing import Optional

import numpy as np

import oracle
import synth

TOL = {"f32": 1e-4, "bf16": 2e-2}


def tol_of(shape) -> float:
    return TOL[shape.dtype]


@functools.lru_cache(maxsize=2)
def weights(shape, seed):
    return synth.make_weights(shape, seed)


@functools.lru_cache(maxsize=2)
def kv_prefix(shape, seed, prefix):
    return synth.make_kv_prefix(shape, seed, prefix)


def clear_rows(logits: np.ndarray, tol: float) -> np.ndarray:
    """Row is clear when its top-2 logit gap exceeds tol * max|logit|."""
    top2 = np.sort(logits, axis=1)[:, -2:]
    scale = np.abs(logits).max(axis=1)
    return (top2[:, 1] - top2[:, 0]) > tol * scale


def rel_err_rows(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    return np.abs(got - ref).max(axis=1) / np.abs(ref).max(axis=1)


def check_accept_against_oracle(res, ores, ologits, tol):
    """Greedy acceptance must agree with the oracle along the oracle's path as
    long as every row on it is clear of near-ties; at a near-tie both
    choices are valid and the comparison stops."""
    clear = clear_rows(ologits, tol)
    path = ores["path"]
    for d, u in enumerate(path):
        if not clear[u]:
            return False
        assert int(res["pred"][u]) == int(ores["pred"][u]), (d, u)
        if d + 1 < len(path):
            assert int(res["path"][d + 1]) == path[d + 1]
    assert int(res["accept_len"]) == ores["accept_len"]
    assert int(res["bonus"]) == ores["bonus"]
    return True


def draft_dict(d) -> dict:
    n = int(d["n_nodes"])
    return {"n_nodes": n, "token": np.array(d["token"][:n]), "parent": np.array(d["parent"][:n]),
            "depth": np.array(d["depth"][:n]), "anc": np.array(d["anc"][:n])}


def assert_same_draft(d, od, tree: bool):
    n = od["n_nodes"]
    assert int(d["n_nodes"]) == n
    assert list(d["token"][:n]) == list(od["token"])
    assert list(d["parent"][:n]) == list(od["parent"])
    assert list(d["depth"][:n]) == list(od["depth"])
    if tree or n <= 64:
        assert [int(x) for x in d["anc"][:n]] == [int(x) for x in od["anc"]]
    f = od["n_found"]
    assert int(d["n_found"]) == f
    assert list(d["cand_len"][:f]) == list(od["cand_len"])
    assert list(d["cand_pos"][:f]) == list(od["cand_pos"])


class Gpu:
    """One model + cache on the GPU for a workload (weights from synth)."""

    def __init__(self, shape, w, kv_host, prefix: int, capacity: int):
        import paper_2609_32166_amd as pf
        import torch

        self.pf, self.torch = pf, torch
        self.shape = shape
        self.prefix = prefix
        self.model = pf.pf_model_create(pf.model_config(shape), pf.weights_to_device(w, shape.dtype))
        self.kv = pf.KVCache(self.model, capacity)
        self.kv_host_dev = pf.array_to_device(kv_host)
        pf.pf_kv_import(self.kv, self.kv_host_dev, prefix)
        self.draft = pf.new_draft()
        self.res = pf.new_result()

    def reset(self):
        self.pf.pf_kv_set_len(self.kv, self.prefix)

    def step(self, store_obj, ctx_tokens, k_max, tree=False, n_cand=1, max_nodes=64,
             rows=None, commit=True, want_logits=True, ctx_capacity=None):
        pf, torch = self.pf, self.torch
        rows = rows or ((max_nodes + 1) if tree else (k_max + 1))
        self.reset()
        ctx = pf.Context(ctx_tokens, ctx_capacity or (len(ctx_tokens) + 4 * 65))
        logits = (torch.zeros(rows, self.shape.vocab, device="cuda") if want_logits else None)
        pf.pf_draft_lookup(store_obj, ctx, k_max, tree, n_cand, max_nodes, self.draft)
        pf.pf_verify_step(self.model, self.kv, self.draft, rows, tree, logits, self.res)
        kv_rows = self.export(self.prefix, rows)
        if commit:
            pf.pf_kv_commit(self.kv, self.res, ctx)
        torch.cuda.synchronize()
        out = {"draft": pf.read_draft(self.draft), "res": pf.read_result(self.res),
               "logits": logits.cpu().numpy() if want_logits else None, "kv_rows": kv_rows,
               "ctx": ctx, "rows": rows}
        if commit:
            out["kv_len"] = int(self.kv.len.item())
            out["ctx_tokens"] = ctx.tokens()
        return out

    def export(self, start, n):
        torch = self.torch
        s = self.shape
        dt = torch.bfloat16 if s.dtype == "bf16" else torch.float32
        buf = torch.zeros(s.n_layers, 2, s.n_kv_heads, n, s.head_dim, dtype=dt, device="cuda")
        self.pf.pf_kv_export(self.kv, buf, start, n)
        return buf

    @staticmethod
    def to_np(t):
        import torch
        return t.to(torch.float64).cpu().numpy()


def splice(wl, om, kv_host, store, ctx, seed, j):
    """Append a store sequence [query | oracle greedy continuation (j) | random]."""
    g = oracle.greedy_decode(om, kv_host, int(ctx[-1]), j)["tokens"] if j else np.zeros(0, np.int32)
    seq = synth.splice_sequence(wl, seed, ctx[-wl.ngram:], g, wl.k_max + 2)
    return store.append(seq), g
