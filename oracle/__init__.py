"""CPU oracle for the retrieval-drafted verify step -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. The product library never calls it and
shares no code with it; the two meet only in the seeded inputs of ``synth``.

It computes, with plain fp64 loops in ``oracle.c``, what the paper
(arXiv 2609.32166, Section 3.2) defines:

* retrieval over the decoding experience memory: one shared token array,
  per-entry output-sequence boundary ``b``, eligibility ``p < b`` plus a token
  match, proposals truncated at ``b``, and an ordinary greedy pass when
  nothing is eligible ("Decoding experience memory", "Context-compatible
  retrieval");
* single-pass verification: one forward over the current token and the
  proposal, greedy predictions at every row, acceptance of the longest
  matching proposal prefix plus the model's next token, which must equal
  greedy decoding ("Single-pass token verification");
* the KV commit implied by that acceptance, the prompt-prefix carryover
  that resumes computation right after a reused prefix, and the rolling-image
  carryover that moves retained spans and re-rotates their keys (Section 3.4);
* the paper's own retrieval keys and lookup: final-layer states projected to
  256-dimensional int8 keys by a fixed random projection (Section 4) and the
  cosine argmax over the entries whose stored token matches the query token
  and that precede their boundary (Section 3.2).

Parity of the forward's logit values is pinned only by the invariants and
closed forms in the tests; the paper prints no worked numeric example for it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c (gcc, OpenMP). Building the checker is not using it."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O3", "-mavx2", "-mfma", "-fopenmp", "-fPIC", "-shared",
                               os.path.join(_HERE, "oracle.c"), "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class _Model(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int), ("H", ctypes.c_int), ("nq", ctypes.c_int),
                ("nkv", ctypes.c_int), ("hd", ctypes.c_int), ("F", ctypes.c_int),
                ("V", ctypes.c_int), ("theta", ctypes.c_double), ("eps", ctypes.c_double),
                ("bf16", ctypes.c_int),
                ("embed", ctypes.c_void_p), ("lm_head", ctypes.c_void_p),
                ("wqkv", ctypes.c_void_p), ("wo", ctypes.c_void_p), ("wgu", ctypes.c_void_p),
                ("wd", ctypes.c_void_p), ("attn_norm", ctypes.c_void_p),
                ("ffn_norm", ctypes.c_void_p), ("final_norm", ctypes.c_void_p)]


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        L = ctypes.CDLL(_LIB_PATH)
        vp, i32, i64, f64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_double
        L.or_forward.restype = i32
        L.or_forward.argtypes = [ctypes.POINTER(_Model), vp, i64, vp, i64, i32, vp, vp, vp, i32,
                                 vp, vp, vp, vp]
        L.or_layer.restype = None
        L.or_layer.argtypes = [ctypes.POINTER(_Model), i32, vp, i64, vp, i64, i32, vp, vp, vp, vp]
        L.or_head.restype = None
        L.or_head.argtypes = [ctypes.POINTER(_Model), vp, i32, vp, vp]
        L.or_lookup_candidates.restype = i32
        L.or_lookup_candidates.argtypes = [vp, vp, i64, i32, vp, i64, i32, i32, vp, vp]
        L.or_build_draft.restype = i32
        L.or_build_draft.argtypes = [vp, vp, vp, i32, i32, i32, i32, vp, vp, vp, vp]
        L.or_round_bf16.restype = f64
        L.or_round_bf16.argtypes = [f64]
        L.or_double_to_bf16_bits.restype = ctypes.c_uint16
        L.or_double_to_bf16_bits.argtypes = [f64]
        L.or_bf16_to_double.restype = f64
        L.or_bf16_to_double.argtypes = [ctypes.c_uint16]
        L.or_rmsnorm.restype = None
        L.or_rmsnorm.argtypes = [vp, vp, i32, f64, vp]
        L.or_rope.restype = None
        L.or_rope.argtypes = [vp, i32, f64, f64]
        L.or_swiglu.restype = f64
        L.or_swiglu.argtypes = [f64, f64]
        L.or_linear.restype = None
        L.or_linear.argtypes = [vp, i32, i64, i64, i32, vp, vp]
        L.or_attend.restype = None
        L.or_attend.argtypes = [vp, vp, vp, i64, i32, f64, vp]
        L.or_argmax.restype = ctypes.c_int32
        L.or_argmax.argtypes = [vp, i64]
        L.or_key_project.restype = None
        L.or_key_project.argtypes = [vp, i32, i32, vp, i64, vp]
        L.or_key_encode.restype = None
        L.or_key_encode.argtypes = [vp, i32, i32, vp, i64, vp]
        L.or_cos_candidates.restype = i32
        L.or_cos_candidates.argtypes = [vp, vp, i64, vp, i32, ctypes.c_int32, vp, i32, i32, vp,
                                        vp, vp]
        L.or_set_threads.restype = None
        L.or_set_threads.argtypes = [i32]
        L.or_get_threads.restype = i32
        L.or_get_threads.argtypes = []
        n = _affinity()
        L.or_set_threads(n)
        _lib = L
    return _lib


def _affinity() -> int:
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def threads() -> int:
    return lib().or_get_threads()


def set_threads(n: int) -> None:
    lib().or_set_threads(int(n))


def _ptr(a: Optional[np.ndarray]) -> Optional[int]:
    return None if a is None else a.ctypes.data


# ----------------------------------------------------------------------------
# Building blocks (exposed for the pins)
# ----------------------------------------------------------------------------

def round_bf16(x: float) -> float:
    return lib().or_round_bf16(float(x))


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    x = np.ascontiguousarray(x, np.float64)
    g = np.ascontiguousarray(g, np.float32)
    y = np.empty_like(x)
    lib().or_rmsnorm(_ptr(x), _ptr(g), len(x), eps, _ptr(y))
    return y


def rope(v: np.ndarray, pos: float, theta: float) -> np.ndarray:
    v = np.array(v, np.float64, copy=True)
    lib().or_rope(_ptr(v), len(v), float(pos), float(theta))
    return v


def swiglu(g: float, u: float) -> float:
    return lib().or_swiglu(float(g), float(u))


def linear(W: np.ndarray, x: np.ndarray) -> np.ndarray:
    """y = x @ W.T with W fp32 or bf16 bits (uint16), x fp64 [M][K]."""
    W = np.ascontiguousarray(W)
    x = np.ascontiguousarray(x, np.float64)
    N, K = W.shape
    M = x.shape[0]
    y = np.empty((M, N), np.float64)
    lib().or_linear(_ptr(W), int(W.dtype == np.uint16), N, K, M, _ptr(x), _ptr(y))
    return y


def attend(q: np.ndarray, keys: np.ndarray, vals: np.ndarray, scale: float) -> np.ndarray:
    q = np.ascontiguousarray(q, np.float64)
    keys = np.ascontiguousarray(keys, np.float64)
    vals = np.ascontiguousarray(vals, np.float64)
    nk, d = keys.shape
    kp = (ctypes.c_void_p * max(nk, 1))(*[keys.ctypes.data + 8 * d * t for t in range(nk)])
    vpp = (ctypes.c_void_p * max(nk, 1))(*[vals.ctypes.data + 8 * d * t for t in range(nk)])
    out = np.empty(d, np.float64)
    lib().or_attend(_ptr(q), kp, vpp, nk, d, scale, _ptr(out))
    return out


def argmax(v: np.ndarray) -> int:
    v = np.ascontiguousarray(v, np.float32)
    return int(lib().or_argmax(_ptr(v), len(v)))


# ----------------------------------------------------------------------------
# Model
# ----------------------------------------------------------------------------

class Model:
    """Holds a reference to the host weights (synth layout) for the oracle."""

    def __init__(self, shape, weights: Dict[str, np.ndarray]):
        self.shape = shape
        self.w = {k: np.ascontiguousarray(v) for k, v in weights.items()}
        self.bf16 = shape.dtype == "bf16"
        s = shape
        self._c = _Model(s.n_layers, s.hidden, s.n_heads, s.n_kv_heads, s.head_dim, s.ffn,
                         s.vocab, float(s.rope_theta), float(s.rms_eps), int(self.bf16),
                         *[self.w[k].ctypes.data for k in
                           ("embed", "lm_head", "wqkv", "wo", "wgu", "wd", "attn_norm",
                            "ffn_norm", "final_norm")])

    def forward(self, kv_prefix: np.ndarray, tok: Sequence[int], pos: Sequence[int],
                vis: np.ndarray, kv_extra: Optional[np.ndarray] = None, logits_from: int = 0,
                want_logits: bool = True, want_kv: bool = True, hidden: Optional[np.ndarray] = None,
                resid: Optional[np.ndarray] = None):
        """Forward of M new rows. Returns (logits [M][V] fp32 or None, kv_new
        [L][2][nkv][M][hd] fp64 or None). kv_prefix: [L][2][nkv][P][hd].
        hidden, if given ([M][H] fp64), receives the final-layer states of
        rows >= logits_from (the lm_head input); resid, if given
        ([L+1][M][H] fp64), the embeddings and the residual stream after
        every layer."""
        s = self.shape
        kv_prefix = np.ascontiguousarray(kv_prefix)
        P = kv_prefix.shape[3]
        tok = np.ascontiguousarray(tok, np.int32)
        pos = np.ascontiguousarray(pos, np.int64)
        M = len(tok)
        vis = np.ascontiguousarray(vis, np.uint8).reshape(M, M)
        if kv_extra is not None:
            kv_extra = np.ascontiguousarray(kv_extra, np.float64)
            E = kv_extra.shape[3]
        else:
            E = 0
        logits = np.zeros((M, s.vocab), np.float32) if want_logits else None
        kv_new = (np.zeros((s.n_layers, 2, s.n_kv_heads, M, s.head_dim), np.float64)
                  if want_kv else None)
        if hidden is not None:
            assert hidden.dtype == np.float64 and hidden.shape == (M, s.hidden)
            assert hidden.flags.c_contiguous
        if resid is not None:
            assert resid.dtype == np.float64 and resid.shape == (s.n_layers + 1, M, s.hidden)
            assert resid.flags.c_contiguous
        lib().or_forward(ctypes.byref(self._c), _ptr(kv_prefix), P, _ptr(kv_extra), E, M,
                         _ptr(tok), _ptr(pos), _ptr(vis), int(logits_from), _ptr(logits),
                         _ptr(kv_new), _ptr(hidden), _ptr(resid))
        return logits, kv_new

    def layer(self, l: int, kv_prefix: np.ndarray, x: np.ndarray, pos: Sequence[int],
              vis: np.ndarray, kv_extra: Optional[np.ndarray] = None, want_kv: bool = False):
        """Decoder layer l applied to the residual stream x [M][H]; returns
        the stream after the layer (x itself is not modified), and with
        want_kv also the layer's K/V of the new rows ([2][nkv][M][hd])."""
        s = self.shape
        kv_prefix = np.ascontiguousarray(kv_prefix)
        P = kv_prefix.shape[3]
        x = np.array(x, np.float64, copy=True, order="C")
        M = x.shape[0]
        assert x.shape == (M, s.hidden)
        pos = np.ascontiguousarray(pos, np.int64)
        vis = np.ascontiguousarray(vis, np.uint8).reshape(M, M)
        E = 0
        if kv_extra is not None:
            kv_extra = np.ascontiguousarray(kv_extra, np.float64)
            E = kv_extra.shape[3]
        kv_new = (np.zeros((s.n_layers, 2, s.n_kv_heads, M, s.head_dim), np.float64)
                  if want_kv else None)
        lib().or_layer(ctypes.byref(self._c), int(l), _ptr(kv_prefix), P, _ptr(kv_extra), E, M,
                       _ptr(pos), _ptr(vis), _ptr(x), _ptr(kv_new))
        return (x, kv_new[l]) if want_kv else x

    def head(self, x: np.ndarray, want_hidden: bool = False):
        """Final norm and lm_head of the residual stream x [M][H]: logits
        [M][V] fp32 (and the lm_head input with want_hidden)."""
        s = self.shape
        x = np.ascontiguousarray(x, np.float64)
        M = x.shape[0]
        logits = np.zeros((M, s.vocab), np.float32)
        hidden = np.zeros((M, s.hidden), np.float64) if want_hidden else None
        lib().or_head(ctypes.byref(self._c), _ptr(x), M, _ptr(logits), _ptr(hidden))
        return (logits, hidden) if want_hidden else logits


# ----------------------------------------------------------------------------
# Retrieval
# ----------------------------------------------------------------------------

MAX_NODES = 65


def lookup(tokens: np.ndarray, seq_offsets: np.ndarray, ngram: int, ctx: np.ndarray,
           k_max: int, n_cand: int = 1, tree: bool = False, max_nodes: int = 64) -> dict:
    """Exhaustive-scan retrieval and draft construction (see oracle.c)."""
    tokens = np.ascontiguousarray(tokens, np.int32)
    seq_offsets = np.ascontiguousarray(seq_offsets, np.int64)
    ctx = np.ascontiguousarray(ctx, np.int32)
    nc = max(1, n_cand)
    cpos = np.zeros(nc, np.int64)
    clen = np.zeros(nc, np.int32)
    found = lib().or_lookup_candidates(_ptr(tokens), _ptr(seq_offsets), len(seq_offsets) - 1,
                                       ngram, _ptr(ctx), len(ctx), k_max, nc, _ptr(cpos),
                                       _ptr(clen))
    ntok = np.zeros(MAX_NODES, np.int32)
    par = np.zeros(MAX_NODES, np.int32)
    dep = np.zeros(MAX_NODES, np.int32)
    anc = np.zeros(MAX_NODES, np.uint64)
    cur = int(ctx[-1]) if len(ctx) else 0
    n = lib().or_build_draft(_ptr(tokens), _ptr(cpos), _ptr(clen), found, cur, int(tree),
                             max_nodes, _ptr(ntok), _ptr(par), _ptr(dep), _ptr(anc))
    return {"n_nodes": int(n), "token": ntok[:n].copy(), "parent": par[:n].copy(),
            "depth": dep[:n].copy(), "anc": anc[:n].copy(), "n_found": int(found),
            "cand_pos": cpos[:found].copy(), "cand_len": clen[:found].copy()}


KEY_DIM = 256  # Section 4: 256-dimensional int8 retrieval keys


def key_project(R: np.ndarray, h: np.ndarray) -> np.ndarray:
    """The fp64 projection v = R h of hidden states h [n][H] (plain index-order
    sums, see or_key_project): [n][KEY_DIM]."""
    R = np.ascontiguousarray(R, np.float64)
    h = np.ascontiguousarray(np.atleast_2d(h), np.float64)
    kd, H = R.shape
    assert h.shape[1] == H
    v = np.zeros((h.shape[0], kd), np.float64)
    lib().or_key_project(_ptr(R), kd, H, _ptr(h), h.shape[0], _ptr(v))
    return v


def key_encode(R: np.ndarray, h: np.ndarray) -> np.ndarray:
    """int8 retrieval keys of hidden states h [n][H] under the projection R
    [KEY_DIM][H] (see or_key_encode)."""
    R = np.ascontiguousarray(R, np.float64)
    h = np.ascontiguousarray(np.atleast_2d(h), np.float64)
    kd, H = R.shape
    assert h.shape[1] == H and kd <= 1024
    out = np.zeros((h.shape[0], kd), np.int8)
    lib().or_key_encode(_ptr(R), kd, H, _ptr(h), h.shape[0], _ptr(out))
    return out


def cos_lookup(tokens: np.ndarray, seq_offsets: np.ndarray, keys: np.ndarray, y: int,
               qkey: np.ndarray, k_max: int, n_cand: int = 1, tree: bool = False,
               max_nodes: int = 64) -> dict:
    """Cosine retrieval over keyed store entries (see or_cos_candidates) and
    the same draft construction as the n-gram lookup; node 0 is y."""
    tokens = np.ascontiguousarray(tokens, np.int32)
    seq_offsets = np.ascontiguousarray(seq_offsets, np.int64)
    keys = np.ascontiguousarray(keys, np.int8)
    qkey = np.ascontiguousarray(qkey, np.int8).reshape(-1)
    kd = qkey.shape[0]
    assert keys.shape == (len(tokens), kd)
    nc = max(1, n_cand)
    cpos = np.zeros(nc, np.int64)
    clen = np.zeros(nc, np.int32)
    ccos = np.zeros(nc, np.float64)
    found = lib().or_cos_candidates(_ptr(tokens), _ptr(seq_offsets), len(seq_offsets) - 1,
                                    _ptr(keys), kd, int(y), _ptr(qkey), k_max, nc, _ptr(cpos),
                                    _ptr(clen), _ptr(ccos))
    ntok = np.zeros(MAX_NODES, np.int32)
    par = np.zeros(MAX_NODES, np.int32)
    dep = np.zeros(MAX_NODES, np.int32)
    anc = np.zeros(MAX_NODES, np.uint64)
    n = lib().or_build_draft(_ptr(tokens), _ptr(cpos), _ptr(clen), found, int(y), int(tree),
                             max_nodes, _ptr(ntok), _ptr(par), _ptr(dep), _ptr(anc))
    return {"n_nodes": int(n), "token": ntok[:n].copy(), "parent": par[:n].copy(),
            "depth": dep[:n].copy(), "anc": anc[:n].copy(), "n_found": int(found),
            "cand_pos": cpos[:found].copy(), "cand_len": clen[:found].copy(),
            "cand_cos": ccos[:found].copy()}


def visibility(draft: dict, rows: int, tree: bool) -> np.ndarray:
    """vis[j][i] = row j attends to new row i. Rows past n_nodes are padding:
    linear padding keeps the causal pattern; tree padding sees the root and
    itself. Real rows never see padding rows."""
    n = draft["n_nodes"]
    vis = np.zeros((rows, rows), np.uint8)
    for j in range(rows):
        if not tree:
            vis[j, :j + 1] = 1
        elif j < n:
            u = j
            while u >= 0:
                vis[j, u] = 1
                u = int(draft["parent"][u])
        else:
            vis[j, 0] = 1
            vis[j, j] = 1
    return vis


def draft_rows(draft: dict, rows: int, tree: bool):
    """(tokens, depths) of the padded verify rows: padding rows use token 0;
    their depth is the row index (linear) or 1 (tree)."""
    n = draft["n_nodes"]
    tok = np.zeros(rows, np.int32)
    dep = np.zeros(rows, np.int64)
    tok[:n] = draft["token"]
    dep[:n] = draft["depth"]
    for j in range(n, rows):
        dep[j] = j if not tree else 1
    return tok, dep


def accept(draft: dict, pred: Sequence[int], tree: bool) -> dict:
    """Longest proposal prefix matching the greedy predictions, plus the
    model's token after it (Section 3.2, single-pass token verification)."""
    n = draft["n_nodes"]
    tokens, parent = draft["token"], draft["parent"]
    path = [0]
    cur = 0
    while True:
        want = int(pred[cur])
        nxt = -1
        if tree:
            for u in range(1, n):
                if int(parent[u]) == cur and int(tokens[u]) == want:
                    nxt = u
                    break
        elif cur + 1 < n and int(tokens[cur + 1]) == want:
            nxt = cur + 1
        if nxt < 0:
            break
        path.append(nxt)
        cur = nxt
    return {"accept_len": len(path) - 1, "bonus": int(pred[cur]), "path": path}


def verify_batched(model: Model, kv_prefix: np.ndarray, draft: dict, rows: int, tree: bool,
                   want_logits: bool = True, want_hidden: bool = False) -> dict:
    """One forward over every verify row, then greedy accept. With
    want_hidden, res["hidden"] holds every row's final-layer state."""
    P = kv_prefix.shape[3]
    tok, dep = draft_rows(draft, rows, tree)
    vis = visibility(draft, rows, tree)
    hidden = np.zeros((rows, model.shape.hidden), np.float64) if want_hidden else None
    logits, kv_new = model.forward(kv_prefix, tok, P + dep, vis, hidden=hidden)
    pred = [argmax(logits[j]) for j in range(rows)]
    res = accept(draft, pred, tree)
    res.update(pred=np.array(pred, np.int32), logits=logits if want_logits else None,
               kv_new=kv_new, tok=tok, pos=P + dep, hidden=hidden)
    return res


def verify_sequential(model: Model, kv_prefix: np.ndarray, draft: dict, tree: bool) -> dict:
    """The definition the batched pass must reproduce: single-token greedy
    decodes from the current token, following the proposal while it agrees
    with the greedy choice, stopping at the first disagreement."""
    P = kv_prefix.shape[3]
    n = draft["n_nodes"]
    tokens, parent = draft["token"], draft["parent"]
    extra = None
    cur = 0
    path = [0]
    preds = []
    step_logits = []
    one = np.ones((1, 1), np.uint8)
    while True:
        d = len(path) - 1
        lg, kv1 = model.forward(kv_prefix, [int(tokens[cur])], [P + d], one, kv_extra=extra)
        g = argmax(lg[0])
        preds.append(g)
        step_logits.append(lg[0])
        extra = kv1 if extra is None else np.concatenate([extra, kv1], axis=3)
        nxt = -1
        if tree:
            for u in range(1, n):
                if int(parent[u]) == cur and int(tokens[u]) == g:
                    nxt = u
                    break
        elif cur + 1 < n and int(tokens[cur + 1]) == g:
            nxt = cur + 1
        if nxt < 0:
            break
        path.append(nxt)
        cur = nxt
    return {"accept_len": len(path) - 1, "bonus": preds[-1], "path": path,
            "pred_path": np.array(preds, np.int32), "kv_path": extra,
            "logits": np.stack(step_logits)}


def greedy_decode(model: Model, kv_prefix: np.ndarray, first_token: int, steps: int,
                  want_hidden: bool = False) -> dict:
    """`steps` plain greedy decodes starting from `first_token` at position P.
    Also returns each step's top-2 logit gap relative to the largest |logit|
    ("margin") and, with want_hidden, the final-layer state that produced
    each output token ("hidden", [steps][H])."""
    P = kv_prefix.shape[3]
    extra = None
    tok = int(first_token)
    out, margin = [], []
    hid = np.zeros((steps, model.shape.hidden), np.float64) if want_hidden else None
    one = np.ones((1, 1), np.uint8)
    for d in range(steps):
        h = np.zeros((1, model.shape.hidden), np.float64) if want_hidden else None
        lg, kv1 = model.forward(kv_prefix, [tok], [P + d], one, kv_extra=extra, hidden=h)
        tok = argmax(lg[0])
        out.append(tok)
        top2 = np.sort(lg[0].astype(np.float64))[-2:]
        margin.append((top2[1] - top2[0]) / max(np.abs(lg[0]).max(), 1e-30))
        if want_hidden:
            hid[d] = h[0]
        extra = kv1 if extra is None else np.concatenate([extra, kv1], axis=3)
    return {"tokens": np.array(out, np.int32), "kv": extra, "margin": np.array(margin),
            "hidden": hid}


def commit(kv_new: np.ndarray, path: Sequence[int]) -> np.ndarray:
    """KV rows kept after acceptance: node path[d] lands at depth slot d."""
    return kv_new[:, :, :, list(path), :]


def kv_carry(kv: np.ndarray, spans: Sequence[Sequence[int]], theta: float) -> np.ndarray:
    """Rolling-image KV-state carryover (Section 3.4): each retained span
    (src, dst, n) of cached tokens moves from positions src..src+n-1 to
    dst..dst+n-1; a key cached at position m becomes R(m') R(m)^-1 of it at
    m' = m + dst - src (R: the model's rotary embedding, inverted as the
    rotation by -m), values move unchanged. Spans apply one after another,
    each reading the cache as the previous ones left it. kv: logical layout
    [L][2][n_kv][T][head_dim]; returns a new fp64 array."""
    out = np.array(kv, np.float64, copy=True)
    for src, dst, n in spans:
        src, dst, n = int(src), int(dst), int(n)
        keys = out[:, 0, :, src:src + n, :].copy()
        vals = out[:, 1, :, src:src + n, :].copy()
        L, nkv = keys.shape[0], keys.shape[1]
        for l in range(L):
            for g in range(nkv):
                for i in range(n):
                    back = rope(keys[l, g, i], -(src + i), theta)       # R(m)^-1
                    keys[l, g, i] = rope(back, dst + i, theta)          # R(m')
        out[:, 0, :, dst:dst + n, :] = keys
        out[:, 1, :, dst:dst + n, :] = vals
    return out


def prefill(model: Model, kv_prefix: np.ndarray, tokens: Sequence[int], chunk: int) -> dict:
    """Prompt-prefix carryover (Section 3.4): the reused prefix's KV is kept and
    computation resumes at the first new token, here in causal chunks. Returns
    the new rows' KV and the last row's logits."""
    P = kv_prefix.shape[3]
    tokens = np.asarray(tokens, np.int32)
    n = len(tokens)
    extra = None
    logits = None
    for c0 in range(0, n, chunk):
        c1 = min(n, c0 + chunk)
        m = c1 - c0
        vis = np.tril(np.ones((m, m), np.uint8))
        last = c1 == n
        lg, kv1 = model.forward(kv_prefix, tokens[c0:c1], P + np.arange(c0, c1), vis,
                                kv_extra=extra, logits_from=m - 1 if last else m,
                                want_logits=last)
        if last:
            logits = lg[m - 1]
        extra = kv1 if extra is None else np.concatenate([extra, kv1], axis=3)
    return {"kv_new": extra, "logits_last": logits}
