"""Seeded synthetic inputs shared by the oracle and the HIP path.

This package holds workload shapes and input generators only: model weights,
KV prefixes, experience stores, decoding contexts. It contains none of the
decoding method's arithmetic. Both sides consume the exact same bytes.

Random draws come from one counter-based SplitMix64 stream per (seed, tensor)
implemented in ``synth.c`` (bulk tensors) and mirrored here in numpy for
small integer draws; the two implementations are checked against each other
in the CPU tests.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess
from typing import Dict, List, Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None

GOLDEN = np.uint64(0x9E3779B97F4A7C15)


def build(force: bool = True) -> str:
    """Compile synth.c into libsynth.so (gcc, -O2, pthreads)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-pthread",
                               os.path.join(_HERE, "synth.c"), "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        u64, i64, f64, vp, i32 = (ctypes.c_uint64, ctypes.c_int64, ctypes.c_double,
                                  ctypes.c_void_p, ctypes.c_int)
        lib.sy_key.restype = u64
        lib.sy_key.argtypes = [u64, u64]
        lib.sy_draw.restype = u64
        lib.sy_draw.argtypes = [u64, u64]
        for fn in (lib.sy_normal_f32, lib.sy_normal_bf16, lib.sy_normal_bf16_as_f32):
            fn.restype = None
            fn.argtypes = [u64, i64, f64, f64, vp, i32]
        lib.sy_draws.restype = None
        lib.sy_draws.argtypes = [u64, u64, i64, vp]
        _lib = lib
    return _lib


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


# ----------------------------------------------------------------------------
# Counter-based stream (numpy mirror of synth.c)
# ----------------------------------------------------------------------------

def _mix64(z: np.ndarray) -> np.ndarray:
    z = z.astype(np.uint64, copy=True)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        z = z ^ (z >> np.uint64(31))
    return z


def key(seed: int, tensor_id: int) -> int:
    """Stream key for (seed, tensor id); same definition as sy_key in synth.c."""
    with np.errstate(over="ignore"):
        a = _mix64(np.array([np.uint64(seed) + GOLDEN], dtype=np.uint64))[0]
        b = np.uint64(tensor_id) * np.uint64(0xD1B54A32D192ED03)
        return int(_mix64(np.array([a ^ b], dtype=np.uint64))[0])


def draws(k: int, n: int, first: int = 0) -> np.ndarray:
    """Raw uint64 draws i = first..first+n-1 of stream k."""
    idx = np.arange(first, first + n, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(k) + (idx + np.uint64(1)) * GOLDEN
    return _mix64(z)


def uniform(k: int, n: int, first: int = 0) -> np.ndarray:
    """53-bit uniforms in [0, 1)."""
    return (draws(k, n, first) >> np.uint64(11)).astype(np.float64) * (1.0 / 9007199254740992.0)


def randint(k: int, n: int, lo: int, hi: int, first: int = 0) -> np.ndarray:
    """Integers in [lo, hi) (hi > lo), by scaling a 53-bit uniform."""
    u = uniform(k, n, first)
    return np.minimum(lo + np.floor(u * (hi - lo)).astype(np.int64), hi - 1)


def normal_f32(k: int, n: int, std: float = 1.0, mean: float = 0.0) -> np.ndarray:
    out = np.empty(n, dtype=np.float32)
    _load().sy_normal_f32(k, n, mean, std, out.ctypes.data, _threads())
    return out


def normal_bf16(k: int, n: int, std: float = 1.0, mean: float = 0.0) -> np.ndarray:
    """bf16 bit patterns (uint16) of round-to-nearest-even(mean + std*N(0,1))."""
    out = np.empty(n, dtype=np.uint16)
    _load().sy_normal_bf16(k, n, mean, std, out.ctypes.data, _threads())
    return out


def normal_bf16_as_f32(k: int, n: int, std: float = 1.0, mean: float = 0.0) -> np.ndarray:
    out = np.empty(n, dtype=np.float32)
    _load().sy_normal_bf16_as_f32(k, n, mean, std, out.ctypes.data, _threads())
    return out


def zipf(k: int, n: int, vocab: int, s: float = 1.1, first: int = 0) -> np.ndarray:
    """Zipf(s) token ids over ranks 1..vocab by inverse CDF; id = rank - 1."""
    cdf = np.cumsum(np.arange(1, vocab + 1, dtype=np.float64) ** (-s))
    cdf /= cdf[-1]
    u = uniform(k, n, first)
    return np.minimum(np.searchsorted(cdf, u, side="right"), vocab - 1).astype(np.int32)


# ----------------------------------------------------------------------------
# Workload shapes
# ----------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class ModelShape:
    n_layers: int
    hidden: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    rope_theta: float
    rms_eps: float
    dtype: str  # "f32" or "bf16"

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def with_layers(self, n: int) -> "ModelShape":
        return dataclasses.replace(self, n_layers=n)

    def weight_bytes(self) -> int:
        esz = 4 if self.dtype == "f32" else 2
        per_layer = (self.hidden * (self.q_dim + 2 * self.kv_dim) + self.q_dim * self.hidden
                     + 3 * self.hidden * self.ffn)
        return esz * (self.n_layers * per_layer + self.hidden * self.vocab)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    index: int          # position in the workload list (1-based)
    model: ModelShape
    prefix: int         # cached KV prefix length P
    k_max: int          # draft tokens per verify
    ngram: int          # lookup n
    tree: bool          # prefix-shared token tree draft
    n_cand: int         # candidates merged into the tree
    max_nodes: int      # non-root tree node cap
    store_seqs: int
    store_len: Tuple[int, int]   # inclusive length range
    store_tokens: str   # "uniform" or "zipf"
    planted: int        # planted repeated 16-grams (uniform store)
    prefill_reuse: int = 0       # reused prefix before the new chunk (carry-forward)
    prefill_new: int = 0         # new tokens prefilled
    prefill_chunk: int = 0

    @property
    def rows(self) -> int:
        """Verify rows M (padded draft + the current token)."""
        return (self.max_nodes + 1) if self.tree else (self.k_max + 1)

    def verify_bytes(self) -> int:
        """Algorithmic HBM bytes of one verify step: every weight once, the KV
        prefix read, the draft rows' KV read and written."""
        m = self.model
        esz = 4 if m.dtype == "f32" else 2
        kv_row = 2 * m.n_kv_heads * m.head_dim * esz * m.n_layers
        M = self.rows
        return m.weight_bytes() + kv_row * (self.prefix + M) + kv_row * M


TINY = ModelShape(2, 256, 4, 2, 64, 688, 4096, 1e4, 1e-6, "f32")
M3B = ModelShape(36, 2048, 16, 2, 128, 11008, 151936, 1e6, 1e-6, "bf16")
M7B = ModelShape(28, 3584, 28, 4, 128, 18944, 152064, 1e6, 1e-6, "bf16")

WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", 1, TINY, 512, 8, 3, False, 1, 8, 64, (128, 128), "uniform", 8),
    "3b": Workload("3b", 2, M3B, 4096, 16, 4, False, 1, 16, 2000, (64, 256), "zipf", 0),
    "7b": Workload("7b", 3, M7B, 8192, 32, 4, False, 1, 32, 10000, (64, 512), "zipf", 0),
    "3b_tree": Workload("3b_tree", 4, M3B, 4096, 16, 4, True, 4, 48, 2000, (64, 256), "zipf", 0),
    "7b_carry": Workload("7b_carry", 5, M7B, 8192, 16, 4, False, 1, 16, 10000, (64, 512), "zipf",
                         0, prefill_reuse=6144, prefill_new=2048, prefill_chunk=512),
}

# Tensor ids of the generator streams.
_TID = {"embed": 1, "lm_head": 2, "final_norm": 3, "attn_norm": 10, "wqkv": 11, "wo": 12,
        "ffn_norm": 13, "wgu": 14, "wd": 15, "kv": 20, "ctx": 30, "store_len": 40,
        "store_tok": 41, "plant": 42, "query": 43, "splice": 44, "prefill_tok": 45}

WEIGHT_STD = 0.02
GAIN_STD = 0.1


def _gen(dtype: str, k: int, n: int, std: float, mean: float = 0.0) -> np.ndarray:
    if dtype == "bf16":
        return normal_bf16(k, n, std, mean)
    return normal_f32(k, n, std, mean)


def make_weights(shape: ModelShape, seed: int) -> Dict[str, np.ndarray]:
    """Random-init decoder weights, N(0, 0.02^2), bf16 bits or fp32.

    Layouts (row-major): embed, lm_head [V][H]; wqkv [L][q+2kv][H] (rows: all
    query heads, then keys, then values); wo [L][H][q]; wgu [L][2F][H] (gate
    rows then up rows); wd [L][H][F]. Norm gains are fp32, bf16-representable,
    1 + 0.1*N(0,1).
    """
    L, H, V, F = shape.n_layers, shape.hidden, shape.vocab, shape.ffn
    q, kv = shape.q_dim, shape.kv_dim
    dt = shape.dtype
    w = {}
    w["embed"] = _gen(dt, key(seed, _TID["embed"]), V * H, WEIGHT_STD).reshape(V, H)
    w["lm_head"] = _gen(dt, key(seed, _TID["lm_head"]), V * H, WEIGHT_STD).reshape(V, H)
    w["wqkv"] = _gen(dt, key(seed, _TID["wqkv"]), L * (q + 2 * kv) * H, WEIGHT_STD).reshape(
        L, q + 2 * kv, H)
    w["wo"] = _gen(dt, key(seed, _TID["wo"]), L * H * q, WEIGHT_STD).reshape(L, H, q)
    w["wgu"] = _gen(dt, key(seed, _TID["wgu"]), L * 2 * F * H, WEIGHT_STD).reshape(L, 2 * F, H)
    w["wd"] = _gen(dt, key(seed, _TID["wd"]), L * H * F, WEIGHT_STD).reshape(L, H, F)
    w["attn_norm"] = normal_bf16_as_f32(key(seed, _TID["attn_norm"]), L * H, GAIN_STD,
                                        1.0).reshape(L, H)
    w["ffn_norm"] = normal_bf16_as_f32(key(seed, _TID["ffn_norm"]), L * H, GAIN_STD,
                                       1.0).reshape(L, H)
    w["final_norm"] = normal_bf16_as_f32(key(seed, _TID["final_norm"]), H, GAIN_STD, 1.0)
    return w


def make_kv_prefix(shape: ModelShape, seed: int, prefix: int) -> np.ndarray:
    """Synthetic cached K/V for positions 0..P-1, N(0,1).

    Logical layout [L][2][n_kv][P][head_dim] (index 0 = keys, 1 = values),
    bf16 bits or fp32.
    """
    n = shape.n_layers * 2 * shape.n_kv_heads * prefix * shape.head_dim
    arr = _gen(shape.dtype, key(seed, _TID["kv"]), n, 1.0)
    return arr.reshape(shape.n_layers, 2, shape.n_kv_heads, prefix, shape.head_dim)


# ----------------------------------------------------------------------------
# Experience store and contexts
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class Store:
    tokens: np.ndarray        # int32 [T], all output sequences concatenated
    seq_offsets: np.ndarray   # int64 [n_seqs + 1]
    planted: List[np.ndarray] = dataclasses.field(default_factory=list)

    @property
    def n_seqs(self) -> int:
        return len(self.seq_offsets) - 1

    def append(self, seq: np.ndarray) -> "Store":
        seq = np.asarray(seq, dtype=np.int32)
        toks = np.concatenate([self.tokens, seq]).astype(np.int32)
        offs = np.concatenate([self.seq_offsets, [self.seq_offsets[-1] + len(seq)]]).astype(np.int64)
        return Store(toks, offs, list(self.planted))


def make_store(wl: Workload, seed: int) -> Store:
    V = wl.model.vocab
    lo, hi = wl.store_len
    lens = randint(key(seed, _TID["store_len"]), wl.store_seqs, lo, hi + 1)
    offs = np.zeros(wl.store_seqs + 1, dtype=np.int64)
    offs[1:] = np.cumsum(lens)
    T = int(offs[-1])
    kt = key(seed, _TID["store_tok"])
    if wl.store_tokens == "uniform":
        toks = randint(kt, T, 0, V).astype(np.int32)
    else:
        toks = zipf(kt, T, V)
    store = Store(toks, offs)
    if wl.planted:
        store = _plant(store, wl, seed)
    return store


def _plant(store: Store, wl: Workload, seed: int, gram: int = 16, copies: int = 4) -> Store:
    """Plant `wl.planted` distinct random 16-grams, each in `copies` distinct
    sequences at non-overlapping offsets."""
    V = wl.model.vocab
    kp = key(seed, _TID["plant"])
    ctr = 0
    toks = store.tokens.copy()
    used: Dict[int, List[Tuple[int, int]]] = {}
    grams = []
    for g in range(wl.planted):
        gtoks = randint(kp, gram, 0, V, first=ctr).astype(np.int32)
        ctr += gram
        grams.append(gtoks)
        seqs_done = set()
        while len(seqs_done) < copies:
            s = int(randint(kp, 1, 0, store.n_seqs, first=ctr)[0])
            ctr += 1
            if s in seqs_done:
                continue
            a, b = int(store.seq_offsets[s]), int(store.seq_offsets[s + 1])
            if b - a < gram + 1:
                continue
            off = int(randint(kp, 1, 0, b - a - gram, first=ctr)[0])
            ctr += 1
            span = (a + off, a + off + gram)
            if any(not (span[1] <= u0 or span[0] >= u1) for (u0, u1) in used.get(s, [])):
                continue
            used.setdefault(s, []).append(span)
            toks[span[0]:span[1]] = gtoks
            seqs_done.add(s)
    return Store(toks, store.seq_offsets.copy(), grams)


def make_context(wl: Workload, seed: int, store: Store, hit: Optional[bool] = None,
                 length: Optional[int] = None) -> Tuple[np.ndarray, dict]:
    """Decoding context: prompt + output history of `length` (default P+1)
    tokens, the last one being the current token.

    Tiny workload: uniform ids. Larger workloads: 64 Zipf text tokens, a run
    of image-patch placeholder ids (V-1) up to ~61% of the prompt, then Zipf
    text history. With `hit` (default: 90% of seeds) the last n tokens are a
    copy of an n-window of a random stored sequence that ends before that
    sequence's last token, so at least one eligible store entry exists.
    """
    V = wl.model.vocab
    n = wl.ngram
    T = (wl.prefix + 1) if length is None else length
    kc = key(seed, _TID["ctx"])
    if wl.store_tokens == "uniform":
        ctx = randint(kc, T, 0, V).astype(np.int32)
    else:
        ctx = zipf(kc, T, V)
        img0 = min(64, T)
        img1 = min(T, img0 + int(round(0.61 * wl.prefix)))
        ctx[img0:img1] = V - 1
    kq = key(seed, _TID["query"])
    if hit is None:
        hit = bool(uniform(kq, 1, first=0)[0] < 0.9)
    info = {"hit": hit}
    if hit and T >= n:
        for attempt in range(1000):
            s = int(randint(kq, 1, 0, store.n_seqs, first=1 + 2 * attempt)[0])
            a, b = int(store.seq_offsets[s]), int(store.seq_offsets[s + 1])
            if b - a < n + 1:
                continue
            # window end p in [a+n-1, b-2] so that p < b-1 (the boundary)
            p = int(randint(kq, 1, a + n - 1, b - 1, first=2 + 2 * attempt)[0])
            ctx[T - n:] = store.tokens[p - n + 1:p + 1]
            info.update(seq=s, pos=p)
            break
    return ctx.astype(np.int32), info


def splice_sequence(wl: Workload, seed: int, query: np.ndarray, cont: np.ndarray,
                    extra: int) -> np.ndarray:
    """A store sequence [query n-gram | cont | `extra` random tokens]."""
    V = wl.model.vocab
    tail = randint(key(seed, _TID["splice"]), extra, 0, V).astype(np.int32)
    return np.concatenate([np.asarray(query, np.int32), np.asarray(cont, np.int32), tail])


def make_prefill_tokens(wl: Workload, seed: int, n: int) -> np.ndarray:
    V = wl.model.vocab
    return zipf(key(seed, _TID["prefill_tok"]), n, V)


def case_seed(wl: Workload, case: int) -> int:
    return 1000 * wl.index + case


# tensor ids of the retrieval-key inputs
_T_KEYPROJ, _T_KEYS, _T_HID = 901, 902, 903
KEY_DIM = 256


def key_projection(hidden: int, seed: int) -> np.ndarray:
    """The fixed random projection of the retrieval keys: [KEY_DIM][hidden]
    N(0, 1) values in fp32 (exact in fp64)."""
    return normal_f32(key(seed, _T_KEYPROJ), KEY_DIM * hidden).reshape(KEY_DIM, hidden)


def random_keys(n: int, seed: int, first: int = 0) -> np.ndarray:
    """Arbitrary int8 key codes in [-127, 127], [n][KEY_DIM] (store keys for
    lookup tests and timing)."""
    return (randint(key(seed, _T_KEYS), n * KEY_DIM, -127, 128, first * KEY_DIM)
            .astype(np.int8).reshape(n, KEY_DIM))


def perturb_key(k: np.ndarray, seed: int, changes: int = 8, delta: int = 3) -> np.ndarray:
    """A near copy of key k: `changes` codes moved by up to +-delta (clipped),
    for queries that should find k's entry."""
    out = np.array(k, np.int16).reshape(-1).copy()
    kk = key(seed, _T_KEYS + 1)
    idx = randint(kk, changes, 0, out.shape[0])
    d = randint(kk, changes, -delta, delta + 1, changes)
    out[idx] = np.clip(out[idx] + d, -127, 127)
    return out.astype(np.int8)


def hidden_states(n: int, hidden: int, seed: int) -> np.ndarray:
    """Synthetic final-layer states [n][hidden], N(0, 1) in fp32."""
    return normal_f32(key(seed, _T_HID), n * hidden).reshape(n, hidden)


def bf16_bits_to_f32(a: np.ndarray) -> np.ndarray:
    return (a.astype(np.uint32) << np.uint32(16)).view(np.float32)


_T_REPLAY = 904


def replay_store(base: Store, base_keys: np.ndarray, first_token: int, outputs: np.ndarray,
                 output_keys: np.ndarray, mutate: float, seed: int, vocab: int):
    """A store that holds a prior execution of the same task (the paper's
    premise: agents repeat tasks, so earlier output sequences recur): the
    base store plus one sequence [first_token, outputs...] whose tokens past
    the second are replaced, each with probability `mutate`, by a different
    uniform token (a prior run that drifted). Entry p's key describes the
    context that produced token p: output_keys[i] for outputs[i], a zero key
    for first_token. Returns (tokens, seq_offsets, keys)."""
    seq = np.concatenate([[first_token], outputs]).astype(np.int32)
    k = key(seed, _T_REPLAY)
    n = len(seq)
    hit = uniform(k, n, first=0) < mutate
    hit[:2] = False
    repl = randint(k, n, 0, vocab - 1, first=n)
    repl = np.where(repl >= seq, repl + 1, repl)   # uniform over the other tokens
    seq = np.where(hit, repl, seq).astype(np.int32)
    keys = np.concatenate([np.zeros((1, KEY_DIM), np.int8),
                           np.asarray(output_keys, np.int8).reshape(-1, KEY_DIM)])
    tokens = np.concatenate([base.tokens, seq]).astype(np.int32)
    offs = np.concatenate([base.seq_offsets, [base.seq_offsets[-1] + n]]).astype(np.int64)
    return tokens, offs, np.concatenate([base_keys, keys]).astype(np.int8)
