"""Python binding of libpf, the MI355X (gfx950) retrieval-drafted verify step.

Thin ctypes marshalling over the C ABI in ``include/pf.h``: every function
here packs arguments and calls the library; all computation runs in the HIP
kernels. torch supplies device memory (tensors) and streams. There is no CPU
fallback: importing works anywhere, but any call raises if ``libpf.so`` is
missing or no GPU is present.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpf.so")

PF_OK, PF_EINVAL, PF_ENOMEM, PF_EHIP, PF_ECAPACITY, PF_ESTATE, PF_EUNSUPPORTED = 0, -1, -2, -3, -4, -5, -6
PF_DTYPE_F32, PF_DTYPE_BF16 = 0, 1
PF_MAX_DRAFT, PF_MAX_NODES, PF_MAX_CAND, PF_MAX_TREE_NODES = 64, 65, 4, 63
PF_VSTATUS_NAN, PF_VSTATUS_CTX_FULL = 1, 2

# Device records, same layout as pf_draft / pf_verify_result in pf.h.
DRAFT_DTYPE = np.dtype([("n_nodes", "<i4"), ("tree", "<i4"), ("n_found", "<i4"),
                        ("n_eligible", "<i4"), ("token", "<i4", 65), ("parent", "<i4", 65),
                        ("depth", "<i4", 65), ("reserved0", "<i4"), ("anc", "<u8", 65),
                        ("cand_len", "<i4", 4), ("cand_pos", "<i8", 4),
                        ("cand_score", "<f4", 4)])
RESULT_DTYPE = np.dtype([("accept_len", "<i4"), ("bonus", "<i4"), ("rows", "<i4"),
                         ("status", "<i4"), ("kv_base", "<i8"), ("path", "<i4", 65),
                         ("pred", "<i4", 65), ("out_tokens", "<i4", 65), ("reserved0", "<i4")])
assert DRAFT_DTYPE.itemsize == 1384 and RESULT_DTYPE.itemsize == 808
KEY_DIM = 256

EXPORTED = ["pf_last_error", "pf_version", "pf_context_init", "pf_context_sync_bound",
            "pf_store_build", "pf_store_destroy", "pf_store_size", "pf_draft_lookup",
            "pf_model_create", "pf_model_destroy", "pf_model_bytes", "pf_kv_bytes", "pf_kv_init",
            "pf_kv_import", "pf_kv_export", "pf_kv_set_len", "pf_kv_sync_bound", "pf_verify_step",
            "pf_kv_commit", "pf_prefill", "pf_verify_step_profiled", "pf_verify_step_trace",
            "pf_verify_kernel_repeat", "pf_read_stream",
            "pf_keyproj_create",
            "pf_keyproj_destroy", "pf_key_encode", "pf_key_encode_static", "pf_store_attach_keys",
            "pf_draft_lookup_cosine", "pf_verify_query_key", "pf_verify_row_keys",
            "pf_ctl_create", "pf_ctl_destroy", "pf_ctl_get_state", "pf_ctl_set_state",
            "pf_ctl_objective", "pf_ctl_choose", "pf_ctl_observe", "pf_decode_iteration",
            "pf_kv_carry", "pf_store_reserve", "pf_store_begin_sequence", "pf_store_append",
            "pf_store_append_verified", "pf_store_appended", "pf_store_compact"]

PF_PROF_KINDS = 11
PROF_NAMES = ["setup", "qkv", "qkv_post", "attn", "o_proj", "norm", "gate_up", "down",
              "lm_head", "accept", "event_pair"]


class PfError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"pf status {status}: {msg}")
        self.status = status


class pf_context(ctypes.Structure):
    _fields_ = [("tokens", ctypes.c_void_p), ("len", ctypes.c_void_p),
                ("capacity", ctypes.c_int64), ("host_bound", ctypes.c_int64)]


class pf_kv_cache(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("len", ctypes.c_void_p), ("capacity", ctypes.c_int64),
                ("host_bound", ctypes.c_int64), ("n_layers", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("pending", ctypes.c_int32),
                ("pending_tree", ctypes.c_int32)]


class pf_model_config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("ffn", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("rope_theta", ctypes.c_double),
                ("rms_eps", ctypes.c_double)]


class pf_model_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("embed", "lm_head", "wqkv", "wo", "wgu", "wd", "attn_norm", "ffn_norm",
                 "final_norm")]


_lib = None


def lib():
    """Load libpf.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: run __graft_entry__.build() first")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        sig = {
            "pf_last_error": (ctypes.c_char_p, []),
            "pf_version": (ctypes.c_char_p, []),
            "pf_context_init": (i32, [vp, vp, vp, i64, i64, vp]),
            "pf_context_sync_bound": (i32, [vp, vp]),
            "pf_store_build": (i32, [vp, vp, i64, i32, vp, vp]),
            "pf_store_destroy": (None, [vp]),
            "pf_store_size": (i64, [vp]),
            "pf_draft_lookup": (i32, [vp, vp, i32, i32, i32, i32, vp, vp]),
            "pf_model_create": (i32, [vp, vp, vp, vp]),
            "pf_model_destroy": (None, [vp]),
            "pf_model_bytes": (i64, [vp]),
            "pf_kv_bytes": (i64, [vp, i64]),
            "pf_kv_init": (i32, [vp, vp, vp, vp, i64]),
            "pf_kv_import": (i32, [vp, vp, i64, vp]),
            "pf_kv_export": (i32, [vp, vp, i64, i64, vp]),
            "pf_kv_set_len": (i32, [vp, i64, vp]),
            "pf_kv_sync_bound": (i32, [vp, vp]),
            "pf_verify_step": (i32, [vp, vp, vp, i32, i32, vp, vp, vp]),
            "pf_kv_commit": (i32, [vp, vp, vp, vp]),
            "pf_prefill": (i32, [vp, vp, vp, i32, i32, vp, vp]),
            "pf_verify_step_profiled": (i32, [vp, vp, vp, i32, i32, vp, vp, vp, vp, vp]),
            "pf_verify_step_trace": (i32, [vp, vp, vp, i32, i32, vp, vp, vp, vp]),
            "pf_verify_kernel_repeat": (i32, [vp, vp, vp, i32, i32, i32, vp, vp]),
            "pf_read_stream": (i32, [vp, i64, vp, vp]),
            "pf_keyproj_create": (i32, [vp, i32, vp]),
            "pf_keyproj_destroy": (None, [vp]),
            "pf_key_encode": (i32, [vp, vp, i32, i64, i64, vp, vp]),
            "pf_key_encode_static": (i32, [vp, vp, i32, i64, i64, vp, vp]),
            "pf_store_attach_keys": (i32, [vp, vp, vp]),
            "pf_draft_lookup_cosine": (i32, [vp, vp, vp, i32, i32, i32, i32, vp, vp]),
            "pf_verify_query_key": (i32, [vp, vp, vp, vp, vp]),
            "pf_verify_row_keys": (i32, [vp, vp, i32, vp, vp]),
            "pf_ctl_create": (i32, [vp, vp]),
            "pf_ctl_destroy": (None, [vp]),
            "pf_ctl_get_state": (i32, [vp, vp]),
            "pf_ctl_set_state": (i32, [vp, vp]),
            "pf_ctl_objective": (i32, [vp, ctypes.c_double, i32, vp, vp]),
            "pf_ctl_choose": (i32, [vp, ctypes.c_double, i32, vp]),
            "pf_ctl_observe": (i32, [vp, i32, ctypes.c_double, i32, ctypes.c_double]),
            "pf_decode_iteration": (i32, [vp, vp, vp, vp, vp, vp, i32, i32, vp, vp, vp, vp, vp]),
            "pf_store_reserve": (i32, [vp, i64, i32, vp]),
            "pf_store_begin_sequence": (i32, [vp, vp]),
            "pf_store_append": (i32, [vp, vp, vp, vp, i32, vp]),
            "pf_store_append_verified": (i32, [vp, vp, vp, vp, vp]),
            "pf_store_appended": (i32, [vp, vp, vp]),
            "pf_store_compact": (i32, [vp, i64, vp]),
            "pf_kv_carry": (i32, [vp, vp, i32, vp, vp, vp, vp]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def last_error() -> str:
    return lib().pf_last_error().decode()


def _check(status: int) -> None:
    if status != PF_OK:
        raise PfError(status, last_error())


def _torch():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("libpf needs a ROCm GPU (torch.cuda.is_available() is False)")
    return torch


def _stream(stream=None) -> int:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


# ----------------------------------------------------------------------------
# objects
# ----------------------------------------------------------------------------

class Context:
    """Device token buffer + length of the decoding context."""

    def __init__(self, tokens: np.ndarray, capacity: int, stream=None):
        torch = _torch()
        tokens = np.asarray(tokens, np.int32)
        self.buf = torch.zeros(capacity, dtype=torch.int32, device="cuda")
        self.buf[:len(tokens)] = torch.from_numpy(tokens).cuda()
        self.len = torch.zeros(1, dtype=torch.int32, device="cuda")
        self.c = pf_context()
        pf_context_init(self, len(tokens), stream)

    def tokens(self) -> np.ndarray:
        n = int(self.len.item())
        return self.buf[:n].cpu().numpy()


def pf_context_init(ctx: Context, length: int, stream=None) -> None:
    _check(lib().pf_context_init(ctypes.byref(ctx.c), ctx.buf.data_ptr(), ctx.len.data_ptr(),
                                 ctx.buf.numel(), int(length), _stream(stream)))


def pf_context_sync_bound(ctx: Context, stream=None) -> None:
    _check(lib().pf_context_sync_bound(ctypes.byref(ctx.c), _stream(stream)))


class Store:
    def __init__(self, handle: int):
        self.h = handle

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.pf_store_destroy(self.h)
            self.h = None

    @property
    def size(self) -> int:
        return int(lib().pf_store_size(self.h))


def pf_store_build(tokens: np.ndarray, seq_offsets: np.ndarray, ngram: int, stream=None) -> Store:
    tokens = np.ascontiguousarray(tokens, np.int32)
    offs = np.ascontiguousarray(seq_offsets, np.int64)
    out = ctypes.c_void_p()
    _check(lib().pf_store_build(tokens.ctypes.data, offs.ctypes.data, len(offs) - 1, int(ngram),
                                _stream(stream), ctypes.byref(out)))
    return Store(out.value)


def pf_store_size(store: "Store") -> int:
    return int(lib().pf_store_size(store.h))


def new_draft():
    torch = _torch()
    return torch.zeros(DRAFT_DTYPE.itemsize, dtype=torch.uint8, device="cuda")


def new_result():
    torch = _torch()
    return torch.zeros(RESULT_DTYPE.itemsize, dtype=torch.uint8, device="cuda")


def read_draft(t) -> np.ndarray:
    return np.frombuffer(t.cpu().numpy().tobytes(), DRAFT_DTYPE)[0]


def read_result(t) -> np.ndarray:
    return np.frombuffer(t.cpu().numpy().tobytes(), RESULT_DTYPE)[0]


def pf_draft_lookup(store: Store, ctx: Context, k_max: int, tree: bool, n_cand: int,
                    max_nodes: int, draft, stream=None) -> None:
    _check(lib().pf_draft_lookup(store.h, ctypes.byref(ctx.c), int(k_max), int(bool(tree)),
                                 int(n_cand), int(max_nodes), draft.data_ptr(), _stream(stream)))


class pf_ctl_params(ctypes.Structure):
    _fields_ = [("l_max", ctypes.c_int32), ("explore_every", ctypes.c_int32),
                ("lr", ctypes.c_double), ("forget", ctypes.c_double),
                ("prior_var", ctypes.c_double)]


class pf_ctl_state(ctypes.Structure):
    _fields_ = [("w_first", ctypes.c_double * 3), ("w_cont", ctypes.c_double * 3),
                ("theta", ctypes.c_double * 3), ("P", ctypes.c_double * 9),
                ("n_choose", ctypes.c_int64), ("n_explore", ctypes.c_int64),
                ("n_observe", ctypes.c_int64)]


class Controller:
    """Handle of a proposal-length controller (host state in the library)."""

    def __init__(self, handle: int, l_max: int):
        self.h = handle
        self.l_max = l_max

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.pf_ctl_destroy(self.h)
            self.h = None


def pf_ctl_create(l_max: int = 64, explore_every: int = 16, lr: float = 0.05,
                  forget: float = 0.98, prior_var: float = 100.0) -> Controller:
    p = pf_ctl_params(int(l_max), int(explore_every), float(lr), float(forget), float(prior_var))
    out = ctypes.c_void_p()
    _check(lib().pf_ctl_create(ctypes.byref(p), ctypes.byref(out)))
    return Controller(out.value, int(l_max))


def pf_ctl_get_state(ctl: Controller) -> pf_ctl_state:
    st = pf_ctl_state()
    _check(lib().pf_ctl_get_state(ctl.h, ctypes.byref(st)))
    return st


def pf_ctl_set_state(ctl: Controller, st: pf_ctl_state) -> None:
    _check(lib().pf_ctl_set_state(ctl.h, ctypes.byref(st)))


def pf_ctl_objective(ctl: Controller, s: float, avail: int):
    """(objective values for l = 0..L as an array, argmin)."""
    L = max(0, min(ctl.l_max, int(avail)))
    out = np.zeros(L + 1, np.float64)
    best = ctypes.c_int32()
    _check(lib().pf_ctl_objective(ctl.h, float(s), int(avail), out.ctypes.data, ctypes.byref(best)))
    return out, int(best.value)


def pf_ctl_choose(ctl: Controller, s: float, avail: int) -> int:
    l = ctypes.c_int32()
    _check(lib().pf_ctl_choose(ctl.h, float(s), int(avail), ctypes.byref(l)))
    return int(l.value)


def pf_ctl_observe(ctl: Controller, l: int, s: float, accepted: int, latency_ms: float) -> None:
    _check(lib().pf_ctl_observe(ctl.h, int(l), float(s), int(accepted), float(latency_ms)))


class pf_iteration(ctypes.Structure):
    _fields_ = [("n_found", ctypes.c_int32), ("avail", ctypes.c_int32), ("l", ctypes.c_int32),
                ("accepted", ctypes.c_int32), ("bonus", ctypes.c_int32),
                ("status", ctypes.c_int32), ("s", ctypes.c_double), ("ms", ctypes.c_double)]


def pf_decode_iteration(model: "Model", kv: "KVCache", ctx: "Context", store: "Store",
                        kp: "KeyProj", ctl: Optional[Controller], l_fixed: int, qkey, draft,
                        result, append: bool = False, stream=None) -> dict:
    it = pf_iteration()
    _check(lib().pf_decode_iteration(model.h, ctypes.byref(kv.c), ctypes.byref(ctx.c), store.h,
                                     kp.h, ctl.h if ctl is not None else None, int(l_fixed),
                                     int(bool(append)), qkey.data_ptr(), draft.data_ptr(),
                                     result.data_ptr(), ctypes.byref(it), _stream(stream)))
    return {k: getattr(it, k) for k, _ in pf_iteration._fields_}


class KeyProj:
    """Device copy of the fixed random projection of the retrieval keys."""

    def __init__(self, handle: int, hidden: int):
        self.h = handle
        self.hidden = hidden

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.pf_keyproj_destroy(self.h)
            self.h = None


def pf_keyproj_create(R: np.ndarray) -> KeyProj:
    R = np.ascontiguousarray(R, np.float32)
    assert R.ndim == 2 and R.shape[0] == KEY_DIM
    out = ctypes.c_void_p()
    _check(lib().pf_keyproj_create(R.ctypes.data, int(R.shape[1]), ctypes.byref(out)))
    return KeyProj(out.value, int(R.shape[1]))


def pf_key_encode(kp: KeyProj, h, keys, stream=None) -> None:
    """h: device tensor [n][ld] (float32 or bfloat16); keys: device int8 [n][KEY_DIM]."""
    torch = _torch()
    dt = {torch.float32: PF_DTYPE_F32, torch.bfloat16: PF_DTYPE_BF16}[h.dtype]
    assert h.dim() == 2 and h.stride(1) == 1 and keys.dtype == torch.int8
    assert keys.shape == (h.shape[0], KEY_DIM) and keys.is_contiguous()
    _check(lib().pf_key_encode(kp.h, h.data_ptr(), dt, int(h.stride(0)), int(h.shape[0]),
                               keys.data_ptr(), _stream(stream)))


def pf_key_encode_static(kp: KeyProj, h, keys, stream=None) -> None:
    """pf_key_encode through the library's static projection buffer (no
    allocation); same arguments."""
    torch = _torch()
    dt = {torch.float32: PF_DTYPE_F32, torch.bfloat16: PF_DTYPE_BF16}[h.dtype]
    assert h.dim() == 2 and h.stride(1) == 1 and keys.dtype == torch.int8
    assert keys.shape == (h.shape[0], KEY_DIM) and keys.is_contiguous()
    _check(lib().pf_key_encode_static(kp.h, h.data_ptr(), dt, int(h.stride(0)), int(h.shape[0]),
                                      keys.data_ptr(), _stream(stream)))


def pf_store_attach_keys(store: "Store", keys: np.ndarray, stream=None) -> None:
    keys = np.ascontiguousarray(keys, np.int8)
    assert keys.shape == (store.size, KEY_DIM)
    _check(lib().pf_store_attach_keys(store.h, keys.ctypes.data, _stream(stream)))


def pf_store_reserve(store: "Store", capacity: int, max_seqs: int, stream=None) -> None:
    _check(lib().pf_store_reserve(store.h, int(capacity), int(max_seqs), _stream(stream)))


def pf_store_begin_sequence(store: "Store", stream=None) -> None:
    _check(lib().pf_store_begin_sequence(store.h, _stream(stream)))


def pf_store_append(store: "Store", tokens, keys, n_dev, n_max: int, stream=None) -> None:
    _check(lib().pf_store_append(store.h, tokens.data_ptr(), keys.data_ptr(), n_dev.data_ptr(),
                                 int(n_max), _stream(stream)))


def pf_store_append_verified(store: "Store", model: "Model", kp: "KeyProj", result,
                             stream=None) -> None:
    _check(lib().pf_store_append_verified(store.h, model.h, kp.h, result.data_ptr(),
                                          _stream(stream)))


def pf_store_appended(store: "Store", stream=None) -> int:
    n = ctypes.c_int64()
    _check(lib().pf_store_appended(store.h, _stream(stream), ctypes.byref(n)))
    return int(n.value)


def pf_store_compact(store: "Store", budget: int = 0, stream=None) -> None:
    _check(lib().pf_store_compact(store.h, int(budget), _stream(stream)))


def pf_draft_lookup_cosine(store: "Store", ctx: Context, qkey, k_max: int, tree: bool, n_cand: int,
                           max_nodes: int, draft, stream=None) -> None:
    """qkey: device int8 [KEY_DIM] (the query state's key)."""
    _check(lib().pf_draft_lookup_cosine(store.h, ctypes.byref(ctx.c), qkey.data_ptr(), int(k_max),
                                        int(bool(tree)), int(n_cand), int(max_nodes),
                                        draft.data_ptr(), _stream(stream)))


def pf_verify_query_key(model: "Model", kp: KeyProj, result, qkey, stream=None) -> None:
    _check(lib().pf_verify_query_key(model.h, kp.h, result.data_ptr(), qkey.data_ptr(),
                                     _stream(stream)))


def pf_verify_row_keys(model: "Model", kp: KeyProj, rows: int, keys, stream=None) -> None:
    _check(lib().pf_verify_row_keys(model.h, kp.h, int(rows), keys.data_ptr(), _stream(stream)))


class Model:
    def __init__(self, handle: int, cfg: pf_model_config):
        self.h = handle
        self.cfg = cfg

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.pf_model_destroy(self.h)
            self.h = None

    @property
    def bytes(self) -> int:
        return int(lib().pf_model_bytes(self.h))


def model_config(shape) -> pf_model_config:
    """pf_model_config from a shape object with the synth.ModelShape fields."""
    return pf_model_config(shape.n_layers, shape.hidden, shape.n_heads, shape.n_kv_heads,
                           shape.head_dim, shape.ffn, shape.vocab,
                           PF_DTYPE_BF16 if shape.dtype == "bf16" else PF_DTYPE_F32,
                           float(shape.rope_theta), float(shape.rms_eps))


def pf_model_create(cfg: pf_model_config, weights: Dict[str, "object"], stream=None) -> Model:
    """weights: device tensors named embed, lm_head, wqkv, wo, wgu, wd,
    attn_norm, ffn_norm, final_norm in the layouts of pf_model_weights."""
    w = pf_model_weights(*[_ptr(weights[k]) for k in
                           ("embed", "lm_head", "wqkv", "wo", "wgu", "wd", "attn_norm",
                            "ffn_norm", "final_norm")])
    out = ctypes.c_void_p()
    _check(lib().pf_model_create(ctypes.byref(cfg), ctypes.byref(w), _stream(stream),
                                 ctypes.byref(out)))
    return Model(out.value, cfg)


class KVCache:
    def __init__(self, model: Model, capacity: int):
        torch = _torch()
        nbytes = int(lib().pf_kv_bytes(model.h, capacity))
        if nbytes < 0:
            raise PfError(PF_EINVAL, "pf_kv_bytes failed")
        self.data = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        self.len = torch.zeros(1, dtype=torch.int32, device="cuda")
        self.c = pf_kv_cache()
        _check(lib().pf_kv_init(ctypes.byref(self.c), model.h, self.data.data_ptr(),
                                self.len.data_ptr(), int(capacity)))


def pf_kv_import(kv: KVCache, src, n: int, stream=None) -> None:
    _check(lib().pf_kv_import(ctypes.byref(kv.c), _ptr(src), int(n), _stream(stream)))


def pf_kv_export(kv: KVCache, dst, start: int, n: int, stream=None) -> None:
    _check(lib().pf_kv_export(ctypes.byref(kv.c), dst.data_ptr(), int(start), int(n),
                              _stream(stream)))


def pf_kv_set_len(kv: KVCache, n: int, stream=None) -> None:
    _check(lib().pf_kv_set_len(ctypes.byref(kv.c), int(n), _stream(stream)))


def pf_kv_carry(kv: KVCache, model: "Model", spans, stream=None) -> None:
    """spans: sequence of (src, dst, len) slot spans, applied in order."""
    sp = np.asarray(spans, np.int64).reshape(-1, 3)
    src, dst, ln = (np.ascontiguousarray(sp[:, i]) for i in range(3))
    _check(lib().pf_kv_carry(ctypes.byref(kv.c), model.h, len(sp), src.ctypes.data,
                             dst.ctypes.data, ln.ctypes.data, _stream(stream)))


def pf_kv_sync_bound(kv: KVCache, stream=None) -> None:
    _check(lib().pf_kv_sync_bound(ctypes.byref(kv.c), _stream(stream)))


def pf_verify_step(model: Model, kv: KVCache, draft, rows: int, tree: bool, logits, result,
                   stream=None) -> None:
    _check(lib().pf_verify_step(model.h, ctypes.byref(kv.c), draft.data_ptr(), int(rows),
                                int(bool(tree)), _ptr(logits), result.data_ptr(),
                                _stream(stream)))


def pf_verify_step_trace(model: Model, kv: KVCache, draft, rows: int, tree: bool, logits, result,
                         resid, stream=None) -> None:
    """pf_verify_step plus the residual stream after every layer into resid
    (device fp32 [n_layers + 1][rows][hidden])."""
    _check(lib().pf_verify_step_trace(model.h, ctypes.byref(kv.c), draft.data_ptr(), int(rows),
                                      int(bool(tree)), _ptr(logits), result.data_ptr(),
                                      _ptr(resid), _stream(stream)))


def pf_verify_kernel_repeat(model: Model, kv: KVCache, draft, rows: int, tree: bool, kind: int,
                            result, stream=None) -> None:
    """Only the launches of one profiling kind of a verify step (benchmark)."""
    _check(lib().pf_verify_kernel_repeat(model.h, ctypes.byref(kv.c), draft.data_ptr(), int(rows),
                                         int(bool(tree)), int(kind), result.data_ptr(),
                                         _stream(stream)))


def pf_read_stream(buf, sink, stream=None) -> None:
    """Plain streaming read of a device tensor (benchmark calibration)."""
    nbytes = buf.numel() * buf.element_size()
    _check(lib().pf_read_stream(_ptr(buf), int(nbytes), _ptr(sink), _stream(stream)))


def pf_verify_step_profiled(model: Model, kv: KVCache, draft, rows: int, tree: bool, logits,
                            result, stream=None):
    """Returns (ms per kernel kind, launches per kind) for one verify step."""
    ms = np.zeros(PF_PROF_KINDS, np.float64)
    cnt = np.zeros(PF_PROF_KINDS, np.int32)
    _check(lib().pf_verify_step_profiled(model.h, ctypes.byref(kv.c), draft.data_ptr(), int(rows),
                                         int(bool(tree)), _ptr(logits), result.data_ptr(),
                                         _stream(stream), ms.ctypes.data, cnt.ctypes.data))
    return ms, cnt


def pf_kv_commit(kv: KVCache, result, ctx: Optional[Context], stream=None) -> None:
    _check(lib().pf_kv_commit(ctypes.byref(kv.c), result.data_ptr(),
                              ctypes.byref(ctx.c) if ctx is not None else None, _stream(stream)))


def pf_prefill(model: Model, kv: KVCache, tokens, n: int, chunk: int, logits_last=None,
               stream=None) -> None:
    _check(lib().pf_prefill(model.h, ctypes.byref(kv.c), tokens.data_ptr(), int(n), int(chunk),
                            _ptr(logits_last), _stream(stream)))


# ----------------------------------------------------------------------------
# host arrays -> device tensors in the pf_model_weights layouts
# ----------------------------------------------------------------------------

def weights_to_device(w: Dict[str, np.ndarray], dtype: str) -> Dict[str, "object"]:
    """Copy host weights (bf16 bit patterns as uint16, or fp32) to the GPU."""
    torch = _torch()
    out = {}
    for k, v in w.items():
        v = np.ascontiguousarray(v)
        if v.dtype == np.uint16:
            t = torch.from_numpy(v.view(np.int16)).cuda().view(torch.bfloat16)
        else:
            t = torch.from_numpy(v.astype(np.float32, copy=False)).cuda()
        out[k] = t
    return out


def array_to_device(a: np.ndarray):
    torch = _torch()
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(a).cuda()
