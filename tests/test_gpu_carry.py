"""GPU parity of the rolling-image KV-state carryover (Section 3.4) through
pf_kv_carry: retained spans move, keys are re-rotated by R(m') R(m)^-1,
values move unchanged, spans apply in order (memmove semantics when a span
overlaps its own source).

Bar: values and every slot a span does not write are bit-exact; keys match
the oracle's fp64 re-rotation rounded to the cache dtype (bf16: at most one
ulp apart and equal except where the fp32 rotation sits within rounding of
a bf16 tie; fp32: within 1e-6 of the row's largest magnitude). The last test
chains a carry with the prefill of the new tokens and compares logits."""
import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pf():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_32166_amd as pf
    pf.lib()
    return pf


def _setup(pf, name, layers, cap, seed):
    wl = synth.WORKLOADS[name]
    shape = wl.model if layers is None else wl.model.with_layers(layers)
    w = synth.make_weights(shape, seed)
    model = pf.pf_model_create(pf.model_config(shape), pf.weights_to_device(w, shape.dtype))
    kv = pf.KVCache(model, cap)
    host = synth.make_kv_prefix(shape, seed, cap)
    pf.pf_kv_import(kv, pf.array_to_device(host), cap)
    return shape, w, model, kv, host


def _as_f64(shape, a):
    if shape.dtype == "bf16":
        return synth.bf16_bits_to_f32(a).astype(np.float64)
    return a.astype(np.float64)


def _export(pf, kv, shape, cap):
    import torch
    dt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    buf = torch.zeros(shape.n_layers, 2, shape.n_kv_heads, cap, shape.head_dim, dtype=dt,
                      device="cuda")
    pf.pf_kv_export(kv, buf, 0, cap)
    torch.cuda.synchronize()
    return buf.to(torch.float64).cpu().numpy()


def _bf16_round(x):
    import torch
    return torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()


def _rotations(spans, cap):
    """How many re-rotations the content of each slot went through."""
    cnt = np.zeros(cap, np.int64)
    for src, dst, n in spans:
        if src != dst and n:
            c = cnt[src:src + n].copy()
            cnt[dst:dst + n] = c + 1
    return cnt


def _check(shape, got, ref, before, written, cnt):
    # values and unwritten slots exact
    assert np.array_equal(got[:, 1], ref[:, 1])
    keep = np.ones(got.shape[3], bool)
    keep[written] = False
    assert np.array_equal(got[:, :, :, keep], before[:, :, :, keep])
    gk, rk = got[:, 0][:, :, written], ref[:, 0][:, :, written]
    if gk.size == 0:
        return
    c = cnt[written][None, None, :, None].astype(np.float64)
    h = rk.shape[-1] // 2
    pair = np.maximum(np.abs(rk[..., :h]), np.abs(rk[..., h:]))
    pair = np.concatenate([pair, pair], axis=-1)
    if shape.dtype == "bf16":
        # each re-rotation rounds the pair to bf16 (half an ulp of its larger
        # element, spread over both by the next rotation)
        want = _bf16_round(rk)
        bound = np.maximum(np.abs(want) * 2.0 ** -7, c * pair * 2.0 ** -8) + 1e-38
        assert (np.abs(gk - want) <= bound).all(), np.abs(gk - want).max()
        once = cnt[written] == 1
        assert (gk[:, :, once] != want[:, :, once]).mean() < 1e-3
    else:
        assert (np.abs(gk - rk) <= 1e-6 * c * pair + 1e-30).all()


CASES = [
    ("left", [(100, 20, 60)]),
    ("right_overlap", [(10, 13, 50)]),
    ("left_overlap", [(40, 33, 70)]),
    ("rolling_window", [(120, 60, 60), (180, 120, 60)]),
    ("zero_and_empty", [(5, 5, 30), (7, 200, 0)]),
    ("to_the_end", [(0, 192, 64)]),
    ("odd_distances", [(50, 121, 30), (150, 3, 45), (201, 0, 1)]),
]


@pytest.mark.parametrize("name,layers", [("tiny", None), ("3b", 2)])
@pytest.mark.parametrize("label,spans", CASES, ids=[c[0] for c in CASES])
def test_carry_matches_oracle(pf, name, layers, label, spans):
    cap = 256
    shape, _, model, kv, host = _setup(pf, name, layers, cap, 77)
    before = _as_f64(shape, host)
    pf.pf_kv_carry(kv, model, spans)
    got = _export(pf, kv, shape, cap)
    ref = oracle.kv_carry(before, spans, shape.rope_theta)
    written = sorted({d + i for s, d, n in spans if s != d for i in range(n)})
    _check(shape, got, ref, before, np.array(written, np.int64), _rotations(spans, cap))
    assert int(kv.len.item()) == cap   # the length is not changed


def test_carry_argument_errors(pf):
    cap = 128
    shape, _, model, kv, _ = _setup(pf, "tiny", None, cap, 78)
    for spans in ([(0, 100, 40)], [(-1, 0, 4)], [(0, 0, -2)], [(120, 0, 16)]):
        with pytest.raises(pf.PfError) as e:
            pf.pf_kv_carry(kv, model, spans)
        assert e.value.status == -1


def test_rolling_window_step_with_prefill(pf):
    """One agent step with a rolling image window, tiny fp32 model: the cache
    holds [prefix | img1 | img2 | text]; the next prompt keeps the prefix,
    drops img1, keeps img2 at img1's place and adds new text. The carried
    cache plus the prefill of the new text gives the oracle's logits for the
    same carry and prefill (the oracle computing its own first step)."""
    import torch
    wl = synth.WORKLOADS["tiny"]
    shape = wl.model
    seed = 79
    w = synth.make_weights(shape, seed)
    P0, n_img, n_txt = 32, 24, 8
    kv0 = synth.make_kv_prefix(shape, seed, P0)
    rng = np.random.default_rng(seed)
    step1 = rng.integers(0, shape.vocab, 2 * n_img + n_txt).astype(np.int32)
    step2 = rng.integers(0, shape.vocab, n_txt).astype(np.int32)
    cap = 128
    model = pf.pf_model_create(pf.model_config(shape), pf.weights_to_device(w, shape.dtype))
    kv = pf.KVCache(model, cap)
    pf.pf_kv_import(kv, pf.array_to_device(kv0), P0)
    pf.pf_prefill(model, kv, torch.from_numpy(step1).cuda(), len(step1), 16)
    span = (P0 + n_img, P0, n_img)
    pf.pf_kv_carry(kv, model, [span])
    pf.pf_kv_set_len(kv, P0 + n_img)
    logits = torch.zeros(shape.vocab, device="cuda")
    pf.pf_prefill(model, kv, torch.from_numpy(step2).cuda(), n_txt, 16, logits)
    torch.cuda.synchronize()
    got = logits.cpu().numpy()

    om = oracle.Model(shape, w)
    s1 = oracle.prefill(om, kv0, step1, 16)
    full = np.concatenate([kv0.astype(np.float64), s1["kv_new"]], axis=3)
    carried = oracle.kv_carry(full, [span], shape.rope_theta)[:, :, :, :P0 + n_img]
    # the oracle reads a cached prefix in the cache's storage type (fp32 here)
    ref = oracle.prefill(om, carried.astype(np.float32), step2, 16)["logits_last"]
    assert np.isfinite(got).all() and np.isfinite(ref).all()
    err = np.abs(got - ref).max() / np.abs(ref).max()
    assert err < 1e-4, err
