"""Pins of the benchmark's accounting against totals worked out by hand from
the workload shapes (not from the formulas under test): the algorithmic HBM
bytes of one verify step (every weight once, the KV prefix read, the draft
rows' K/V read and written) and the algorithmic FLOPs of the carry-forward
prefill (every linear layer once per new token, causal attention over the
reused prefix and the earlier new tokens)."""
import importlib.util
import os

import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _hand_bytes(L, H, nq, nkv, hd, F, V, P, M):
    # bf16: QKV (H x (q + 2 kv)), O (q x H), gate, up, down (3 x H x F) per
    # layer, the LM head (V x H), fp32 norm gains, the embedding rows read
    # for M tokens; K/V of the prefix read and of M rows read and written
    q, kv = nq * hd, nkv * hd
    weights = 2 * (L * (H * (q + 2 * kv) + q * H + 3 * H * F) + V * H)
    return weights, 2 * 2 * L * kv * (P + M) + 2 * 2 * L * kv * M


@pytest.mark.parametrize("name,total_gb", [("3b", 6.324), ("7b", 14.614), ("3b_tree", 6.326)])
def test_verify_bytes_match_the_hand_totals(name, total_gb):
    wl = synth.WORKLOADS[name]
    m = wl.model
    w, kvb = _hand_bytes(m.n_layers, m.hidden, m.n_heads, m.n_kv_heads, m.head_dim, m.ffn,
                         m.vocab, wl.prefix, wl.rows)
    got = wl.verify_bytes()
    # the accounting may add the small per-layer norm gains and embedding
    # rows on top of the matrices; nothing larger
    assert 0 <= got - (w + kvb) < 2e6, (got, w + kvb)
    assert abs(got / 1e9 - total_gb) < 0.0015, got


def test_prefill_flops_match_the_hand_total():
    b = _bench()
    wl = synth.WORKLOADS["7b_carry"]
    # 7B widths: linear 2 * 2048 tokens * 28 layers * (3584 * (3584 + 1024) +
    # 3584 * 3584 + 3 * 3584 * 18944); attention 4 * 28 * 28 * 128 * keys with
    # keys = 2048 * 6144 + 2048 * 2049 / 2
    linear = 2.0 * 2048 * 28 * (3584 * 4608 + 3584 * 3584 + 3 * 3584 * 18944)
    attn = 4.0 * 28 * 28 * 128 * (2048 * 6144 + 2048 * 2049 / 2)
    assert abs(linear / 1e12 - 26.73) < 0.01 and abs(attn / 1e12 - 5.89) < 0.01
    assert b.prefill_flops(wl) == pytest.approx(linear + attn, rel=1e-12)
