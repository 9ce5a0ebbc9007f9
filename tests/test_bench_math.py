"""The bench's algorithmic byte and flop counts on hand-worked cases (CPU).

These counts are the numerators of every bandwidth and roofline figure the
bench reports, so they are pinned against values computed by hand here."""
import numpy as np

import bench
import workloads as W


def small_case():
    # request 0: 10 context keys + a 3-row block; request 1: a sentinel
    rng = np.random.default_rng(0)
    return W.make_attn_inputs(rng, ctx_lens=[10, 0], qlens=[3, 0], capacity=5,
                              num_q_heads=4, num_kv_heads=2, head_dim=64)


def test_attention_bytes_by_hand():
    a = small_case()
    kv = 13 * 2 * 64 * 2 * 2        # 13 visible keys, 2 KV heads, K and V, bf16
    qo = 3 * 4 * 64 * 2 * 2         # 3 live rows, 4 q heads, q read + out written
    meta = (3 + 2 + 1) * 4          # offsets [B+1], contexts [B], one page id
    assert bench.attention_bytes(a, 2, 4, 64) == kv + qo + meta == 9752


def test_attention_flops_by_hand():
    a = small_case()
    # rows see 11, 12 and 13 keys; q.k and p.v are 2*D flops each per key
    assert bench.attention_flops(a, 4, 64) == (11 + 12 + 13) * 4 * 4 * 64 == 36864


def test_accept_bytes_by_hand():
    a = small_case()
    acc = W.make_accept_inputs(np.random.default_rng(1), cu_qlens=a.cu_qlens, capacity=5,
                               vocab=1000, dtype="bf16", p_accept=0.3)
    # 3 live logit rows, their draft tokens, offsets, and two int outputs per request
    assert bench.accept_bytes(acc, 2) == 3 * 1000 * 2 + 3 * 4 + 3 * 4 + 2 * 2 * 4


def test_config4_bytes_in_expected_range():
    # the seeded batch reads about 0.55 GB; the expectation over the context
    # and length distributions is about 0.61 GB
    a = W.config_attn_inputs(4, poison=False)
    b = bench.attention_bytes(a, 8, 32, 128)
    assert 0.45e9 < b < 0.70e9


def test_cpu_threads_is_bounded(monkeypatch):
    monkeypatch.setenv("OMP_NUM_THREADS", "16")
    assert 1 <= bench.cpu_threads() <= 16
    monkeypatch.setenv("OMP_NUM_THREADS", "100000")
    assert bench.cpu_threads() <= (__import__("os").cpu_count() or 1)


def test_row_padding_eq2_by_hand():
    # k = 16, 5, 1 live (and a sentinel) at G = 4: the paper's tiles hold k
    # rows per head, the live-row tiles hold 4k rows (64, 20, 4 -> 4, 2, 1
    # tiles of 16)
    p = bench.row_padding([16, 5, 0, 1], 4)
    assert p["paper_128_row_tiles"] == round(1 - 22 / 384, 4)
    assert p["paper_16_row_tiles"] == round(1 - 22 / 48, 4)
    assert p["live_row_mfma_tiles"] == round(1 - 88 / 112, 4)
    # a full block leaves no padding at tile height 16
    assert bench.row_padding([16], 1)["paper_16_row_tiles"] == 0.0
