"""The seeded input generators: determinism, shapes, length recipe, poison."""
import numpy as np

import workloads as W


def test_seeded_presets_are_deterministic():
    a = W.config_attn_inputs(1)
    b = W.config_attn_inputs(1)
    for f in ("q", "cu_qlens", "kv_pages", "page_table", "ctx_lens"):
        assert np.array_equal(getattr(a, f), getattr(b, f))


def test_tiny_preset_shape():
    a = W.config_attn_inputs(1)
    assert list(a.cu_qlens) == [0, 16, 21] and list(a.ctx_lens) == [37, 100]
    assert a.capacity == 32 and a.num_pages == 4 + 7
    assert a.q.shape == (32, 4, 64) and a.kv_pages.shape == (11, 2, 1, 16 * 64)
    assert a.scale == 0.125
    # every pool page is used exactly once, in a permuted order
    used = np.sort(a.page_table[a.page_table >= 0])
    assert np.array_equal(used, np.arange(11))


def test_verify_length_recipe():
    rng = np.random.default_rng(0)
    ks = np.concatenate([W.verify_lengths(rng, 32, 256) for _ in range(200)])
    assert ks.min() >= 1 and ks.max() <= 16
    # E[min(G,16)] for G ~ Geometric(0.25) is (1 - 0.75**16) / 0.25 = 3.96
    assert abs(ks.mean() - (1 - 0.75 ** 16) / 0.25) < 0.1
    tight = W.verify_lengths(np.random.default_rng(1), 16, 20)
    assert tight.sum() <= 20 and tight.min() >= 1


def test_cu_from_lengths():
    assert list(W.cu_from_lengths([6, 10, 7, 9])) == [0, 6, 16, 23, 32]
    assert list(W.cu_from_lengths([0, 3, 0])) == [0, 0, 3, 3]


def test_bf16_round_trip_and_rounding():
    x = np.array([1.0, -2.5, 3.14159, 1e-3, 65504.0], np.float32)
    b = W.bf16_bits(x)
    y = W.bf16_to_f32(b)
    assert np.all(np.abs(y - x) <= np.abs(x) * 2.0 ** -8)
    # round-to-nearest-even on an exact tie: 1 + 2^-8 lies halfway between
    # 1 and 1 + 2^-7 and rounds to the even one (1.0)
    assert W.bf16_to_f32(W.bf16_bits(np.array([1 + 2.0 ** -8], np.float32)))[0] == 1.0


def test_poison_only_where_unread():
    a = W.make_attn_inputs(np.random.default_rng(2), ctx_lens=[5, 20], qlens=[3, 1],
                           capacity=6, num_q_heads=2, num_kv_heads=1, head_dim=16,
                           spare_pages=1)
    nan = W.BF16_NAN
    assert (a.q[4:] == nan).all() and not (a.q[:4] == nan).any()
    # request 0: 8 keys in one page -> slots 8..15 dead; request 1: 21 keys
    p0 = a.page_table[0, 0]
    for s in range(16):
        koff = W.k_tile_offset(s, np.arange(16))
        dead = s >= 8
        assert ((a.kv_pages[p0, 0, 0, koff] == nan).all()) == dead
    spare = set(range(a.num_pages)) - set(a.page_table[a.page_table >= 0].tolist())
    assert len(spare) == 1 and (a.kv_pages[spare.pop()] == nan).all()


def test_planted_accept_construction():
    rng = np.random.default_rng(4)
    cu = W.cu_from_lengths([5, 0, 16, 1])
    acc = W.make_accept_inputs(rng, cu_qlens=cu, capacity=25, vocab=300)
    k = np.diff(cu)
    assert (acc.planted_accept_len <= np.maximum(k - 1, 0)).all()
    assert acc.planted_next[1] == -1 and acc.planted_accept_len[1] == 0
    assert np.isnan(acc.logits[22:]).all()


def test_repack_moves_rows_and_keeps_pool():
    a = W.make_attn_inputs(np.random.default_rng(6), ctx_lens=[3, 9, 1], qlens=[2, 4, 1],
                           capacity=8, num_q_heads=2, num_kv_heads=1, head_dim=16)
    b = W.repack(a, [2, 0, 1], capacity=12, gaps=[1, 0, 2, 1])
    assert list(np.diff(b.cu_qlens)) == [0, 1, 2, 0, 0, 4, 0]
    assert b.kv_pages is a.kv_pages
    for old_i, new_i, o_old, o_new, k in b.meta["moves"]:
        assert np.array_equal(b.q[o_new:o_new + k], a.q[o_old:o_old + k])
        assert np.array_equal(b.page_table[new_i], a.page_table[old_i])
