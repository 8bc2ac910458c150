"""Seeded input generators: determinism, page-table validity, NaN poison,
length distributions and bf16 rounding."""
import numpy as np
import pytest

import workloads as W


def test_bf16_round_to_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 3.0e-3, 65504.0], dtype=np.float32)
    bits = W.f32_to_bf16_bits(x)
    # 1 + 2^-8 is a tie -> even (1.0); 1 + 3*2^-8 is a tie -> even (1 + 2^-6... = 1 + 4*2^-8)
    assert bits[0] == 0x3F80 and bits[1] == 0x3F80 and bits[2] == 0x3F82
    back = W.bf16_bits_to_f32(bits)
    assert back[3] == -2.5
    assert abs(back[4] - 3.0e-3) <= 2 ** -8 * 3.0e-3
    assert np.array_equal(W.f32_to_bf16_bits(back), bits)


def test_quantile_normals_have_unit_moments():
    rng = np.random.Generator(np.random.PCG64(0))
    x = W.bf16_bits_to_f32(W._normal_bf16(rng, (1 << 20,))).astype(np.float64)
    assert abs(x.mean()) < 5e-3 and abs(x.std() - 1.0) < 5e-3
    y = W.bf16_bits_to_f32(W._normal_bf16(rng, (1 << 20,), 0.5)).astype(np.float64)
    assert abs(y.std() - 0.5) < 3e-3


@pytest.mark.parametrize("name", ["tiny", "llama8b"])
def test_named_workloads_deterministic(name):
    a = W.make(name)
    b = W.make(name)
    for f in ("q", "k_cache", "v_cache", "block_table", "context_lens"):
        assert np.array_equal(getattr(a, f), getattr(b, f))


def test_named_shapes():
    t = W.make("tiny")
    assert t.q.shape == (1, 8, 64) and t.k_cache.shape == (64, 16, 2, 64) and t.block_table.shape == (1, 16)
    assert t.algorithmic_bytes() == 4 * 64 * 2 * 256 + 4 * 8 * 64 + 4 * 16 + 4 == 133188
    lens = W.lengths_of("batched")
    assert lens.shape == (64,) and lens.min() >= 128 and lens.max() <= 8192
    z = W.lengths_of("ragged")
    assert z.min() >= 15 and z.max() <= 32767 and not (z % 32 == 0).any()
    assert 0.3 < (z <= 16).mean() < 0.6


def test_page_tables_valid_and_disjoint():
    w = W.build([5, 40, 16, 0, 33], 4, 2, 64, 16, seed=1, pool="holes:0.2")
    seen = set()
    for b in range(w.batch):
        n = (int(w.context_lens[b]) + 15) // 16
        row = w.block_table[b]
        assert (row[:n] >= 0).all() and (row[:n] < w.num_pages).all()
        assert (row[n:] == -1).all()
        for p in row[:n]:
            assert p not in seen
            seen.add(int(p))
    assert len(seen) < w.num_pages  # holes exist


def test_poison_marks_exactly_the_dead_slots():
    w = W.build([5, 40, 16], 4, 2, 64, 16, seed=1, pool="holes:0.2")
    kf = W.bf16_bits_to_f32(w.k_cache)
    live = np.zeros(w.k_cache.shape[:2], dtype=bool)
    for b in range(w.batch):
        for t in range(int(w.context_lens[b])):
            live[w.block_table[b, t // 16], t % 16] = True
    assert np.isfinite(kf[live]).all()
    assert np.isnan(kf[~live]).all()


def test_permute_pages_keeps_logical_kv():
    w = W.build([50, 7], 4, 2, 64, 16, seed=2, pool="holes:0.5")
    w2 = W.permute_pages(w, 9)
    for b in range(w.batch):
        for t in range(int(w.context_lens[b])):
            a = w.k_cache[w.block_table[b, t // 16], t % 16]
            c = w2.k_cache[w2.block_table[b, t // 16], t % 16]
            assert np.array_equal(a, c)


def test_variant_workloads_shapes_and_bytes():
    lens = W.lengths_of("window")
    assert (lens == 16384).all()
    w = W.build([100, 5, 0], 8, 2, 64, 16, seed=3, num_queries=3, window=10, poison=False)
    assert w.q.shape == (3, 3, 8, 64) and w.num_queries == 3 and w.window == 10
    assert w.num_q_heads == 8 and w.head_dim == 64
    # union of the visible ranges: [L - Tq + 1 - W, L) clipped at 0
    assert W.window_start(100, 3, 10) == 88 and W.window_start(5, 3, 10) == 0
    live = (100 - 88) + 5
    pages = (7 - 88 // 16) + 1
    assert w.algorithmic_bytes() == 4 * 64 * 2 * live + 4 * 3 * 3 * 8 * 64 + 4 * pages + 4 * 3


def test_window_poison_releases_whole_pages_only():
    w = W.build([100, 40], 8, 2, 64, 16, seed=4, num_queries=2, window=20)
    # sequence 0 sees tokens 79..99: pages 0..3 (tokens < 64) are released, page 4 holds 79
    assert (w.block_table[0, :4] == -1).all() and (w.block_table[0, 4:7] >= 0).all()
    page4 = w.block_table[0, 4]
    assert not np.isnan(W.bf16_bits_to_f32(w.k_cache[page4, :16])).any()   # live page: all finite
    # sequence 1 (L = 40) sees tokens 19..39: only page 0 (tokens < 16) is released
    assert w.block_table[1, 0] == -1 and (w.block_table[1, 1:3] >= 0).all()
