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
