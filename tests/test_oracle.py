"""Pins of the fp64 oracle against facts that do not come from the oracle:
closed forms, invariants, a library routine, brute force with exactly rounded
sums.  Each is chosen so that a plausible slip in the oracle (wrong head
mapping, wrong page/slot index, dropped scale, missing max shift, off-by-one
length, transposed operand) fails at least one of them."""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from _golden import cases as golden_cases


def small(lengths, hq=8, hkv=2, d=64, p=16, seed=11, **kw):
    return W.build(lengths, hq, hkv, d, p, seed, **kw)


def run(w):
    return oracle.attend(w.q, w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale)


def flat_gather_dense(w):
    """Independent gather: flat token index page*P + slot into the pool
    reshaped to [N*P, Hkv, D]; returns per-sequence contiguous K, V with kv
    heads repeated G times ([L, Hq, D] fp64)."""
    n, p, hkv, d = w.k_cache.shape
    g = w.num_q_heads // hkv
    kf = W.bf16_bits_to_f32(w.k_cache).astype(np.float64).reshape(n * p, hkv, d)
    vf = W.bf16_bits_to_f32(w.v_cache).astype(np.float64).reshape(n * p, hkv, d)
    res = []
    for b in range(w.batch):
        L = int(w.context_lens[b])
        idx = np.array([int(w.block_table[b, t // p]) * p + (t % p) for t in range(L)], dtype=np.int64)
        res.append((np.repeat(kf[idx], g, axis=1), np.repeat(vf[idx], g, axis=1)))
    return res


# ---------------------------------------------------------------- closed forms
@pytest.mark.parametrize("name,w,expected", golden_cases(), ids=lambda x: x if isinstance(x, str) else "")
def test_golden_closed_forms(name, w, expected):
    out, _ = run(w)
    np.testing.assert_allclose(out, expected, rtol=0, atol=1e-14)


def test_length_one_returns_v_exactly():
    w = small([1, 1, 1], hq=8, hkv=2)
    out, lse = run(w)
    g = w.num_q_heads // w.num_kv_heads
    for b in range(w.batch):
        page = w.block_table[b, 0]
        for h in range(w.num_q_heads):
            v0 = oracle.bf16_to_f64(w.v_cache[page, 0, h // g])
            assert np.array_equal(out[b, h], v0)


def test_constant_v_returns_constant():
    w = small([37, 300, 16], hq=8, hkv=2)
    consts = np.array([1.5, -2.25], dtype=np.float32)
    live = ~np.isnan(W.bf16_bits_to_f32(w.v_cache))
    for g in range(2):
        vg = w.v_cache[:, :, g, :]
        vg[live[:, :, g, :]] = W.f32_to_bf16_bits(consts[g:g + 1])[0]
    out, _ = run(w)
    for h in range(8):
        np.testing.assert_allclose(out[:, h, :], consts[h // 4], rtol=1e-13, atol=0)


def test_zero_query_gives_mean_of_values():
    w = small([5, 129, 64], hq=4, hkv=4, d=128)
    w.q[:] = 0
    out, lse = run(w)
    dense = flat_gather_dense(w)
    for b in range(w.batch):
        _, vd = dense[b]
        np.testing.assert_allclose(out[b], vd.mean(axis=0), rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse[b], math.log(int(w.context_lens[b])), rtol=1e-14)


def test_weights_sum_to_one():
    w = small([200, 17], hq=8, hkv=2)
    for b in range(2):
        for h in range(8):
            wt = oracle.weights(w.q, w.k_cache, w.block_table, w.context_lens, w.scale, b, h)
            assert wt.shape == (int(w.context_lens[b]),)
            assert abs(wt.sum() - 1.0) < 1e-12
            assert (wt >= 0).all()


def test_page_permutation_invariance_bitwise():
    w = small([100, 257, 33], hq=8, hkv=2, pool="holes:0.3")
    w2 = W.permute_pages(w, seed=5)
    assert not np.array_equal(w.block_table, w2.block_table)
    a, la = run(w)
    b, lb = run(w2)
    assert np.array_equal(a, b) and np.array_equal(la, lb)


def test_brute_force_dense_independent_gather():
    w = small([1, 15, 16, 17, 200], hq=12, hkv=3, d=64, p=16, pool="holes:0.2")
    out, lse = run(w)
    dense = flat_gather_dense(w)
    sigma = float(np.float32(w.scale))
    qf = W.bf16_bits_to_f32(w.q).astype(np.float64)
    for b in range(w.batch):
        kd, vd = dense[b]
        s = sigma * np.einsum("hd,thd->ht", qf[b], kd)
        mx = s.max(axis=1, keepdims=True)
        ex = np.exp(s - mx)
        ref = np.einsum("ht,thd->hd", ex, vd) / ex.sum(axis=1)[:, None]
        np.testing.assert_allclose(out[b], ref, rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse[b], (mx[:, 0] + np.log(ex.sum(axis=1))), rtol=1e-13)


def test_matches_torch_sdpa_fp64():
    w = small([300, 1, 64, 65], hq=32, hkv=8, d=128, p=16, scale=0.0883883)
    out, _ = run(w)
    dense = flat_gather_dense(w)
    qf = torch.from_numpy(W.bf16_bits_to_f32(w.q).astype(np.float64))
    for b in range(w.batch):
        kd, vd = dense[b]
        qq = qf[b][:, None, :]                                     # [Hq, 1, D]
        kk = torch.from_numpy(kd).permute(1, 0, 2).contiguous()    # [Hq, L, D]
        vv = torch.from_numpy(vd).permute(1, 0, 2).contiguous()
        ref = torch.nn.functional.scaled_dot_product_attention(
            qq, kk, vv, scale=float(np.float32(w.scale)))[:, 0, :].numpy()
        np.testing.assert_allclose(out[b], ref, rtol=0, atol=1e-12)


def test_split_merge_identity_any_chunking():
    w = small([1, 2, 97, 400], hq=8, hkv=2, d=64, p=16)
    ref, _ = run(w)
    rng = np.random.default_rng(3)
    for trial in range(6):
        bounds = []
        for L in w.context_lens:
            L = int(L)
            cuts = sorted(rng.integers(0, L + 1, size=rng.integers(0, 6)).tolist())
            if trial == 0:
                cuts = list(range(1, L))               # size-1 chunks
            bounds.append([0] + cuts + [L] + ([L] if trial == 1 else []))  # incl. empty tail chunk
        got = oracle.split_merge(w.q, w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale, bounds)
        np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_gqa_mapping_probe():
    # V of kv head g is the constant g: out[b, h] must be h // G (consecutive
    # query heads share a kv head; h % Hkv would give a different pattern)
    w = small([50, 3], hq=8, hkv=2, d=64)
    live = ~np.isnan(W.bf16_bits_to_f32(w.v_cache))
    for g in range(2):
        vg = w.v_cache[:, :, g, :]
        vg[live[:, :, g, :]] = W.f32_to_bf16_bits(np.float32([g]))[0]
    out, _ = run(w)
    for h in range(8):
        np.testing.assert_allclose(out[:, h, :], h // 4, rtol=0, atol=1e-13)


def test_dominant_token_no_overflow():
    # k_t* = 128 q gives a score near 1e3 for that token; the output must be
    # v_t* and finite (a missing max shift overflows exp)
    w = small([300], hq=2, hkv=2, d=64, scale=1.0 / 8)
    q = W.bf16_bits_to_f32(w.q)
    t_star = 123
    page, slot = w.block_table[0, t_star // 16], t_star % 16
    for g in range(2):
        w.k_cache[page, slot, g] = W.f32_to_bf16_bits(q[0, g] * 128)
    out, lse = run(w)
    assert np.isfinite(out).all() and np.isfinite(lse).all()
    sc = float(np.float32(w.scale)) * (W.bf16_bits_to_f32(w.k_cache[page, slot, 0]).astype(np.float64)
                                        @ q[0, 0].astype(np.float64))
    assert sc > 710  # exp(710) overflows fp64
    for g in range(2):
        np.testing.assert_allclose(out[0, g], oracle.bf16_to_f64(w.v_cache[page, slot, g]), rtol=0, atol=1e-12)


def test_nan_poison_is_never_read():
    a = small([33, 16, 100], hq=8, hkv=2, pool="holes:0.25", poison=True, seed=21)
    b = small([33, 16, 100], hq=8, hkv=2, pool="holes:0.25", poison=False, seed=21)
    assert np.isnan(W.bf16_bits_to_f32(a.k_cache)).any()
    oa, la = run(a)
    ob, lb = run(b)
    assert np.array_equal(oa, ob) and np.array_equal(la, lb)


def test_empty_sequence_gives_zero_row():
    w = small([0, 20, 0], hq=4, hkv=2, d=64)
    out, lse = run(w)
    assert np.array_equal(out[0], np.zeros_like(out[0])) and np.isneginf(lse[0]).all()
    assert np.array_equal(out[2], np.zeros_like(out[2]))
    assert np.abs(out[1]).sum() > 0


def test_brute_force_fsum_tiny():
    w = W.build([1, 5, 3], 4, 2, 8, 2, seed=9, pool="holes:0.5")
    out, _ = run(w)
    bf = np.array(oracle.brute_force_tiny(w.q, w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale))
    np.testing.assert_allclose(out, bf, rtol=0, atol=1e-15)


def test_attend_pairs_matches_full():
    w = small([70, 5], hq=8, hkv=2)
    out, lse = run(w)
    res = oracle.attend_pairs(w.q, w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale,
                              [(1, 1), (0, 0)])
    assert np.array_equal(res[(1, 1)][0], out[1, 4:8]) and np.array_equal(res[(0, 0)][1], lse[0, 0:4])


# ---------------------------------------------------------------- kv append
def test_kv_append_writes_exactly_the_new_slot():
    w = small([1, 16, 17, 0, 40], hq=8, hkv=2, d=64, pool="holes:0.3", seed=31)
    rng = np.random.default_rng(0)
    kn = rng.integers(0, 1 << 15, size=(5, 2, 64)).astype(np.uint16)
    vn = rng.integers(0, 1 << 15, size=(5, 2, 64)).astype(np.uint16)
    k2, v2 = oracle.kv_append(w.k_cache, w.v_cache, kn, vn, w.block_table, w.context_lens)
    changed = np.zeros(w.k_cache.shape[:2], dtype=bool)
    for b, L in enumerate(w.context_lens):
        if L == 0:
            continue
        t = int(L) - 1
        page, slot = w.block_table[b, t // 16], t % 16
        assert np.array_equal(k2[page, slot], kn[b]) and np.array_equal(v2[page, slot], vn[b])
        changed[page, slot] = True
    assert np.array_equal(k2[~changed], w.k_cache[~changed])
    assert np.array_equal(v2[~changed], w.v_cache[~changed])
    assert changed.sum() == 4


def test_append_then_attend_equals_attend_on_the_full_cache():
    # blank the newest token of every sequence, append it back, attend
    w = small([3, 33, 100, 0, 257], hq=8, hkv=2, d=64, seed=32)
    kn = np.zeros((w.batch, 2, 64), dtype=np.uint16)
    vn = np.zeros_like(kn)
    kb, vb = w.k_cache.copy(), w.v_cache.copy()
    for b, L in enumerate(w.context_lens):
        if L == 0:
            continue
        t = int(L) - 1
        page, slot = w.block_table[b, t // 16], t % 16
        kn[b], vn[b] = kb[page, slot], vb[page, slot]
        kb[page, slot] = 0x7FC0
        vb[page, slot] = 0x7FC0
    k2, v2 = oracle.kv_append(kb, vb, kn, vn, w.block_table, w.context_lens)
    a, _ = oracle.attend(w.q, k2, v2, w.block_table, w.context_lens, w.scale)
    ref, _ = run(w)
    assert np.array_equal(a, ref)



# ------------------------------------------- several query tokens, sliding window
def masked(w, window=None):
    q = w.q if w.q.ndim == 4 else w.q[:, None]
    return oracle.attend_masked(q, w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale,
                                w.window if window is None else window)


def test_masked_single_query_without_window_is_attend():
    w = small([1, 33, 300, 0, 17], seed=40)
    ref, lse_ref = run(w)
    out, lse = masked(w, 0)
    assert np.array_equal(out[:, 0], ref) and np.array_equal(lse[:, 0], lse_ref)
    out, _ = masked(w, 300)  # a window as long as the longest sequence cuts nothing
    assert np.array_equal(out[:, 0], ref)


def test_masked_queries_are_causal_prefixes():
    # query j of Tq equals one query over the first L - Tq + 1 + j tokens
    tq = 3
    w = small([2, 40, 77, 129], hq=8, hkv=2, num_queries=tq, seed=41, poison=False)
    out, _ = masked(w, 0)
    for j in range(tq):
        lens = np.maximum(w.context_lens - tq + 1 + j, 0).astype(np.int32)
        ref, _ = oracle.attend(np.ascontiguousarray(w.q[:, j]), w.k_cache, w.v_cache, w.block_table, lens,
                               w.scale)
        np.testing.assert_allclose(out[:, j], ref, rtol=0, atol=1e-15)


@pytest.mark.parametrize("tq,window", [(1, 5), (2, 16), (4, 1), (3, 40), (2, 0)])
def test_masked_matches_torch_sdpa_with_boolean_mask(tq, window):
    w = small([3, 50, 97, 200], hq=8, hkv=2, d=64, num_queries=tq, window=window, seed=42, poison=False)
    out, _ = masked(w)
    dense = flat_gather_dense(w)
    q4 = w.q if w.q.ndim == 4 else w.q[:, None]
    for b in range(w.batch):
        L = int(w.context_lens[b])
        kd, vd = dense[b]
        pos = torch.arange(tq, dtype=torch.int64)[:, None] + (L - tq)   # query positions
        key = torch.arange(L, dtype=torch.int64)[None, :]
        allowed = key <= pos
        if window:
            allowed &= key > pos - window
        qd = torch.from_numpy(oracle.bf16_to_f64(q4[b])).permute(1, 0, 2)        # [Hq, Tq, D]
        kt = torch.from_numpy(kd).permute(1, 0, 2)                               # [Hq, L, D]
        vt = torch.from_numpy(vd).permute(1, 0, 2)
        ref = torch.nn.functional.scaled_dot_product_attention(
            qd, kt, vt, attn_mask=allowed, scale=float(np.float32(w.scale))).permute(1, 0, 2).numpy()
        rows = allowed.any(dim=1).numpy()
        np.testing.assert_allclose(out[b][rows], ref[rows], rtol=0, atol=1e-12)
        assert np.array_equal(out[b][~rows], np.zeros_like(out[b][~rows]))


def test_window_of_one_returns_the_own_value():
    w = small([5, 16, 33], hq=8, hkv=2, num_queries=2, window=1, seed=43, poison=False)
    out, _ = masked(w)
    g = 4
    for b in range(w.batch):
        L = int(w.context_lens[b])
        for j in range(2):
            t = L - 2 + j
            page, slot = w.block_table[b, t // 16], t % 16
            for h in range(8):
                assert np.array_equal(out[b, j, h], oracle.bf16_to_f64(w.v_cache[page, slot, h // g]))


def test_window_released_pages_are_never_read():
    lens = [100, 300, 47, 64]
    clean = small(lens, num_queries=2, window=40, seed=44, poison=False)
    dirty = small(lens, num_queries=2, window=40, seed=44, poison=True)
    assert (dirty.block_table[1, :10] == -1).all()   # tokens < 259 are outside every window
    a, _ = masked(clean)
    b_, _ = masked(dirty)
    assert np.isfinite(b_).all() and np.array_equal(a, b_)


def test_queries_before_the_first_token_are_zero():
    w = small([0, 1, 2, 5], hq=4, hkv=2, num_queries=3, seed=45)
    out, lse = masked(w, 0)
    for b, L in enumerate(w.context_lens):
        for j in range(3):
            if L - 3 + j < 0:
                assert np.array_equal(out[b, j], np.zeros_like(out[b, j])) and np.isneginf(lse[b, j]).all()
            else:
                assert np.isfinite(lse[b, j]).all()


def test_kv_append_of_several_tokens_equals_one_at_a_time():
    w = small([3, 40, 17, 2], hq=8, hkv=2, d=64, seed=33)
    rng = np.random.default_rng(1)
    T = 3
    kn = rng.integers(0, 1 << 15, size=(4, T, 2, 64)).astype(np.uint16)
    vn = rng.integers(0, 1 << 15, size=(4, T, 2, 64)).astype(np.uint16)
    k1, v1 = oracle.kv_append(w.k_cache, w.v_cache, kn, vn, w.block_table, w.context_lens)
    k2, v2 = w.k_cache, w.v_cache
    for j in range(T):
        lens = (w.context_lens - T + 1 + j).astype(np.int32)
        live = lens > 0
        kj, vj = kn[:, j].copy(), vn[:, j].copy()
        k2, v2 = oracle.kv_append(k2, v2, kj, vj, w.block_table, np.where(live, lens, 0))
    assert np.array_equal(k1, k2) and np.array_equal(v1, v2)
    # the sequence of length 2 takes only its last two tokens (positions 0 and 1)
    page = w.block_table[3, 0]
    assert np.array_equal(k1[page, 0], kn[3, 1]) and np.array_equal(k1[page, 1], kn[3, 2])
