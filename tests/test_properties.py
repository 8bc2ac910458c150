"""Property tests over random small shapes (hypothesis, derandomized so every
run draws the same examples): head groups of 1 to 16, page sizes from 1 to
64, lengths at and around page boundaries, empty sequences, several causal
query tokens and sliding windows.

CPU: the fp64 oracle against torch's fp64 scaled_dot_product_attention on
an independently gathered dense copy of the cache.
GPU: the HIP path through the C ABI against the oracle, at the required
tolerance and within one bf16 spacing.
"""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
import workloads as W

SETTINGS = dict(deadline=None, derandomize=True, database=None,
                suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])


@st.composite
def shapes(draw, head_dims):
    d = draw(st.sampled_from(head_dims))
    hkv = draw(st.sampled_from([1, 2, 4, 8]))
    nq = draw(st.sampled_from([1, 1, 1, 2, 3, 4]))
    group = draw(st.integers(1, 16 // nq))
    p = draw(st.sampled_from([1, 2, 4, 8, 16, 32, 64]))
    batch = draw(st.integers(1, 4))
    near = [0, 1, p - 1, p, p + 1, 2 * p + 1, 3 * p - 1]
    lens = draw(st.lists(st.one_of(st.sampled_from([x for x in near if x >= 0]), st.integers(0, 300)),
                         min_size=batch, max_size=batch))
    window = draw(st.sampled_from([0, 0, 1, 5, 40]))
    seed = draw(st.integers(0, 2 ** 16))
    return d, hkv * group, hkv, p, lens, nq, window, seed


def dense_reference(w):
    """torch fp64 SDPA per sequence on a dense copy gathered by flat token
    index (page * P + slot) with a boolean mask of the visible keys (a key t
    is visible to the query at position p when t <= p and, with a window,
    t > p - window)."""
    import torch
    q = w.q if w.q.ndim == 4 else w.q[:, None]
    b_, tq, hq, d = q.shape
    hkv = w.k_cache.shape[2]
    g = hq // hkv
    kf = W.bf16_bits_to_f32(w.k_cache).astype(np.float64).reshape(-1, hkv, d)
    vf = W.bf16_bits_to_f32(w.v_cache).astype(np.float64).reshape(-1, hkv, d)
    qf = W.bf16_bits_to_f32(q).astype(np.float64)
    p = w.k_cache.shape[1]
    out = np.zeros(q.shape, dtype=np.float64)
    for b in range(b_):
        L = int(w.context_lens[b])
        if L == 0:
            continue
        # keys before the first one any query sees may sit on released pages
        t = np.arange(W.window_start(L, tq, w.window), L)
        flat = w.block_table[b, t // p].astype(np.int64) * p + t % p
        kd = torch.from_numpy(np.repeat(kf[flat], g, axis=1).transpose(1, 0, 2).copy())  # [hq, L, d]
        vd = torch.from_numpy(np.repeat(vf[flat], g, axis=1).transpose(1, 0, 2).copy())
        qd = torch.from_numpy(qf[b].transpose(1, 0, 2).copy())                            # [hq, tq, d]
        pos = L - tq + np.arange(tq)
        mask = t[None, :] <= pos[:, None]
        if w.window:
            mask &= t[None, :] > pos[:, None] - w.window
        rows = mask.any(axis=1)
        if not rows.any():
            continue
        o = torch.nn.functional.scaled_dot_product_attention(
            qd[:, rows], kd, vd, attn_mask=torch.from_numpy(mask[rows]), scale=float(np.float32(w.scale)))
        out[b, rows] = o.numpy().transpose(1, 0, 2)
    return out


@settings(max_examples=40, **SETTINGS)
@given(shapes(head_dims=[8, 16, 64]))
def test_oracle_matches_torch_sdpa(shape):
    d, hq, hkv, p, lens, nq, window, seed = shape
    w = W.build(lens, hq, hkv, d, p, seed=seed, pool="holes:0.3", num_queries=nq, window=window)
    q = w.q if w.q.ndim == 4 else w.q[:, None]
    got = oracle.attend_masked(q, w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale, w.window)[0]
    ref = dense_reference(w)
    assert np.isfinite(got).all()
    assert np.abs(got - ref).max() <= 1e-12


@pytest.mark.gpu
@settings(max_examples=60, **SETTINGS)
@given(shapes(head_dims=[64, 128, 256]))
def test_gpu_matches_oracle_on_random_shapes(gpu_lib, shape):
    import torch
    from _gpu import check, log, to_gpu
    d, hq, hkv, p, lens, nq, window, seed = shape
    w = W.build(lens, hq, hkv, d, p, seed=seed, pool="holes:0.3", num_queries=nq, window=window)
    log(f"property case D={d} {hq}:{hkv} P={p} lens={lens} Tq={nq} W={window} seed={seed}")
    dev = to_gpu(w)
    q = dev["q"] if dev["q"].dim() == 4 else dev["q"].unsqueeze(1)
    out = torch.full(tuple(q.shape), float("nan"), dtype=torch.bfloat16, device="cuda")
    gpu_lib.paged_decode_attention_ext(q.contiguous(), dev["k"], dev["v"], dev["bt"], dev["lens"], out,
                                       float(w.scale), window=window)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy().astype(np.float64)
    qh = w.q if w.q.ndim == 4 else w.q[:, None]
    ref = oracle.attend_masked(qh, w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale, w.window)[0]
    check(got, ref, "property")
