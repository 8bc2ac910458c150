"""Pins of the prelude oracle (QKV projection + RoPE + optional per-head
Q/K RMSNorm) against facts that do not come from it: exact integer
arithmetic, the complex-number form of the rotation, the relative-position
property that defines RoPE, torch's own RMSNorm, and an independent torch
formulation of the whole prelude."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W


def small(batch=3, hidden=64, hq=4, hkv=2, d=16, seed=5, **kw):
    lens = np.random.default_rng(seed).integers(1, 5000, size=batch)
    return W.build_prelude(batch, hidden, hq, hkv, d, seed, lengths=lens, **kw)


def run(w, **over):
    kw = dict(bias=w.bias, q_norm=w.q_norm, k_norm=w.k_norm, eps=w.eps, rotary_dim=w.rotary_dim,
              interleaved=w.interleaved)
    kw.update(over)
    return oracle.prelude(w.x, w.w_qkv, w.num_q_heads, w.num_kv_heads, w.head_dim, w.context_lens, w.theta,
                          **kw)


def test_integer_projection_is_exact_and_blocks_are_ordered_q_k_v():
    # small integers are exact in bf16 and in fp64 sums; position 0 turns nothing
    rng = np.random.default_rng(0)
    b, h, hq, hkv, d = 3, 40, 4, 2, 8
    n = (hq + 2 * hkv) * d
    xi = rng.integers(-8, 9, size=(b, h))
    wi = rng.integers(-8, 9, size=(n, h))
    x = W.f32_to_bf16_bits(xi.astype(np.float32))
    w = W.f32_to_bf16_bits(wi.astype(np.float32))
    q, k, v = oracle.prelude(x, w, hq, hkv, d, np.ones(b, dtype=np.int32), 1.0e4)
    y = xi @ wi.T                                       # exact int64
    assert np.array_equal(q.reshape(b, -1), y[:, :hq * d])
    assert np.array_equal(k.reshape(b, -1), y[:, hq * d:(hq + hkv) * d])
    assert np.array_equal(v.reshape(b, -1), y[:, (hq + hkv) * d:])


def test_bias_adds_to_every_row():
    w = small(bias=True)
    q, k, v = run(w)
    q0, k0, v0 = run(w, bias=None)
    bias = oracle.bf16_to_f64(w.bias)
    # v is untouched by rotation, so the difference is the bias itself
    np.testing.assert_allclose((v - v0).reshape(w.batch, -1),
                               np.broadcast_to(bias[(w.num_q_heads + w.num_kv_heads) * w.head_dim:],
                                               (w.batch, w.num_kv_heads * w.head_dim)), rtol=0, atol=1e-12)


@pytest.mark.parametrize("interleaved", [False, True])
@pytest.mark.parametrize("rd", [16, 8])
def test_rope_is_complex_multiplication(interleaved, rd):
    rng = np.random.default_rng(1)
    t = rng.standard_normal((3, 2, 16))
    pos = np.array([0, 7, 131071])
    got = oracle.rope(t, pos, 5.0e5, rd, interleaved)
    half = rd // 2
    idx_a = np.arange(0, rd, 2) if interleaved else np.arange(half)
    idx_b = idx_a + 1 if interleaved else idx_a + half
    z = t[..., idx_a] + 1j * t[..., idx_b]
    freq = np.float64(np.float32(5.0e5)) ** (-np.arange(0, rd, 2, dtype=np.float64) / rd)
    zr = z * np.exp(1j * np.outer(pos, freq))[:, None, :]
    np.testing.assert_allclose(got[..., idx_a], zr.real, rtol=0, atol=1e-12)
    np.testing.assert_allclose(got[..., idx_b], zr.imag, rtol=0, atol=1e-12)
    rest = np.setdiff1d(np.arange(16), np.concatenate([idx_a, idx_b]))
    assert np.array_equal(got[..., rest], t[..., rest])   # partial rotary passes the rest through


def test_rope_scores_depend_only_on_relative_position():
    rng = np.random.default_rng(2)
    q = rng.standard_normal((1, 1, 64))
    k = rng.standard_normal((1, 1, 64))
    def score(p, r):
        return float(np.sum(oracle.rope(q, [p], 1.0e4, 64) * oracle.rope(k, [r], 1.0e4, 64)))
    for p, r, s in [(5, 2, 100), (1000, 999, 30000), (0, 0, 77)]:
        assert abs(score(p, r) - score(p + s, r + s)) < 1e-9


def test_rope_at_position_zero_is_identity_and_keeps_pair_norms():
    rng = np.random.default_rng(3)
    t = rng.standard_normal((2, 3, 32))
    assert np.array_equal(oracle.rope(t, [0, 0], 1.0e6, 32), t)
    r = oracle.rope(t, [12345, 9], 1.0e6, 32)
    np.testing.assert_allclose(r[..., :16] ** 2 + r[..., 16:] ** 2, t[..., :16] ** 2 + t[..., 16:] ** 2,
                               rtol=1e-12)


def test_rms_norm_matches_torch():
    rng = np.random.default_rng(4)
    t = rng.standard_normal((3, 5, 128)) * 3.0
    wbits = W.f32_to_bf16_bits((1.0 + 0.1 * rng.standard_normal(128)).astype(np.float32))
    eps = np.float32(1e-6)
    got = oracle.rms_norm(t, wbits, eps)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(t), (128,),
                                       weight=torch.from_numpy(oracle.bf16_to_f64(wbits)),
                                       eps=float(eps)).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=0)


def _torch_prelude(w):
    """Independent fp64 formulation: linear, rms_norm, rotate-half / interleaved
    rotation built from a cos/sin table of torch.outer(pos, inv_freq)."""
    f = lambda a: torch.from_numpy(oracle.bf16_to_f64(a))
    x, wt = f(w.x), f(w.w_qkv)
    y = torch.nn.functional.linear(x, wt, None if w.bias is None else f(w.bias))
    hq, hkv, d, b = w.num_q_heads, w.num_kv_heads, w.head_dim, w.batch
    q, k, v = y.split([hq * d, hkv * d, hkv * d], dim=1)
    q, k, v = q.reshape(b, hq, d), k.reshape(b, hkv, d), v.reshape(b, hkv, d)
    if w.q_norm is not None:
        q = torch.nn.functional.rms_norm(q, (d,), weight=f(w.q_norm), eps=float(w.eps))
        k = torch.nn.functional.rms_norm(k, (d,), weight=f(w.k_norm), eps=float(w.eps))
    rd = w.rotary_dim
    pos = torch.clamp(torch.from_numpy(w.context_lens.astype(np.int64)) - 1, min=0).double()
    inv = float(w.theta) ** (-torch.arange(0, rd, 2, dtype=torch.float64) / rd)
    ang = torch.outer(pos, inv)[:, None, :]
    cos, sin = torch.cos(ang), torch.sin(ang)

    def rot(t):
        r, rest = t[..., :rd], t[..., rd:]
        if w.interleaved:
            a, c = r[..., 0::2], r[..., 1::2]
            out = torch.stack((a * cos - c * sin, c * cos + a * sin), dim=-1).flatten(-2)
        else:
            a, c = r[..., :rd // 2], r[..., rd // 2:]
            out = torch.cat((a * cos - c * sin, c * cos + a * sin), dim=-1)
        return torch.cat((out, rest), dim=-1)
    return rot(q).numpy(), rot(k).numpy(), v.numpy()


@pytest.mark.parametrize("kw", [dict(), dict(qk_norm=True), dict(bias=True, rotary_dim=8, interleaved=True),
                                dict(qk_norm=True, rotary_dim=8)],
                         ids=["plain", "qk_norm", "bias-partial-interleaved", "norm-partial"])
def test_prelude_matches_independent_torch_formulation(kw):
    w = small(**kw)
    got = run(w)
    ref = _torch_prelude(w)
    for g, r in zip(got, ref):
        np.testing.assert_allclose(g, r, rtol=0, atol=1e-12)


def test_position_is_length_minus_one_and_empty_slots_use_zero():
    # lengths 1 and 0 both put the token at position 0, where nothing turns
    w = small(batch=2)
    w.context_lens[:] = [1, 0]
    q, k, _ = run(w)
    y = oracle.bf16_to_f64(w.x) @ oracle.bf16_to_f64(w.w_qkv).T
    hq, hkv, d = w.num_q_heads, w.num_kv_heads, w.head_dim
    assert np.array_equal(q.reshape(2, -1), y[:, :hq * d])
    assert np.array_equal(k.reshape(2, -1), y[:, hq * d:(hq + hkv) * d])
    w.context_lens[:] = [2, 2]                        # position 1: q turns
    q1, _, _ = run(w)
    assert not np.allclose(q1, q)
