"""Pins of the o_proj + residual + RMSNorm oracle: exact integer arithmetic,
the defining properties of RMSNorm, torch's linear and rms_norm."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W


def test_integer_projection_plus_residual_is_exact():
    rng = np.random.default_rng(0)
    b, k, h = 3, 64, 48
    ai, wi, ri = rng.integers(-8, 9, (b, k)), rng.integers(-8, 9, (h, k)), rng.integers(-50, 51, (b, h))
    bits = lambda a: W.f32_to_bf16_bits(a.astype(np.float32))
    z, _ = oracle.o_proj_residual_norm(bits(ai), bits(wi), bits(ri), bits(np.ones(h)), 1e-6)
    assert np.array_equal(z, ai @ wi.T + ri)


def test_norm_output_has_unit_rms_and_ignores_scale():
    w = W.build_oproj(4, 64, 96, seed=1, eps=0.0)
    ones = W.f32_to_bf16_bits(np.ones(96, dtype=np.float32))
    z, h = oracle.o_proj_residual_norm(w.attn, w.w_o, w.residual, ones, 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(h * h, axis=1)), 1.0, rtol=1e-13)
    # doubling every input doubles z and leaves h unchanged (eps = 0)
    dbl = lambda a: W.f32_to_bf16_bits(W.bf16_bits_to_f32(a) * np.float32(2.0))
    z2, h2 = oracle.o_proj_residual_norm(dbl(w.attn), w.w_o, dbl(w.residual), ones, 0.0)
    np.testing.assert_allclose(z2, 2 * z, rtol=1e-13)
    np.testing.assert_allclose(h2, h, rtol=1e-12)


@pytest.mark.parametrize("eps", [1e-6, 1e-5, 0.5])
def test_matches_torch_linear_and_rms_norm(eps):
    w = W.build_oproj(5, 128, 64, seed=2, eps=eps)
    z, h = oracle.o_proj_residual_norm(w.attn, w.w_o, w.residual, w.norm_w, w.eps)
    f = lambda a: torch.from_numpy(oracle.bf16_to_f64(a))
    zt = torch.nn.functional.linear(f(w.attn), f(w.w_o)) + f(w.residual)
    ht = torch.nn.functional.rms_norm(zt, (64,), weight=f(w.norm_w), eps=float(np.float32(eps)))
    np.testing.assert_allclose(z, zt.numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(h, ht.numpy(), rtol=0, atol=1e-12)
