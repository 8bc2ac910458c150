"""Property tests of the decode GEMV rows on the GPU over random shapes
(hypothesis, derandomized so every run draws the same examples): the o_proj
with residual and RMSNorm, and the attention prelude with and without Q/K
norm, bias and partial or interleaved rotation.  The drawn batch, input and
output sizes reach plans of every form (per-wave with 1 to 4 row tiles per
unit, thin-GEMM) and, in the prelude, every partial-slot bound its epilogue
is instantiated for (4, 8, 12, 16; the o_proj draws reach 4 to 12, and its
16 is reached by a fixed shape in its own tests).  Each output is held to
one bf16 spacing of the fp64 oracle, as in the fixed-shape tests."""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import workloads as W
from test_gpu_oproj import check_ulps as check_oproj
from test_gpu_oproj import ref as ref_oproj
from test_gpu_oproj import run as run_oproj
from test_gpu_prelude import check_ulps as check_prelude
from test_gpu_prelude import host, ref_prelude, run_prelude
from _gpu import log

pytestmark = pytest.mark.gpu

SETTINGS = dict(deadline=None, derandomize=True, database=None,
                suppress_health_check=[HealthCheck.too_slow, HealthCheck.function_scoped_fixture])


@settings(max_examples=30, **SETTINGS)
@given(batch=st.integers(1, 64), k_tiles=st.integers(1, 128), h_tiles=st.integers(1, 256),
       seed=st.integers(0, 2 ** 16))
def test_oproj_random_shapes(gpu_lib, batch, k_tiles, h_tiles, seed):
    k, h = 32 * k_tiles, 16 * h_tiles
    log(f"o_proj property case B={batch} K={k} H={h} seed={seed}")
    w = W.build_oproj(batch, k, h, seed=seed)
    z, hn = run_oproj(gpu_lib, w)
    rz, rh = ref_oproj(w)
    check_oproj(z, rz, "z")
    check_oproj(hn, rh, "h")


@st.composite
def prelude_shapes(draw):
    d = draw(st.sampled_from([64, 128, 256]))
    hkv = draw(st.sampled_from([1, 2, 4, 8]))
    hq = hkv * draw(st.sampled_from([1, 2, 4, 8]))
    batch = draw(st.integers(1, 64))
    hidden = 32 * draw(st.integers(2, 96))
    rot = draw(st.sampled_from(["full", "half", "none"]))
    opt = dict(qk_norm=draw(st.booleans()), bias=draw(st.booleans()), interleaved=draw(st.booleans()),
               rotary_dim={"full": None, "half": d // 2, "none": 0}[rot])
    return batch, hidden, hq, hkv, d, opt, draw(st.integers(0, 2 ** 16))


@settings(max_examples=30, **SETTINGS)
@given(prelude_shapes())
def test_prelude_random_shapes(gpu_lib, shape):
    batch, hidden, hq, hkv, d, opt, seed = shape
    log(f"prelude property case B={batch} H={hidden} {hq}:{hkv} D={d} {opt} seed={seed}")
    lens = np.random.default_rng(seed).integers(0, 100000, size=batch)
    w = W.build_prelude(batch, hidden, hq, hkv, d, seed=seed, lengths=lens, theta=1.0e6, **opt)
    got = run_prelude(gpu_lib, w)
    for name, g, r in zip("qkv", got, ref_prelude(w)):
        check_prelude(host(g), r, name)
