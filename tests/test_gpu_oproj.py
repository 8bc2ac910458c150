"""GPU parity of the output projection with residual add and RMSNorm
(o_proj GEMV + residual + post-RMSNorm) through the C ABI, against the fp64
oracle: every bf16 output within one bf16 spacing of the fp64 value."""
import numpy as np
import pytest

import oracle
import workloads as W
from _gpu import bf16_ulps, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib(gpu_lib):
    return gpu_lib


def dev_bf16(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def host(t):
    return t.float().cpu().numpy().astype(np.float64)


def check_ulps(got, ref, what, max_ulps=1.0):
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    u = bf16_ulps(got, ref, floor=2.0 ** -10)
    log(f"  {what}: max {u.max():.2f} bf16 ulp (n={got.size})")
    assert u.max() <= max_ulps, f"{what}: {u.max():.2f} bf16 ulps"


def run(lib, w, in_place=False, stream=None):
    import torch
    attn, res, nw = dev_bf16(w.attn), dev_bf16(w.residual), dev_bf16(w.norm_w)
    wp = lib.pack_weights(dev_bf16(w.w_o))
    z = res if in_place else torch.full_like(res, float("nan"))
    h = torch.full_like(res, float("nan"))
    lib.o_proj_residual_norm(attn, wp, res, nw, z, h, eps=float(w.eps), stream=stream)
    torch.cuda.synchronize()
    return host(z), host(h)


def ref(w):
    return oracle.o_proj_residual_norm(w.attn, w.w_o, w.residual, w.norm_w, w.eps)


SMALL = [(1, 32, 16), (3, 96, 48), (17, 4096, 2560), (64, 512, 1024), (5, 64, 32768), (33, 8192, 256),
         # one batch tile of more than 4 sequences: four row tiles share each x
         # fragment when the row tiles divide by four (1040 rows do not)
         (8, 96, 48), (12, 2048, 1040), (16, 3072, 3072), (9, 1024, 4096),
         # more than 16 sequences: the thin-GEMM form when the row tiles divide
         # by 8, otherwise the per-wave form with 2, 3 or 4 row tiles per unit
         # (1056 rows: 66 tiles; 1088: 68) or one (1040: 65)
         (32, 256, 1056), (48, 512, 1056), (64, 512, 1088), (40, 1024, 1040), (64, 4096, 4096),
         # above 64 sequences: the thin-GEMM form with 8 or 16 column tiles;
         # above 128 its tile-major partials go to the two-sequence epilogue,
         # whose last workgroup has one sequence at an odd batch
         (65, 1024, 1024), (128, 512, 2048), (200, 256, 384), (256, 2048, 1280),
         (129, 512, 1024), (255, 1024, 640)]


@pytest.mark.parametrize("b,k,h", SMALL, ids=[f"B{c[0]}-K{c[1]}-H{c[2]}" for c in SMALL])
def test_oproj_small_shapes(lib, b, k, h):
    w = W.build_oproj(b, k, h, seed=b + k + h)
    log(f"o_proj B={b} K={k} H={h}")
    z, hn = run(lib, w)
    rz, rh = ref(w)
    check_ulps(z, rz, "z")
    check_ulps(hn, rh, "h")


@pytest.mark.parametrize("name", list(W.OPROJ_CONFIGS))
def test_oproj_named_workloads(lib, name):
    log(f"o_proj workload {name}")
    w = W.make_oproj(name)
    z, hn = run(lib, w)
    rz, rh = ref(w)
    check_ulps(z, rz, f"{name} z")
    check_ulps(hn, rh, f"{name} h")


def test_oproj_in_place_residual_is_bitwise_the_same(lib):
    w = W.build_oproj(7, 1024, 2048, seed=9)
    a = run(lib, w)
    b = run(lib, w, in_place=True)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_oproj_graph_replay(lib):
    import torch
    w = W.build_oproj(4, 2048, 4096, seed=10)
    attn, res, nw = dev_bf16(w.attn), dev_bf16(w.residual), dev_bf16(w.norm_w)
    wp = lib.pack_weights(dev_bf16(w.w_o))
    z = torch.empty_like(res)
    h = torch.empty_like(res)
    s = torch.cuda.Stream()
    lib.o_proj_workspace_reserve(4, 2048, 4096, stream=s)
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=s):
        lib.o_proj_residual_norm(attn, wp, res, nw, z, h, eps=float(w.eps))
    rz, rh = ref(w)
    for rep in range(3):
        z.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        check_ulps(host(z), rz, f"replay {rep} z")
        check_ulps(host(h), rh, f"replay {rep} h")


def test_oproj_rows_not_8_byte_aligned(lib):
    # the one-kernel epilogue (batch <= 16) moves four bf16 features at a
    # time; rows offset by one element take the two passes, same results
    import torch
    w = W.build_oproj(5, 1024, 2048, seed=11)
    attn, nw = dev_bf16(w.attn), dev_bf16(w.norm_w)
    wp = lib.pack_weights(dev_bf16(w.w_o))
    buf = torch.empty(3 * 5 * 2048 + 8, dtype=torch.bfloat16, device="cuda")
    res = buf[1:1 + 5 * 2048].view(5, 2048)
    res.copy_(dev_bf16(w.residual))
    z = buf[2 + 5 * 2048:2 + 10 * 2048].view(5, 2048)
    h = buf[3 + 10 * 2048:3 + 15 * 2048].view(5, 2048)
    lib.o_proj_residual_norm(attn, wp, res, nw, z, h, eps=float(w.eps))
    torch.cuda.synchronize()
    rz, rh = ref(w)
    check_ulps(host(z), rz, "z, unaligned rows")
    check_ulps(host(h), rh, "h, unaligned rows")
    aligned = run(lib, w)
    assert np.array_equal(host(z), aligned[0]) and np.array_equal(host(h), aligned[1])
