"""GPU parity of the attention prelude (QKV projection + per-head RMSNorm +
RoPE, and its fused KV append) through the C ABI, against the fp64 oracle.

The outputs are bf16; every one must be within one bf16 spacing of the fp64
value (the GPU keeps fp32 intermediates and rounds once).  The packing and
the fused append move bits and are checked bitwise.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from _gpu import bf16_ulps, check, log, to_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib(gpu_lib):
    return gpu_lib


def dev_bf16(a):
    import torch
    if a is None:
        return None
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def host(t):
    return t.float().cpu().numpy().astype(np.float64)


def bits(t):
    import torch
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def check_ulps(got, ref, what, max_ulps=1.0):
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    u = bf16_ulps(got, ref, floor=2.0 ** -10)
    log(f"  {what}: max {u.max():.2f} bf16 ulp, {100 * float((u < 0.5).mean()):.1f}% within half a spacing "
        f"(n={got.size})")
    assert u.max() <= max_ulps, f"{what}: {u.max():.2f} bf16 ulps"


def packed_reference(w):
    """The packed order written out with numpy reshapes: tile (t, kt), then
    lane l = 16 * (k block) + row, then 8 consecutive k."""
    n, k = w.shape
    t4 = w.reshape(n // 16, 16, k // 32, 4, 8)          # t, r, kt, g, e
    return np.ascontiguousarray(t4.transpose(0, 2, 3, 1, 4)).reshape(n, k)


def run_prelude(lib, w, stream=None):
    import torch
    b, hq, hkv, d = w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim
    wp = lib.pack_weights(dev_bf16(w.w_qkv))
    lens = torch.from_numpy(w.context_lens).cuda()
    q = torch.full((b, hq, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    k = torch.full((b, hkv, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    v = torch.full((b, hkv, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    lib.attention_prelude(dev_bf16(w.x), wp, lens, q, k, v, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                          rope_theta=float(w.theta), rotary_dim=w.rotary_dim, interleaved=w.interleaved,
                          bias=dev_bf16(w.bias), q_norm=dev_bf16(w.q_norm), k_norm=dev_bf16(w.k_norm),
                          eps=float(w.eps), stream=stream)
    torch.cuda.synchronize()
    return q, k, v


def ref_prelude(w):
    return oracle.prelude(w.x, w.w_qkv, w.num_q_heads, w.num_kv_heads, w.head_dim, w.context_lens, w.theta,
                          bias=w.bias, q_norm=w.q_norm, k_norm=w.k_norm, eps=w.eps, rotary_dim=w.rotary_dim,
                          interleaved=w.interleaved)


@pytest.mark.parametrize("n,k", [(16, 256), (48, 512), (6144, 4096)])
def test_pack_is_the_tile_permutation(lib, n, k):
    import torch
    rng = np.random.default_rng(n + k)
    w = rng.integers(0, 1 << 16, size=(n, k)).astype(np.uint16)
    wp = lib.pack_weights(dev_bf16(w))
    torch.cuda.synchronize()
    assert np.array_equal(bits(wp), packed_reference(w))


# (batch, hidden, Hq, Hkv, D, options)
SMALL = [
    (1, 256, 4, 2, 64, dict()),
    (5, 512, 8, 2, 128, dict(qk_norm=True)),
    (16, 256, 2, 1, 256, dict(bias=True)),
    (17, 768, 4, 4, 128, dict(rotary_dim=64, interleaved=True, bias=True)),
    (33, 512, 6, 2, 64, dict(qk_norm=True, rotary_dim=32)),
    (64, 1024, 8, 1, 128, dict(qk_norm=True, bias=True)),
    (3, 256, 4, 2, 128, dict(rotary_dim=0)),
    # above 64 sequences (the thin-GEMM form with 8 or 16 column tiles)
    (100, 512, 4, 2, 128, dict(qk_norm=True)),
    (256, 768, 12, 2, 64, dict(bias=True, rotary_dim=32, interleaved=True)),
    (129, 256, 2, 1, 256, dict()),
]


@pytest.mark.parametrize("b,h,hq,hkv,d,opt", SMALL, ids=[f"B{c[0]}-H{c[1]}-{c[2]}:{c[3]}-D{c[4]}" for c in SMALL])
def test_prelude_small_shapes(lib, b, h, hq, hkv, d, opt):
    lens = np.random.default_rng(b + h).integers(0, 200000, size=b)
    lens[0] = 0                                   # an empty slot: position 0
    w = W.build_prelude(b, h, hq, hkv, d, seed=b * 7 + h, lengths=lens, theta=5.0e5, **opt)
    log(f"prelude B={b} H={h} {hq}:{hkv} D={d} {opt}")
    got = run_prelude(lib, w)
    for name, g, r in zip("qkv", got, ref_prelude(w)):
        check_ulps(host(g), r, name)


@pytest.mark.parametrize("name", list(W.PRELUDE_CONFIGS))
def test_prelude_named_workloads(lib, name):
    log(f"prelude workload {name}")
    w = W.make_prelude(name)
    got = run_prelude(lib, w)
    for nm, g, r in zip("qkv", got, ref_prelude(w)):
        check_ulps(host(g), r, f"{name} {nm}")


def test_prelude_append_writes_exactly_its_outputs_into_the_slots(lib):
    import torch
    pw = W.build_prelude(6, 512, 8, 2, 128, seed=31, lengths=[1, 17, 0, 32, 33, 700], qk_norm=True)
    aw = W.build([1, 17, 0, 32, 33, 700], 8, 2, 128, 16, seed=32, pool="holes:0.3")
    q_sep, k_sep, v_sep = run_prelude(lib, pw)
    dev = to_gpu(aw)
    q = torch.empty_like(q_sep)
    wp = lib.pack_weights(dev_bf16(pw.w_qkv))
    lib.attention_prelude_append(dev_bf16(pw.x), wp, dev["lens"], q, dev["k"], dev["v"], dev["bt"],
                                 num_q_heads=8, num_kv_heads=2, head_dim=128, rope_theta=float(pw.theta),
                                 q_norm=dev_bf16(pw.q_norm), k_norm=dev_bf16(pw.k_norm), eps=float(pw.eps))
    torch.cuda.synchronize()
    assert np.array_equal(bits(q), bits(q_sep))
    rk, rv = oracle.kv_append(aw.k_cache, aw.v_cache, bits(k_sep), bits(v_sep), aw.block_table, aw.context_lens)
    assert np.array_equal(bits(dev["k"]), rk) and np.array_equal(bits(dev["v"]), rv)


@pytest.mark.parametrize("hq,hkv,d,hidden", [(32, 8, 128, 1024), (12, 4, 256, 768)], ids=["32:8-D128", "12:4-D256"])
def test_decode_step_prelude_append_then_attention(lib, hq, hkv, d, hidden):
    """One decode step of a layer: the prelude appends k, v into the cache
    and attention reads them back; checked against the oracle's prelude,
    append and attention on the same bf16 values."""
    import torch
    lens = [40, 1, 300, 4096]
    pw = W.build_prelude(4, hidden, hq, hkv, d, seed=41, lengths=lens, theta=5.0e5)
    aw = W.build(lens, hq, hkv, d, 16, seed=42)
    dev = to_gpu(aw)
    q = torch.empty((4, hq, d), dtype=torch.bfloat16, device="cuda")
    out = torch.empty_like(q)
    wp = lib.pack_weights(dev_bf16(pw.w_qkv))
    lib.attention_prelude_append(dev_bf16(pw.x), wp, dev["lens"], q, dev["k"], dev["v"], dev["bt"],
                                 num_q_heads=hq, num_kv_heads=hkv, head_dim=d, rope_theta=float(pw.theta))
    lib.paged_decode_attention(q, dev["k"], dev["v"], dev["bt"], dev["lens"], out, float(aw.scale))
    torch.cuda.synchronize()
    rq, rk, rv = ref_prelude(pw)
    check_ulps(host(q), rq, "q")
    kb, vb = bits(dev["k"]), bits(dev["v"])
    for b, L in enumerate(lens):
        t = L - 1
        page, slot = aw.block_table[b, t // 16], t % 16
        check_ulps(oracle.bf16_to_f64(kb[page, slot]), rk[b], f"k[{b}]")
        check_ulps(oracle.bf16_to_f64(vb[page, slot]), rv[b], f"v[{b}]")
    # attention over exactly the bf16 values the GPU produced
    ref = oracle.attend(bits(q), kb, vb, aw.block_table, aw.context_lens, aw.scale)[0]
    check(host(out), ref, "attention after the prelude")


def test_prelude_empty_batch_is_a_noop(lib):
    import torch
    x = torch.empty((0, 256), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((4 * 64, 256), dtype=torch.bfloat16, device="cuda")
    e = torch.empty((0, 2, 64), dtype=torch.bfloat16, device="cuda")
    lib.attention_prelude(x, lib.pack_weights(w), torch.empty(0, dtype=torch.int32, device="cuda"),
                          e, e[:, :1], e[:, :1], num_q_heads=2, num_kv_heads=1, head_dim=64, rope_theta=1e4)
    torch.cuda.synchronize()


def test_decode_step_graph_replay(lib):
    """prelude_append + attention captured once and replayed for three decode
    steps, the lengths advanced by an elementwise kernel inside the graph."""
    import torch
    steps, final = 3, [40, 200, 3001]
    start = [x - steps for x in final]
    pw = W.build_prelude(3, 512, 16, 4, 128, seed=51, lengths=start, theta=1e6, qk_norm=True)
    aw = W.build(final, 16, 4, 128, 16, seed=52, poison=False)
    aw.context_lens[:] = start
    dev = to_gpu(aw)
    x = torch.empty((3, 512), dtype=torch.bfloat16, device="cuda")
    wp = lib.pack_weights(dev_bf16(pw.w_qkv))
    qn, kn = dev_bf16(pw.q_norm), dev_bf16(pw.k_norm)
    q = torch.empty((3, 16, 128), dtype=torch.bfloat16, device="cuda")
    out = torch.empty_like(q)
    s = torch.cuda.Stream()
    lib.workspace_reserve(3, 16, 4, 128, 16, aw.max_pages, stream=s)
    lib.prelude_workspace_reserve(lib.prelude_dims(3, 512, 16, 4, 128, 128, 0, 1e6, 1e-6), stream=s)
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=s):
        dev["lens"].add_(1)
        lib.attention_prelude_append(x, wp, dev["lens"], q, dev["k"], dev["v"], dev["bt"], num_q_heads=16,
                                     num_kv_heads=4, head_dim=128, rope_theta=1e6, q_norm=qn, k_norm=kn)
        lib.paged_decode_attention(q, dev["k"], dev["v"], dev["bt"], dev["lens"], out, float(aw.scale))
    rng = np.random.default_rng(53)
    kc, vc = aw.k_cache.copy(), aw.v_cache.copy()
    lens = np.asarray(start, dtype=np.int32)
    for step in range(steps):
        xb = W.f32_to_bf16_bits(rng.standard_normal((3, 512)).astype(np.float32))
        x.copy_(dev_bf16(xb))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        lens = lens + 1
        rq, rk, rv = oracle.prelude(xb, pw.w_qkv, 16, 4, 128, lens, np.float32(1e6), q_norm=pw.q_norm,
                                    k_norm=pw.k_norm, eps=np.float32(1e-6))
        check_ulps(host(q), rq, f"step {step} q")
        kb, vb = bits(dev["k"]), bits(dev["v"])
        for b in range(3):
            t = int(lens[b]) - 1
            page, slot = aw.block_table[b, t // 16], t % 16
            check_ulps(oracle.bf16_to_f64(kb[page, slot]), rk[b], f"step {step} k[{b}]")
        ref = oracle.attend(bits(q), kb, vb, aw.block_table, lens, aw.scale)[0]
        check(host(out), ref, f"step {step} attention")
