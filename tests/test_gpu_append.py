"""GPU parity of the KV append and of append-then-attend, through the C ABI,
against the oracle.

The append moves bf16 bit patterns only, so the whole K and V pools are
compared bit for bit with the oracle's (NaN poison included).  Attention
after the append is held to the same bar as attention alone (required
tolerance, and within one bf16 spacing of the fp64 value).
"""
import numpy as np
import pytest

import oracle
import workloads as W
from _gpu import check, log, to_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib(gpu_lib):
    return gpu_lib


def bits(t):
    import torch
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def bf_dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def new_kv(w, seed):
    rng = np.random.default_rng(seed)
    shape = (w.batch, w.num_kv_heads, w.head_dim)
    return (W.f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32)),
            W.f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32)))


# (head_dim, Hq, Hkv, page_size, lengths, pool): first slot of a page, last
# slot, middle, length 1, empty sequences, every page size class
CASES = [
    (64, 8, 2, 16, [256, 1, 0, 17], "perm:64"),
    (128, 32, 8, 16, [1, 2, 31, 32, 33, 100, 1000], "holes:0.3"),
    (128, 5, 1, 32, [16, 31, 32, 33, 95, 0], "exact"),
    (64, 4, 4, 1, [1, 7, 8], "holes:0.2"),
    (128, 8, 8, 1024, [1023, 1024, 1025, 3000], "holes:0.1"),
    (64, 16, 2, 128, [129, 128, 4000], "perm:200"),
    (256, 12, 4, 16, [1, 15, 16, 17, 0, 900], "holes:0.2"),
    (256, 8, 2, 2, [1, 2, 3, 65], "exact"),
]


@pytest.mark.parametrize("d,hq,hkv,p,lens,pool", CASES,
                         ids=[f"D{c[0]}-{c[1]}:{c[2]}-P{c[3]}" for c in CASES])
def test_kv_append_bitwise(lib, d, hq, hkv, p, lens, pool):
    import torch
    w = W.build(lens, hq, hkv, d, p, seed=sum(lens) + 7 * p, pool=pool)
    log(f"append D={d} {hq}:{hkv} P={p} lens={lens} pool={pool}")
    kn, vn = new_kv(w, 1)
    dev = to_gpu(w)
    lib.kv_append(bf_dev(kn), bf_dev(vn), dev["k"], dev["v"], dev["bt"], dev["lens"])
    torch.cuda.synchronize()
    rk, rv = oracle.kv_append(w.k_cache, w.v_cache, kn, vn, w.block_table, w.context_lens)
    assert np.array_equal(bits(dev["k"]), rk)
    assert np.array_equal(bits(dev["v"]), rv)


def test_kv_append_max_batch(lib):
    import torch
    lens = np.random.default_rng(5).integers(0, 64, size=8192).astype(np.int32)
    w = W.build(lens.tolist(), 8, 2, 64, 16, seed=5, pool="exact")
    kn, vn = new_kv(w, 2)
    dev = to_gpu(w)
    lib.kv_append(bf_dev(kn), bf_dev(vn), dev["k"], dev["v"], dev["bt"], dev["lens"])
    torch.cuda.synchronize()
    rk, rv = oracle.kv_append(w.k_cache, w.v_cache, kn, vn, w.block_table, w.context_lens)
    assert np.array_equal(bits(dev["k"]), rk) and np.array_equal(bits(dev["v"]), rv)


def test_kv_append_bad_device_contents_do_not_fault(lib):
    # page ids out of range and lengths beyond the table are clamped into the pool
    import torch
    w = W.build([40, 40, 40], 8, 2, 64, 16, seed=6, poison=False)
    w.block_table[0, 2] = 10 ** 6
    w.block_table[1, 2] = -5
    w.context_lens[2] = 10 ** 6
    kn, vn = new_kv(w, 3)
    dev = to_gpu(w)
    lib.kv_append(bf_dev(kn), bf_dev(vn), dev["k"], dev["v"], dev["bt"], dev["lens"])
    torch.cuda.synchronize()
    assert bits(dev["k"]).shape == w.k_cache.shape


def test_kv_append_argument_error_writes_nothing(lib):
    import torch
    w = W.build([30, 31], 8, 2, 64, 16, seed=7)
    kn, vn = new_kv(w, 4)
    dev = to_gpu(w)
    rc = lib.load().pda_kv_append(bf_dev(kn).data_ptr(), bf_dev(vn).data_ptr() + 2, dev["k"].data_ptr(),
                                  dev["v"].data_ptr(), dev["bt"].data_ptr(), dev["lens"].data_ptr(), 2, 2, 64, 16,
                                  w.num_pages, w.max_pages, None)
    assert rc == 5
    torch.cuda.synchronize()
    assert np.array_equal(bits(dev["k"]), w.k_cache) and np.array_equal(bits(dev["v"]), w.v_cache)


def _append_then_attend(lib, w, seed, what):
    import torch
    kn, vn = new_kv(w, seed)
    dev = to_gpu(w)
    out = torch.full(tuple(w.q.shape), float("nan"), dtype=torch.bfloat16, device="cuda")
    lib.paged_decode_attention_append(dev["q"], bf_dev(kn), bf_dev(vn), dev["k"], dev["v"], dev["bt"],
                                      dev["lens"], out, float(w.scale))
    torch.cuda.synchronize()
    rk, rv = oracle.kv_append(w.k_cache, w.v_cache, kn, vn, w.block_table, w.context_lens)
    assert np.array_equal(bits(dev["k"]), rk) and np.array_equal(bits(dev["v"]), rv)
    ref = oracle.attend(w.q, rk, rv, w.block_table, w.context_lens, w.scale)[0]
    check(out.float().cpu().numpy().astype(np.float64), ref, what)


@pytest.mark.parametrize("d,hq,hkv,p,lens,pool", CASES,
                         ids=[f"D{c[0]}-{c[1]}:{c[2]}-P{c[3]}" for c in CASES])
def test_append_then_attend(lib, d, hq, hkv, p, lens, pool):
    w = W.build(lens, hq, hkv, d, p, seed=sum(lens) + 11 * p, pool=pool)
    log(f"append+attend D={d} {hq}:{hkv} P={p} lens={lens}")
    _append_then_attend(lib, w, 8, "append+attend")


@pytest.mark.parametrize("name", ["tiny", "llama8b", "batched"])
def test_append_then_attend_named_workload(lib, name):
    log(f"workload {name}: append then attend")
    _append_then_attend(lib, W.make(name), 9, name)


def test_decode_loop_in_a_graph(lib):
    """Four decode steps replayed from one captured graph: each replay
    advances the lengths by one (an elementwise kernel inside the graph),
    appends the step's key/value and attends.  Every step must equal the
    oracle's append-then-attend over the same history."""
    import torch
    steps = 4
    final = [40, 47, 48, 300, 1]
    start = [x - steps for x in final[:-1]] + [0]
    final[-1] = steps
    w = W.build(final, 16, 4, 128, 16, seed=21, pool="perm:100", poison=False)
    w.context_lens[:] = np.asarray(start, dtype=np.int32)
    dev = to_gpu(w)
    q = torch.empty_like(dev["q"])
    kn = torch.empty((w.batch, w.num_kv_heads, w.head_dim), dtype=torch.bfloat16, device="cuda")
    vn = torch.empty_like(kn)
    out = torch.empty_like(q)
    s = torch.cuda.Stream()
    lib.workspace_reserve(w.batch, 16, 4, 128, 16, w.max_pages, stream=s)
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=s):
        dev["lens"].add_(1)
        lib.paged_decode_attention_append(q, kn, vn, dev["k"], dev["v"], dev["bt"], dev["lens"], out,
                                          float(w.scale))
    # capture does not run the work: the lengths are still the starting ones
    assert np.array_equal(dev["lens"].cpu().numpy(), np.asarray(start))
    hk, hv, lens = w.k_cache.copy(), w.v_cache.copy(), np.asarray(start, dtype=np.int32)
    rng = np.random.default_rng(22)
    for step in range(steps):
        qb = W.f32_to_bf16_bits(rng.standard_normal(w.q.shape, dtype=np.float32))
        kb, vb = (W.f32_to_bf16_bits(rng.standard_normal(kn.shape, dtype=np.float32)) for _ in range(2))
        q.copy_(bf_dev(qb))
        kn.copy_(bf_dev(kb))
        vn.copy_(bf_dev(vb))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        lens = lens + 1
        hk, hv = oracle.kv_append(hk, hv, kb, vb, w.block_table, lens)
        ref = oracle.attend(qb, hk, hv, w.block_table, lens, w.scale)[0]
        assert np.array_equal(dev["lens"].cpu().numpy(), lens)
        check(out.float().cpu().numpy().astype(np.float64), ref, f"graph step {step}")
    assert np.array_equal(bits(dev["k"]), hk) and np.array_equal(bits(dev["v"]), hv)


@pytest.mark.parametrize("tokens,p,lens", [(4, 16, [1, 3, 4, 5, 33, 700, 0]), (3, 1, [2, 9, 40]),
                                           (16, 1024, [15, 16, 1025, 3000]), (2, 32, [31, 32, 33, 64])])
def test_kv_append_n_bitwise(lib, tokens, p, lens):
    import torch
    w = W.build(lens, 8, 2, 128, p, seed=sum(lens) + tokens, pool="holes:0.2")
    rng = np.random.default_rng(tokens)
    shape = (w.batch, tokens, 2, 128)
    kn = W.f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))
    vn = W.f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))
    dev = to_gpu(w)
    lib.kv_append_n(bf_dev(kn), bf_dev(vn), dev["k"], dev["v"], dev["bt"], dev["lens"])
    torch.cuda.synchronize()
    rk, rv = oracle.kv_append(w.k_cache, w.v_cache, kn, vn, w.block_table, w.context_lens)
    assert np.array_equal(bits(dev["k"]), rk) and np.array_equal(bits(dev["v"]), rv)


def test_multi_token_step_append_then_attend(lib):
    """A step of four new tokens per sequence (e.g. draft tokens): append
    their k, v, then attend with four causal queries."""
    import torch
    tq = 4
    lens = [4, 37, 300, 2049]
    w = W.build(lens, 32, 8, 128, 16, seed=60, num_queries=tq)
    rng = np.random.default_rng(61)
    shape = (w.batch, tq, 8, 128)
    kn = W.f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))
    vn = W.f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))
    dev = to_gpu(w)
    lib.kv_append_n(bf_dev(kn), bf_dev(vn), dev["k"], dev["v"], dev["bt"], dev["lens"])
    out = torch.empty(tuple(w.q.shape), dtype=torch.bfloat16, device="cuda")
    lib.paged_decode_attention_ext(dev["q"], dev["k"], dev["v"], dev["bt"], dev["lens"], out, float(w.scale))
    torch.cuda.synchronize()
    rk, rv = oracle.kv_append(w.k_cache, w.v_cache, kn, vn, w.block_table, w.context_lens)
    assert np.array_equal(bits(dev["k"]), rk) and np.array_equal(bits(dev["v"]), rv)
    ref = oracle.attend_masked(w.q, rk, rv, w.block_table, w.context_lens, w.scale)[0]
    check(out.float().cpu().numpy().astype(np.float64), ref, "4-token step")
