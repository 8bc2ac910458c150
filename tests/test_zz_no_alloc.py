"""The attention entry point that allocates nothing
(paged_decode_attention_noalloc), through the C ABI, against the regular
entry point on the same inputs: the two share their kernels and plan, so the
outputs are bitwise equal, and both are within the attention tolerance of the
fp64 oracle.  Two calls in a row, the second smaller, exercise the shared
per-device scratch holding the first call's contents."""
import numpy as np
import pytest

import oracle
import workloads as W
from _gpu import check, log, to_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib(gpu_lib):
    gpu_lib.set_option(gpu_lib.OPT_BLOCKS_PER_CU, 1)
    gpu_lib.set_option(gpu_lib.OPT_MIN_STEPS, 0)
    return gpu_lib


def _both(lib, w, dev=None):
    import torch
    if dev is None:
        dev = to_gpu(w)
    a = torch.full(tuple(w.q.shape), float("nan"), dtype=torch.bfloat16, device="cuda")
    b = torch.full_like(a, float("nan"))
    lib.paged_decode_attention_noalloc(dev["q"], dev["k"], dev["v"], dev["bt"], dev["lens"], a, float(w.scale))
    lib.paged_decode_attention(dev["q"], dev["k"], dev["v"], dev["bt"], dev["lens"], b, float(w.scale))
    torch.cuda.synchronize()
    return (a.float().cpu().numpy().astype(np.float64), b.float().cpu().numpy().astype(np.float64))


def _ref(w):
    return oracle.attend(w.q, w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale)[0]


def test_two_calls_second_smaller(lib):
    # a ragged, NaN-poisoned batch that spans many workgroups (split pieces
    # and the merge), then a smaller one over the scratch the first one left
    big = W.build([5000, 17, 0, 3001, 1, 700, 8191, 33], 40, 8, 128, 32, seed=201, pool="holes:0.2")
    small = W.build([300, 2, 47], 8, 2, 64, 16, seed=202, pool="holes:0.3")
    for name, w in (("first call", big), ("second call, smaller", small)):
        log(f"no-alloc {name}: batch {w.batch} {w.num_q_heads}:{w.num_kv_heads} D={w.head_dim}")
        got, regular = _both(lib, w)
        assert np.array_equal(got, regular), f"{name}: differs from paged_decode_attention"
        check(got, _ref(w), f"no-alloc {name}")


def test_named_workload_matches_regular_entry(lib):
    w = W.make("batched")
    log("no-alloc batched workload")
    got, regular = _both(lib, w)
    assert np.array_equal(got, regular)
    check(got, _ref(w), "no-alloc batched")


def test_shape_beyond_scratch_is_rejected(lib):
    import torch
    # batch 8192 x 8 kv heads at head_dim 128 plans ~140 MB of partial slots
    b, hq, hkv, d = 8192, 32, 8, 128
    _, _, need = lib.plan(b, hq, hkv, d, 16, 4)
    assert need > lib.NOALLOC_SCRATCH_BYTES
    q = torch.zeros((b, hq, d), dtype=torch.bfloat16, device="cuda")
    kc = torch.zeros((4, 16, hkv, d), dtype=torch.bfloat16, device="cuda")
    bt = torch.zeros((b, 4), dtype=torch.int32, device="cuda")
    lens = torch.ones((b,), dtype=torch.int32, device="cuda")
    out = torch.full_like(q, 3.0)
    with pytest.raises(lib.PdaError) as ei:
        lib.paged_decode_attention_noalloc(q, kc, kc, bt, lens, out, 0.125)
    assert ei.value.code == 3 and "no-allocation" in str(ei.value)
    torch.cuda.synchronize()
    assert bool((out == 3.0).all())


def test_graph_capture_without_reserve(lib):
    # captured on a fresh stream with no workspace reserved for it: nothing
    # to allocate, so capture works; every replay equals the eager call
    import torch
    w = W.build([700, 33, 5000, 1], 32, 8, 128, 16, seed=203, pool="holes:0.2")
    dev = to_gpu(w)
    out = torch.empty(tuple(w.q.shape), dtype=torch.bfloat16, device="cuda")
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        lib.paged_decode_attention_noalloc(dev["q"], dev["k"], dev["v"], dev["bt"], dev["lens"], out,
                                           float(w.scale))
    rng = np.random.default_rng(1)
    for rep in range(3):
        w.q[:] = W.f32_to_bf16_bits(rng.standard_normal(w.q.shape, dtype=np.float32))
        dev["q"].copy_(to_gpu(w)["q"])
        g.replay()
        torch.cuda.synchronize()
        replayed = out.float().cpu().numpy().astype(np.float64)
        eager, regular = _both(lib, w, dev)
        assert np.array_equal(replayed, eager) and np.array_equal(eager, regular), f"replay {rep}"
        check(replayed, _ref(w), f"no-alloc replay {rep}")
