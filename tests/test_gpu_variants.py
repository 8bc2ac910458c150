"""GPU parity of the attention variants (several causal query tokens per
sequence, sliding window, 16 query heads per kv head) through the C ABI,
against the fp64 oracle's ``attend_masked``.

Same bar as the plain path: required tolerance, and every output within one
bf16 spacing of the fp64 value.  Workloads are NaN-poisoned; with a window,
pages wholly before the first visible key are released (page-table entry -1,
NaN contents), so reading one would show up as a non-finite output.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from _gpu import bf16_round, bf16_ulps, check, check_full, log, q4, run_ext, to_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib(gpu_lib):
    return gpu_lib


@pytest.fixture(autouse=True)
def default_options(gpu_lib):
    gpu_lib.set_option(gpu_lib.OPT_BLOCKS_PER_CU, 1)
    gpu_lib.set_option(gpu_lib.OPT_MIN_STEPS, 0)
    yield
    gpu_lib.set_option(gpu_lib.OPT_BLOCKS_PER_CU, 1)
    gpu_lib.set_option(gpu_lib.OPT_MIN_STEPS, 0)


def ref(w):
    return oracle.attend_masked(q4(w), w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale,
                                w.window)[0]


# (head_dim, Hq, Hkv, page_size, lengths, query tokens, window)
CASES = [
    (128, 32, 8, 16, [1, 2, 31, 32, 33, 100, 1000], 4, 0),      # G x Tq = 16
    (128, 32, 8, 16, [1, 2, 31, 32, 33, 100, 1000], 1, 64),
    (128, 32, 8, 16, [5, 33, 66, 1027, 3000], 2, 100),
    (64, 8, 2, 16, [3, 300, 5000], 4, 1),                        # window of one: own value
    (128, 16, 1, 32, [0, 2, 5, 700, 4099], 1, 0),                # G = 16
    (128, 16, 1, 32, [7, 700, 4099], 1, 513),
    (128, 8, 8, 16, [1, 17, 40, 900], 16, 0),                    # 16 query tokens, G = 1
    (128, 8, 8, 16, [20, 900], 16, 30),
    (64, 16, 4, 4, [5, 64, 65, 300], 2, 37),                     # pages below 16 tokens
    (64, 12, 4, 1, [2, 40, 333], 3, 9),
    (128, 8, 8, 1024, [1023, 1025, 3000], 1, 1500),
    (128, 12, 4, 16, [0, 1, 2, 3, 4], 4, 0),                     # L < Tq: leading zero rows
    (64, 4, 2, 64, [129, 4000, 64], 8, 2000),
    (256, 12, 4, 16, [1, 2, 31, 32, 33, 100, 1000], 4, 0),     # head_dim 256
    (256, 8, 2, 16, [5, 33, 66, 1027, 3000], 2, 100),
    (256, 4, 4, 4, [5, 64, 65, 300], 3, 37),
]


@pytest.mark.parametrize("d,hq,hkv,p,lens,tq,window", CASES,
                         ids=[f"D{c[0]}-{c[1]}:{c[2]}-P{c[3]}-T{c[5]}-W{c[6]}" for c in CASES])
def test_variant_shapes(lib, d, hq, hkv, p, lens, tq, window):
    w = W.build(lens, hq, hkv, d, p, seed=sum(lens) + 13 * tq + window, pool="holes:0.2", num_queries=tq,
                window=window)
    log(f"case D={d} {hq}:{hkv} P={p} lens={lens} Tq={tq} W={window}")
    got = run_ext(lib, w)
    check(got, ref(w), "variant")


@pytest.mark.parametrize("min_steps,blocks", [(1, 1), (1, 4), (7, 2), (1 << 20, 1)])
def test_variant_split_sweep(lib, min_steps, blocks):
    # single-step pieces put the last few tokens in pieces that the earlier
    # query tokens cannot see, and the window start in pieces the later
    # tokens cannot see: those pieces carry no weight in the merge
    lib.set_option(lib.OPT_MIN_STEPS, min_steps)
    lib.set_option(lib.OPT_BLOCKS_PER_CU, blocks)
    for tq, window in [(4, 0), (2, 45), (4, 33)]:
        w = W.build([33, 66, 97, 1027, 2050], 32, 8, 128, 16, seed=70 + tq + window, num_queries=tq,
                    window=window)
        log(f"sweep min_steps={min_steps} blocks/CU={blocks} Tq={tq} W={window}")
        check(run_ext(lib, w), ref(w), f"Tq={tq} W={window}")


def test_window_of_one_is_the_own_value_bitwise(lib):
    w = W.build([5, 16, 33, 2000], 32, 8, 128, 16, seed=80, num_queries=2, window=1)
    got = run_ext(lib, w)
    r = ref(w)
    assert np.array_equal(got, r)   # one key: weight exactly 1, the bf16 value itself


def test_single_query_ext_is_bitwise_the_plain_call(lib):
    from _gpu import run
    w = W.build([1, 100, 4000, 0, 33], 32, 8, 128, 16, seed=81)
    assert np.array_equal(run_ext(lib, w)[:, 0], run(lib, w))


def test_multi_query_rows_equal_shorter_single_queries(lib):
    # query j of Tq on the GPU against the GPU's own single query over L - Tq + 1 + j
    # tokens: the same keys, so the same value up to the split plan's rounding
    import torch
    from _gpu import run
    tq = 4
    w = W.build([40, 700, 3001], 32, 8, 128, 16, seed=82, num_queries=tq, poison=False)
    got = run_ext(lib, w)
    for j in range(tq):
        wj = W.Workload(q=np.ascontiguousarray(w.q[:, j]), k_cache=w.k_cache, v_cache=w.v_cache,
                        block_table=w.block_table,
                        context_lens=(w.context_lens - tq + 1 + j).astype(np.int32), scale=w.scale)
        single = run(lib, wj)
        # each is within one bf16 spacing of the same fp64 value
        assert np.max(bf16_ulps(got[:, j], single)) <= 2.0
    torch.cuda.synchronize()


def test_variant_graph_capture_replay(lib):
    import torch
    w = W.build([700, 33, 5000], 32, 8, 128, 16, seed=83, num_queries=4, window=256)
    dev = to_gpu(w)
    out = torch.empty(tuple(w.q.shape), dtype=torch.bfloat16, device="cuda")
    s = torch.cuda.Stream()
    lib.workspace_reserve(3, 32, 8, 128, 16, w.max_pages, stream=s)
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=s):
        lib.paged_decode_attention_ext(dev["q"], dev["k"], dev["v"], dev["bt"], dev["lens"], out,
                                       float(w.scale), window=256)
    r = ref(w)
    for rep in range(3):
        g.replay()
        torch.cuda.synchronize()
        check(out.float().cpu().numpy().astype(np.float64), r, f"replay {rep}")


@pytest.mark.parametrize("name", ["window", "multiq", "gqa16", "falcon3"])
def test_variant_workload_every_output(lib, name, tmp_path):
    # the named variant workloads (sliding window, four query tokens, G = 16,
    # head_dim 256), every output against the oracle
    check_full(name, lambda w: run_ext(lib, w), tmp_path)
