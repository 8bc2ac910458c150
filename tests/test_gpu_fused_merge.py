"""The merge fused into the attention kernel (the last workgroup to finish a
split sequence merges its pieces in slot order) against the fp64 oracle and
against the separate merge kernel.

PDA_OPT_FUSED_MERGE: 0 (default) never fuses, 1 fuses plans with little
partial data per sequence (single requests, small batches), 2 fuses every
plan with several workgroups -- used here to run the fused merge over many
pieces, several passes of a workgroup over the query rows, windows and
several query tokens, head sizes 64/128/256 and both page-size paths.  A
latency-bound call keeps its fixed split under either mode (the pieces of a
sequence are the chunks its length fills); larger calls take the stream-K
split."""
import numpy as np
import pytest

import oracle
import workloads as W
from _gpu import check, log, q4, run, run_ext, to_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib(gpu_lib):
    return gpu_lib


@pytest.fixture(autouse=True)
def default_options(gpu_lib):
    yield
    gpu_lib.set_option(gpu_lib.OPT_FUSED_MERGE, 0)
    gpu_lib.set_option(gpu_lib.OPT_BLOCKS_PER_CU, 1)
    gpu_lib.set_option(gpu_lib.OPT_MIN_STEPS, 0)


def ref(w):
    return oracle.attend(w.q, w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale)[0]


# (head_dim, Hq, Hkv, page_size, lengths)
SHAPES = [
    (128, 32, 8, 16, [4096]),                       # llama8b-shaped single request
    (128, 32, 8, 16, [1, 2, 31, 32, 33, 100, 1000]),
    (128, 64, 8, 16, [3000, 17, 5000]),             # 8 kv heads x 8 columns: several passes over the rows
    (128, 40, 8, 32, [0, 5, 0, 700, 2048]),
    (64, 8, 2, 16, [256, 3000]),
    (64, 16, 4, 4, [5, 64, 65, 1500]),              # pages of fewer than 16 tokens
    (128, 12, 4, 1, [1, 2, 40, 900]),
    (128, 16, 1, 32, [4099, 7]),                    # G = 16
    (256, 12, 4, 16, [1, 33, 1000, 3000]),          # head_dim 256
    (256, 8, 4, 4, [63, 64, 65, 2000]),
]
IDS = [f"D{c[0]}-{c[1]}:{c[2]}-P{c[3]}-{len(c[4])}seq" for c in SHAPES]


@pytest.mark.parametrize("mode", [1, 2])
@pytest.mark.parametrize("min_steps", [1, 2])
@pytest.mark.parametrize("d,hq,hkv,p,lens", SHAPES, ids=IDS)
def test_fused_merge_matches_oracle(lib, d, hq, hkv, p, lens, min_steps, mode):
    w = W.build(lens, hq, hkv, d, p, seed=300 + sum(lens) + d + p, pool="holes:0.2")
    lib.set_option(lib.OPT_FUSED_MERGE, mode)
    lib.set_option(lib.OPT_MIN_STEPS, min_steps)
    log(f"case fused mode {mode} min_steps {min_steps} D={d} {hq}:{hkv} P={p} lens={lens}")
    dev = to_gpu(w)
    got = run(lib, w, dev)
    check(got, ref(w), "fused merge")
    assert np.array_equal(got, run(lib, w, dev)), "fused merge not reproducible"
    lib.set_option(lib.OPT_FUSED_MERGE, 0)
    sep = run(lib, w, dev)
    check(sep, ref(w), "separate merge")


@pytest.mark.parametrize("min_steps,blocks", [(1, 1), (1, 4), (7, 2)])
def test_fused_merge_with_windows_and_query_tokens(lib, min_steps, blocks):
    # pieces that no query of a column reaches carry m = -inf into the merge
    lib.set_option(lib.OPT_FUSED_MERGE, 2)
    lib.set_option(lib.OPT_MIN_STEPS, min_steps)
    lib.set_option(lib.OPT_BLOCKS_PER_CU, blocks)
    for tq, window in [(4, 0), (2, 45), (4, 33), (1, 100)]:
        w = W.build([33, 66, 97, 1027, 2050], 32, 8, 128, 16, seed=310 + tq + window, num_queries=tq,
                    window=window)
        log(f"fused: Tq={tq} W={window} min_steps={min_steps} blocks={blocks}")
        r = oracle.attend_masked(q4(w), w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale, w.window)[0]
        check(run_ext(lib, w), r, f"Tq={tq} W={window}")


def test_fused_merge_graph_replays(lib):
    # the arrival counters reset themselves: every replay merges correctly
    import torch
    lib.set_option(lib.OPT_FUSED_MERGE, 2)
    lib.set_option(lib.OPT_MIN_STEPS, 1)
    w = W.build([700, 33, 5000, 1], 32, 8, 128, 16, seed=320, pool="holes:0.2")
    dev = to_gpu(w)
    out = torch.empty(tuple(w.q.shape), dtype=torch.bfloat16, device="cuda")
    s = torch.cuda.Stream()
    lib.workspace_reserve(4, 32, 8, 128, 16, w.max_pages, stream=s)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        lib.paged_decode_attention(dev["q"], dev["k"], dev["v"], dev["bt"], dev["lens"], out, float(w.scale))
    rng = np.random.default_rng(2)
    for rep in range(4):
        w.q[:] = W.f32_to_bf16_bits(rng.standard_normal(w.q.shape, dtype=np.float32))
        dev["q"].copy_(to_gpu(w)["q"])
        g.replay()
        torch.cuda.synchronize()
        replayed = out.float().cpu().numpy().astype(np.float64)
        eager = run(lib, w, dev)
        assert np.array_equal(replayed, eager), f"replay {rep} differs from the eager call"
        check(replayed, ref(w), f"fused replay {rep}")


def test_fused_merge_through_noalloc_scratch(lib):
    # the counters at the end of the fixed scratch; two calls in a row
    lib.set_option(lib.OPT_FUSED_MERGE, 2)
    import torch
    for lens, seed in (([5000, 17, 3001, 1], 330), ([300, 2, 47], 331)):
        w = W.build(lens, 32, 8, 128, 16, seed=seed, pool="holes:0.2")
        dev = to_gpu(w)
        a = torch.full(tuple(w.q.shape), float("nan"), dtype=torch.bfloat16, device="cuda")
        lib.paged_decode_attention_noalloc(dev["q"], dev["k"], dev["v"], dev["bt"], dev["lens"], a, float(w.scale))
        torch.cuda.synchronize()
        got = a.float().cpu().numpy().astype(np.float64)
        assert np.array_equal(got, run(lib, w, dev))
        check(got, ref(w), "fused merge, no-alloc scratch")


def test_llama8b_single_request_fused_plan(lib):
    # with the option on, the single-request workload keeps the fixed split
    # and each (sequence, kv-head group) is merged by the last of its chunks
    # to finish, in the attention kernel; within one bf16 spacing
    lib.set_option(lib.OPT_FUSED_MERGE, 1)
    w = W.make("llama8b")
    got = run(lib, w)
    check(got, ref(w), "llama8b fused")
