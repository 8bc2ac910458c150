"""GPU parity of the vector-ALU compute path (PDA_OPT_COMPUTE_PATH = 1):
the same stream-K pass over the paged KV with QK^T as bf16 dot2 products
added across lanes by DPP, the online softmax on the vector ALU and P.V as
fp32 FMAs.  It exists to measure the matrix-core path against, so it is held
to the same bar: the required tolerance and one bf16 spacing of the fp64
oracle, bitwise invariance to page order and NaN poison, and determinism.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from _gpu import bf16_ulps, check, check_full, log, run, to_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib(gpu_lib):
    return gpu_lib


@pytest.fixture(autouse=True)
def valu_path(gpu_lib):
    gpu_lib.set_option(gpu_lib.OPT_BLOCKS_PER_CU, 1)
    gpu_lib.set_option(gpu_lib.OPT_MIN_STEPS, 0)
    gpu_lib.set_option(gpu_lib.OPT_COMPUTE_PATH, 1)
    yield
    gpu_lib.set_option(gpu_lib.OPT_COMPUTE_PATH, 0)
    gpu_lib.set_option(gpu_lib.OPT_BLOCKS_PER_CU, 1)
    gpu_lib.set_option(gpu_lib.OPT_MIN_STEPS, 0)


def ref(w):
    return oracle.attend(w.q, w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale)[0]


def q4(w):
    return w.q if w.q.ndim == 4 else w.q[:, None]


def ref_masked(w):
    return oracle.attend_masked(q4(w), w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale,
                                w.window)[0]


def run_ext(lib, w):
    import torch
    dev = to_gpu(w)
    q = dev["q"] if dev["q"].dim() == 4 else dev["q"].unsqueeze(1)
    out = torch.full(tuple(q.shape), float("nan"), dtype=torch.bfloat16, device="cuda")
    lib.paged_decode_attention_ext(q.contiguous(), dev["k"], dev["v"], dev["bt"], dev["lens"], out,
                                   float(w.scale), window=w.window)
    torch.cuda.synchronize()
    return out.float().cpu().numpy().astype(np.float64)


# (Hq, Hkv, page_size, lengths): groups of 1 to 8 (4- and 8-column kernels),
# ragged tails, partial pages, empty sequences
SHAPES = [
    (32, 8, 16, [1, 2, 31, 32, 33, 100, 1000]),
    (40, 8, 32, [0, 16, 31, 32, 33, 95, 2000]),
    (64, 8, 16, [5000, 3, 1]),
    (8, 1, 16, [77, 513]),
    (24, 8, 64, [63, 64, 65, 1000]),
    (8, 8, 16, [1, 17, 40, 900]),
    (12, 4, 1024, [1023, 1025, 3000]),
    (6, 2, 16, [0, 0, 70]),
]


@pytest.mark.parametrize("hq,hkv,p,lens", SHAPES, ids=[f"{c[0]}:{c[1]}-P{c[2]}" for c in SHAPES])
def test_valu_small_shapes(lib, hq, hkv, p, lens):
    w = W.build(lens, hq, hkv, 128, p, seed=sum(lens) + hq + p, pool="holes:0.2")
    log(f"valu case {hq}:{hkv} P={p} lens={lens}")
    check(run(lib, w), ref(w), "valu")


@pytest.mark.parametrize("min_steps,blocks", [(1, 1), (1, 4), (7, 2), (1 << 20, 1)])
def test_valu_split_sweep(lib, min_steps, blocks):
    lib.set_option(lib.OPT_MIN_STEPS, min_steps)
    lib.set_option(lib.OPT_BLOCKS_PER_CU, blocks)
    for hq in (32, 64):
        w = W.build([3000, 17, 700, 1], hq, 8, 128, 16, seed=3 + hq, pool="holes:0.1")
        log(f"valu sweep min_steps={min_steps} blocks/CU={blocks} Hq={hq}")
        check(run(lib, w), ref(w), f"sweep {min_steps}/{blocks}")


# (Hq, Hkv, lengths, query tokens, window): up to 8 columns per kv head
MASKED = [
    (32, 8, [1, 2, 31, 32, 33, 100, 1000], 2, 0),
    (32, 8, [5, 33, 66, 1027, 3000], 2, 100),
    (40, 8, [7, 700, 4099], 1, 64),
    (8, 8, [1, 17, 40, 900], 8, 0),
    (16, 8, [20, 900], 4, 30),
    (12, 4, [0, 1, 2, 3, 4], 2, 0),
]


@pytest.mark.parametrize("hq,hkv,lens,tq,window", MASKED,
                         ids=[f"{c[0]}:{c[1]}-T{c[3]}-W{c[4]}" for c in MASKED])
def test_valu_masked(lib, hq, hkv, lens, tq, window):
    w = W.build(lens, hq, hkv, 128, 16, seed=sum(lens) + 13 * tq + window, pool="holes:0.2", num_queries=tq,
                window=window)
    log(f"valu masked {hq}:{hkv} lens={lens} Tq={tq} W={window}")
    check(run_ext(lib, w), ref_masked(w), "valu masked")


def test_valu_length_one_is_v_exactly(lib):
    w = W.build([1] * 9, 32, 8, 128, 16, seed=2, pool="holes:0.5")
    got = run(lib, w)
    for b in range(9):
        page = w.block_table[b, 0]
        for h in range(32):
            assert np.array_equal(got[b, h], oracle.bf16_to_f64(w.v_cache[page, 0, h // 4]))


def test_valu_page_permutation_and_poison_bitwise(lib):
    a = W.build([100, 2000, 33, 4097], 64, 8, 128, 16, seed=8, pool="holes:0.3", poison=True)
    b = W.build([100, 2000, 33, 4097], 64, 8, 128, 16, seed=8, pool="holes:0.3", poison=False)
    ga = run(lib, a)
    assert np.isfinite(ga).all()
    assert np.array_equal(ga, run(lib, b))
    assert np.array_equal(ga, run(lib, W.permute_pages(a, 11)))
    assert np.array_equal(ga, run(lib, a))  # deterministic


def test_valu_agrees_with_matrix_cores(lib):
    w = W.build([5000, 300, 7, 9000], 64, 8, 128, 16, seed=10)
    got = run(lib, w)
    lib.set_option(lib.OPT_COMPUTE_PATH, 0)
    mfma = run(lib, w)
    r = ref(w)
    check(got, r, "valu")
    check(mfma, r, "mfma")
    # both are within one bf16 spacing of the same fp64 value
    assert bf16_ulps(got, mfma).max() <= 2.0


def test_valu_unsupported_shapes_fail_loudly(lib):
    w64 = W.build([40], 8, 2, 64, 16, seed=1)
    with pytest.raises(RuntimeError, match="vector-ALU"):
        run(lib, w64)
    w16 = W.build([40], 16, 1, 128, 16, seed=1)  # 16 columns
    with pytest.raises(RuntimeError, match="vector-ALU"):
        run(lib, w16)
    wp = W.build([40], 8, 2, 128, 8, seed=1)  # pages below 16 tokens
    with pytest.raises(RuntimeError, match="vector-ALU"):
        run(lib, wp)


def test_valu_long70b_every_output(lib, tmp_path):
    check_full("long70b", lambda w: run(lib, w), tmp_path)


def test_valu_batched_full_oracle(lib):
    log("workload batched: generating")
    w = W.make("batched")
    check(run(lib, w), ref(w), "batched valu")
