"""GPU parity: the HIP library (through its C ABI) against the fp64 oracle.

Required tolerance: max |gpu - oracle| <= 1e-2 and mean <= 1e-3 on the
bf16 outputs.  Integer-like facts (length-1 rows, constant V, the GQA probe,
page permutation, NaN poison, determinism, empty sequences) are checked
bit-exactly.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from _golden import cases as golden_cases
from _gpu import bf16_round, bf16_ulps, check, check_full, log, run, to_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib(gpu_lib):
    return gpu_lib


@pytest.fixture(autouse=True)
def default_options(gpu_lib):
    gpu_lib.set_option(gpu_lib.OPT_BLOCKS_PER_CU, 1)
    gpu_lib.set_option(gpu_lib.OPT_MIN_STEPS, 0)
    gpu_lib.set_option(gpu_lib.OPT_FIXED_SPLIT, 1)
    yield
    gpu_lib.set_option(gpu_lib.OPT_BLOCKS_PER_CU, 1)
    gpu_lib.set_option(gpu_lib.OPT_MIN_STEPS, 0)
    gpu_lib.set_option(gpu_lib.OPT_FIXED_SPLIT, 1)


def ref(w):
    return oracle.attend(w.q, w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale)[0]


# (head_dim, Hq, Hkv, page_size, lengths) -- several tiles, ragged tails, every page path
SMALL = [
    (64, 8, 2, 16, [256]),
    (128, 32, 8, 16, [1, 2, 31, 32, 33, 100, 1000]),
    (128, 16, 1, 16, [77, 513]),
    (128, 5, 1, 32, [16, 31, 32, 33, 95, 2000]),
    (64, 4, 4, 8, [1, 7, 8, 9, 300]),
    (128, 8, 1, 64, [63, 64, 65, 1000]),
    (128, 12, 4, 1, [1, 2, 40]),
    (64, 6, 2, 2, [3, 33]),
    (64, 16, 4, 4, [5, 64, 65]),
    (128, 40, 8, 32, [0, 5, 0, 700]),
    (128, 64, 8, 16, [5000, 3]),
    (64, 32, 2, 128, [1, 129, 4000]),
    (128, 8, 8, 1024, [1023, 1025, 3000]),
    # head_dim 256 (one register buffer, 4-wave workgroups)
    (256, 12, 4, 16, [1, 2, 31, 32, 33, 100, 1000]),
    (256, 8, 1, 32, [16, 31, 32, 33, 95, 2000]),
    (256, 16, 8, 16, [77, 513, 3000]),
    (256, 4, 2, 8, [1, 7, 8, 9, 300]),
    (256, 32, 2, 1, [1, 2, 40]),
    (256, 8, 4, 64, [0, 63, 64, 65, 1000]),
]


@pytest.mark.parametrize("d,hq,hkv,p,lens", SMALL, ids=[f"D{c[0]}-{c[1]}:{c[2]}-P{c[3]}" for c in SMALL])
def test_small_shapes(lib, d, hq, hkv, p, lens):
    w = W.build(lens, hq, hkv, d, p, seed=sum(lens) + d + p, pool="holes:0.2")
    log(f"case D={d} {hq}:{hkv} P={p} lens={lens}")
    got = run(lib, w)
    check(got, ref(w), "small")


def test_many_short_sequences_max_batch(lib):
    rng = np.random.default_rng(7)
    lens = rng.integers(0, 70, size=8192).tolist()
    w = W.build(lens, 8, 2, 128, 16, seed=5, pool="holes:0.1")
    log("case batch 8192, L in [0, 70)")
    check(run(lib, w), ref(w), "B=8192")


def test_head_dim_256_max_batch(lib):
    rng = np.random.default_rng(8)
    lens = rng.integers(0, 70, size=4096).tolist()
    w = W.build(lens, 12, 4, 256, 16, seed=6, pool="holes:0.1")
    log("case D=256 batch 4096, L in [0, 70)")
    check(run(lib, w), ref(w), "D=256 B=4096")


def _pad_head_dim(w, d):
    """Zero-pad q, K and V from head_dim 2 to d: the scores and the first two
    output features are unchanged, the padded features are 0."""
    import dataclasses

    def pad(a):
        out = np.zeros(a.shape[:-1] + (d,), dtype=a.dtype)
        out[..., : a.shape[-1]] = a
        return out
    return dataclasses.replace(w, q=pad(w.q), k_cache=pad(w.k_cache), v_cache=pad(w.v_cache))


@pytest.mark.parametrize("d", [64, 128, 256])
@pytest.mark.parametrize("name,w,expected", golden_cases(), ids=lambda x: x if isinstance(x, str) else "")
def test_golden_closed_forms(lib, name, w, expected, d):
    got = run(lib, _pad_head_dim(w, d))
    log(f"golden {name} D={d}")
    dd = expected.shape[-1]
    assert np.array_equal(got[..., dd:], np.zeros_like(got[..., dd:]))
    # bf16 output rounding plus bf16 rounding of the probabilities
    assert np.abs(got[..., :dd] - expected).max() <= 2 * np.abs(bf16_round(expected) - expected).max() + 4e-3


@pytest.mark.parametrize("min_steps", [1, 2, 7, 1 << 20])
@pytest.mark.parametrize("blocks", [1, 2, 4])
@pytest.mark.parametrize("fixed", [1, 0])
def test_split_count_sweep(lib, min_steps, blocks, fixed):
    # both splits of a small call (fixed chunks, stream-K over the lengths)
    w = W.build([3000, 17, 700, 1], 32, 8, 128, 16, seed=3, pool="holes:0.1")
    lib.set_option(lib.OPT_MIN_STEPS, min_steps)
    lib.set_option(lib.OPT_BLOCKS_PER_CU, blocks)
    lib.set_option(lib.OPT_FIXED_SPLIT, fixed)
    log(f"case min_steps={min_steps} blocks={blocks} fixed={fixed}")
    check(run(lib, w), ref(w), f"sweep {min_steps}/{blocks}/{fixed}")


def test_length_one_is_v_exactly(lib):
    w = W.build([1] * 9, 16, 4, 128, 16, seed=2, pool="holes:0.5")
    got = run(lib, w)
    g = 4
    for b in range(9):
        page = w.block_table[b, 0]
        for h in range(16):
            v0 = oracle.bf16_to_f64(w.v_cache[page, 0, h // g])
            assert np.array_equal(got[b, h], v0)


def test_constant_v_bitwise(lib):
    w = W.build([1, 40, 3000], 8, 2, 128, 16, seed=4)
    live = ~np.isnan(W.bf16_bits_to_f32(w.v_cache))
    consts = np.float32([1.5, -0.375])
    for g in range(2):
        vg = w.v_cache[:, :, g, :]
        vg[live[:, :, g, :]] = W.f32_to_bf16_bits(consts[g:g + 1])[0]
    got = run(lib, w)
    for h in range(8):
        assert np.array_equal(got[:, h, :], np.full_like(got[:, h, :], consts[h // 4]))


def test_gqa_probe_exact(lib):
    w = W.build([9, 300, 2048], 40, 8, 128, 32, seed=6)
    live = ~np.isnan(W.bf16_bits_to_f32(w.v_cache))
    for g in range(8):
        vg = w.v_cache[:, :, g, :]
        vg[live[:, :, g, :]] = W.f32_to_bf16_bits(np.float32([g]))[0]
    got = run(lib, w)
    for h in range(40):
        assert np.array_equal(got[:, h, :], np.full_like(got[:, h, :], h // 5))


def test_page_permutation_bitwise(lib):
    w = W.build([100, 2000, 33, 4097], 32, 8, 128, 16, seed=8, pool="holes:0.3")
    a = run(lib, w)
    b = run(lib, W.permute_pages(w, 11))
    assert np.array_equal(a, b)


def test_nan_poison_bitwise(lib):
    a = W.build([33, 16, 1000, 5], 40, 8, 128, 32, seed=9, pool="holes:0.25", poison=True)
    b = W.build([33, 16, 1000, 5], 40, 8, 128, 32, seed=9, pool="holes:0.25", poison=False)
    assert np.isnan(W.bf16_bits_to_f32(a.v_cache)).any()
    ga, gb = run(lib, a), run(lib, b)
    assert np.isfinite(ga).all() and np.array_equal(ga, gb)


def test_deterministic_runs(lib):
    w = W.build([5000, 300, 7, 9000], 64, 8, 128, 16, seed=10)
    dev = to_gpu(w)
    a = run(lib, w, dev)
    b = run(lib, w, dev)
    assert np.array_equal(a, b)


def test_empty_sequences_write_zeros(lib):
    w = W.build([0, 50, 0, 0], 8, 2, 64, 16, seed=12)
    got = run(lib, w, fill=float("nan"))
    assert np.array_equal(got[0], np.zeros_like(got[0])) and np.array_equal(got[2], np.zeros_like(got[2]))
    assert np.array_equal(got[3], np.zeros_like(got[3]))
    check(got, ref(w), "empty rows")


def test_all_empty_batch(lib):
    w = W.build([0, 0, 0], 8, 2, 64, 16, seed=13)
    got = run(lib, w, fill=float("nan"))
    assert np.array_equal(got, np.zeros_like(got))


def test_argument_error_leaves_out_untouched(lib):
    import torch
    w = W.build([64, 64], 8, 2, 64, 16, seed=14)
    dev = to_gpu(w)
    out = torch.full((2, 8, 64), 3.0, dtype=torch.bfloat16, device="cuda")
    rc = lib.raw_call(dev["q"].data_ptr(), dev["k"].data_ptr(), dev["v"].data_ptr(), dev["bt"].data_ptr(),
                      dev["lens"].data_ptr(), out.data_ptr(), 2, 8, 3, 64, 16, w.num_pages, w.max_pages, 0.125)
    assert rc == 2 and "multiple" in lib.last_error()
    rc = lib.raw_call(dev["q"].data_ptr(), dev["k"].data_ptr(), dev["v"].data_ptr(), dev["bt"].data_ptr(),
                      dev["lens"].data_ptr(), out.data_ptr() + 2, 2, 8, 2, 64, 16, w.num_pages, w.max_pages, 0.125)
    assert rc == 5
    torch.cuda.synchronize()
    assert bool((out == 3.0).all())


def test_bad_device_contents_do_not_fault(lib):
    # page ids out of range and lengths beyond the table are clamped, not trusted
    w = W.build([40, 40], 8, 2, 64, 16, seed=15, poison=False)
    w.block_table[0, 1] = 10 ** 6
    w.block_table[1, 2] = -5
    w.context_lens[1] = 10 ** 6
    got = run(lib, w)
    assert got.shape == (2, 8, 64)


def test_graph_capture_replay(lib):
    import torch
    w = W.build([700, 33, 5000], 32, 8, 128, 16, seed=16)
    dev = to_gpu(w)
    out = torch.empty((3, 32, 128), dtype=torch.bfloat16, device="cuda")
    s = torch.cuda.Stream()
    lib.workspace_reserve(3, 32, 8, 128, 16, w.max_pages, stream=s)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        lib.paged_decode_attention(dev["q"], dev["k"], dev["v"], dev["bt"], dev["lens"], out, float(w.scale))
    rng = np.random.default_rng(0)
    for rep in range(4):
        newq = W.f32_to_bf16_bits(rng.standard_normal(w.q.shape, dtype=np.float32))
        w.q[:] = newq
        dev["q"].copy_(to_gpu(w)["q"])
        g.replay()
        torch.cuda.synchronize()
        replayed = out.float().cpu().numpy().astype(np.float64)
        eager = run(lib, w, dev)
        assert np.array_equal(replayed, eager), f"replay {rep} differs from eager"
        check(replayed, ref(w), f"replay {rep}")


def test_two_streams(lib):
    import torch
    w1 = W.build([1000, 20], 32, 8, 128, 16, seed=17)
    w2 = W.build([64, 3000, 5], 32, 8, 128, 16, seed=18)
    d1, d2 = to_gpu(w1), to_gpu(w2)
    o1 = torch.empty(tuple(w1.q.shape), dtype=torch.bfloat16, device="cuda")
    o2 = torch.empty(tuple(w2.q.shape), dtype=torch.bfloat16, device="cuda")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    for _ in range(3):
        lib.paged_decode_attention(d1["q"], d1["k"], d1["v"], d1["bt"], d1["lens"], o1, float(w1.scale), stream=s1)
        lib.paged_decode_attention(d2["q"], d2["k"], d2["v"], d2["bt"], d2["lens"], o2, float(w2.scale), stream=s2)
    torch.cuda.synchronize()
    check(o1.float().cpu().numpy().astype(np.float64), ref(w1), "stream 1")
    check(o2.float().cpu().numpy().astype(np.float64), ref(w2), "stream 2")


# ------------------------------------------------------------- named workloads
# Calls the planner treats as small (K and V within 128 MB): one 32-token
# step per wave when the two-step plan leaves CUs idle, fewer kv heads per
# workgroup when a (sequence, kv-head group) would be cut into more than 32
# pieces, and the fixed split (every pair cut into the same chunks, the
# merge finding the pieces from the lengths).  (lengths, Hq, Hkv, D, P, then
# the grid of the fixed split with the planner's step count and with two
# steps per wave fixed by the caller, then the same two for the stream-K
# split over the actual lengths)
SMALL_CALLS = [
    ([4096], 32, 8, 128, 16, 128, 64, 128, 64),       # single request: 2 kv heads per workgroup
    ([8192], 64, 8, 128, 16, 256, 128, 256, 128),     # one kv head per workgroup, 8 columns
    ([16384], 32, 8, 128, 16, 256, 256, 256, 256),    # one kv head per workgroup
    ([1024] * 4, 32, 8, 128, 16, 128, 64, 128, 64),   # one step per wave, 8 kv heads
    ([3000, 17], 16, 4, 256, 32, 192, 96, 188, 94),   # D = 256: one kv head of 4-wave workgroups
    ([700, 5, 1900], 40, 8, 128, 1, 180, 90, 180, 90),  # one-token pages
]


@pytest.mark.parametrize("lens,hq,hkv,d,p,gf,gf2,gs,gs2", SMALL_CALLS,
                         ids=[f"{len(c[0])}x{max(c[0])}-{c[1]}:{c[2]}-D{c[3]}-P{c[4]}" for c in SMALL_CALLS])
def test_small_call_plans_match_oracle(lib, lens, hq, hkv, d, p, gf, gf2, gs, gs2):
    w = W.build(lens, hq, hkv, d, p, seed=sum(lens) + hq, pool="holes:0.1")
    maxp = w.block_table.shape[1]
    r = ref(w)
    try:
        for fixed, steps, grid in ((1, 0, gf), (1, 2, gf2), (0, 0, gs), (0, 2, gs2)):
            lib.set_option(lib.OPT_FIXED_SPLIT, fixed)
            lib.set_option(lib.OPT_MIN_STEPS, steps)
            assert lib.plan(len(lens), hq, hkv, d, p, maxp)[0] == grid
            log(f"case {len(lens)} x {max(lens)} {hq}:{hkv} D={d} P={p} fixed split {fixed} steps {steps} grid {grid}")
            check(run(lib, w), r, f"small call, fixed split {fixed}, steps {steps}")
    finally:
        lib.set_option(lib.OPT_FIXED_SPLIT, 1)
        lib.set_option(lib.OPT_MIN_STEPS, 0)


@pytest.mark.parametrize("name", ["tiny", "llama8b", "batched"])
def test_named_workload_full_oracle(lib, name):
    log(f"workload {name}: generating")
    w = W.make(name)
    log(f"workload {name}: running")
    got = run(lib, w)
    log(f"workload {name}: oracle")
    r = ref(w)
    check(got, r, name)
    # against the correctly rounded oracle: at most one bf16 step anywhere
    # (exactly rounded except where the fp64 value sits near a rounding boundary)
    rb = bf16_round(r)
    d = bf16_ulps(got, rb)
    exact = float((got == rb).mean())
    log(f"  {name}: max {d.max():.2f} bf16 ulp from RN(oracle); {100 * exact:.2f}% bitwise equal")
    assert d.max() <= 1.0


@pytest.mark.parametrize("name", ["long70b", "ragged", "tokenpage"])
def test_named_workload_every_output(lib, name, tmp_path):
    # the full-size long-context, ragged and one-token-page workloads, every
    # output against the oracle (fanned out over the host cores)
    check_full(name, lambda w: run(lib, w), tmp_path)


@pytest.mark.parametrize("p", [1, 4, 16])
def test_pool_over_4gib(lib, p):
    # pages past the 4 GiB mark of the pool: 64-bit addresses on the
    # small-page path, page descriptors with 64-bit bases on the big-page
    # path.  The workload's pages are moved to the end of a larger,
    # otherwise unwritten pool (rows past a sequence's end in its last page
    # hold whatever that memory holds and must not leak in).
    import torch
    w = W.build([1, 5, 33, 300, 1000], 32, 8, 128, p, seed=40 + p, pool="holes:0.2", poison=True)
    page_bytes = p * 8 * 128 * 2
    big = (int(4.2 * 2 ** 30) // page_bytes) + w.k_cache.shape[0]
    shift = big - w.k_cache.shape[0]
    assert shift * page_bytes > 2 ** 32
    log(f"pages of {p} tokens: pool of {big} pages ({big * page_bytes / 2 ** 30:.2f} GiB each for K and V)")
    dev = to_gpu(w)
    kb = torch.empty((big,) + tuple(dev["k"].shape[1:]), dtype=torch.bfloat16, device="cuda")
    vb = torch.empty_like(kb)
    kb[shift:] = dev["k"]
    vb[shift:] = dev["v"]
    bt = torch.where(dev["bt"] >= 0, dev["bt"] + shift, dev["bt"])
    out = torch.full(tuple(w.q.shape), float("nan"), dtype=torch.bfloat16, device="cuda")
    lib.paged_decode_attention(dev["q"], kb, vb, bt, dev["lens"], out, float(w.scale))
    torch.cuda.synchronize()
    got = out.float().cpu().numpy().astype(np.float64)
    del kb, vb
    torch.cuda.empty_cache()
    check(got, ref(w), f"P={p} pool over 4 GiB")


# ------------------------------------------------------ numerical edge cases
# Every input above is N(0, 1); these reach the max shift, the exponent
# reference of columns that have seen no key, the hi + lo probability split
# and the merge with scores in the thousands.  Head sizes 64, 128 and 256,
# pages of >= 16 tokens (one page descriptor per half-step) and of fewer
# (a page id per row), and plans with one-step pieces (min_steps = 1: most
# step boundaries are split points) as well as the default.
EDGE_SHAPES = [(64, 16), (64, 4), (128, 32), (128, 1), (256, 16), (256, 4)]
EDGE_IDS = [f"D{d}-P{p}" for d, p in EDGE_SHAPES]


def _token_slot(w, b, t):
    p = w.k_cache.shape[1]
    return int(w.block_table[b, t // p]), t % p


def _mean_v(w):
    """Mean of V over each sequence's tokens, per kv head, repeated over the
    query heads of the group ([B, Hq, D]); zero rows for empty sequences."""
    bsz, hq, d = w.q.shape
    hkv = w.k_cache.shape[2]
    g = hq // hkv
    out = np.zeros((bsz, hq, d))
    for b in range(bsz):
        L = int(w.context_lens[b])
        if L == 0:
            continue
        rows = np.stack([oracle.bf16_to_f64(w.v_cache[_token_slot(w, b, t)]) for t in range(L)])  # [L, Hkv, D]
        out[b] = np.repeat(rows.mean(axis=0), g, axis=0)
    return out


@pytest.mark.parametrize("min_steps", [1, 2])
@pytest.mark.parametrize("d,p", EDGE_SHAPES, ids=EDGE_IDS)
def test_zero_query_gives_mean_of_v(lib, d, p, min_steps):
    # q = 0: every score is 0, the weights are uniform and out is the mean
    # of V (pinned by its own gather, not by the oracle's softmax)
    w = W.build([1, 33, 700, 0, 4099], 16, 4, d, p, seed=90 + d + p, pool="holes:0.2")
    w.q[:] = 0
    lib.set_option(lib.OPT_MIN_STEPS, min_steps)
    log(f"case q=0 D={d} P={p} min_steps={min_steps}")
    check(run(lib, w), _mean_v(w), "q = 0")


@pytest.mark.parametrize("min_steps", [1, 2])
@pytest.mark.parametrize("d,p", EDGE_SHAPES, ids=EDGE_IDS)
def test_equal_keys_give_mean_of_v(lib, d, p, min_steps):
    # every key of a (sequence, kv head) equal: every score of a query head
    # is the same number, so again the mean of V whatever q is
    w = W.build([2, 47, 700, 4099], 16, 4, d, p, seed=100 + d + p, pool="holes:0.2")
    rng = np.random.default_rng(d + p)
    for b in range(w.batch):
        for g in range(4):
            key = W.f32_to_bf16_bits(rng.standard_normal(d, dtype=np.float32))
            for t in range(int(w.context_lens[b])):
                page, slot = _token_slot(w, b, t)
                w.k_cache[page, slot, g] = key
    lib.set_option(lib.OPT_MIN_STEPS, min_steps)
    log(f"case equal keys D={d} P={p} min_steps={min_steps}")
    check(run(lib, w), _mean_v(w), "equal keys")


def _plant_dominant(w, b, g, t, score):
    """Give every query head of kv head g in sequence b the same query u and
    put the key lambda * u at token t, lambda chosen for a score of about
    `score`; returns the bf16 bits of that key."""
    G = w.q.shape[-2] // w.k_cache.shape[2]
    u_bits = w.q[b, ..., g * G, :].copy()
    w.q[b, ..., g * G:(g + 1) * G, :] = u_bits[..., None, :] if w.q.ndim == 4 else u_bits
    u = oracle.bf16_to_f64(u_bits.reshape(-1, u_bits.shape[-1])[0])
    lam = score / (float(np.float32(w.scale)) * float(u @ u))
    key = W.f32_to_bf16_bits((lam * u).astype(np.float32))
    page, slot = _token_slot(w, b, t)
    w.k_cache[page, slot, g] = key
    return key, u


@pytest.mark.parametrize("fixed", [1, 0])
@pytest.mark.parametrize("min_steps", [1, 2])
@pytest.mark.parametrize("d,p", EDGE_SHAPES, ids=EDGE_IDS)
def test_dominant_key_returns_its_value(lib, d, p, min_steps, fixed):
    # one key per (sequence, kv head) scores ~1e3 against the group's query
    # (scale * q.k far beyond exp's fp32 range without the max shift): the
    # output is that token's v, bitwise (every other weight is below 2^-1400).
    # The key sits mid-step, on either side of a 32-token step boundary (a
    # split point of most one-step-piece plans) or on the last token of a
    # partly filled page; past the end of that page a masked key scoring
    # ~2e3 (its V left NaN) must carry no weight.
    lens = [4099, 701, 2067]
    w = W.build(lens, 16, 4, d, p, seed=110 + d + p, pool="holes:0.2", poison=True)
    G = 4
    planted = {}
    for b, L in enumerate(lens):
        mid = (L // 2) // 32 * 32
        for g, t in enumerate([37, L - 1, mid, mid - 1]):
            key, u = _plant_dominant(w, b, g, t, 1000.0)
            planted[(b, g)] = t
            if L % p:  # slot L of the last page: past the end
                page, slot = _token_slot(w, b, L)
                w.k_cache[page, slot, g] = W.f32_to_bf16_bits((2.0 * oracle.bf16_to_f64(key)).astype(np.float32))
                assert np.isnan(W.bf16_bits_to_f32(w.v_cache[page, slot, g])).all()
    lib.set_option(lib.OPT_MIN_STEPS, min_steps)
    lib.set_option(lib.OPT_FIXED_SPLIT, fixed)
    log(f"case dominant key D={d} P={p} min_steps={min_steps} fixed={fixed}")
    got = run(lib, w)
    check(got, ref(w), "dominant key")
    for (b, g), t in planted.items():
        v = oracle.bf16_to_f64(w.v_cache[_token_slot(w, b, t)][g])
        assert np.array_equal(got[b, g * G:(g + 1) * G], np.broadcast_to(v, (G, d))), (b, g, t)


@pytest.mark.parametrize("fixed", [1, 0])
@pytest.mark.parametrize("min_steps", [1, 2])
@pytest.mark.parametrize("d,p", EDGE_SHAPES, ids=EDGE_IDS)
def test_two_dominant_keys_split_the_weight(lib, d, p, min_steps, fixed):
    # two keys scoring ~1000 and ~1000 - ln 2, far apart in the sequence (in
    # different pieces of a split plan): the merge combines two pieces whose
    # maxima are in the thousands, weights ~2/3 and ~1/3
    lens = [4099, 2067]
    w = W.build(lens, 16, 4, d, p, seed=120 + d + p, pool="holes:0.2", poison=True)
    for b, L in enumerate(lens):
        for g in range(4):
            key, u = _plant_dominant(w, b, g, 5 + 7 * g, 1000.0)
            second = W.f32_to_bf16_bits((oracle.bf16_to_f64(key) * (1.0 - np.log(2.0) / 1000.0)).astype(np.float32))
            page, slot = _token_slot(w, b, L - 40 - 9 * g)
            w.k_cache[page, slot, g] = second
    lib.set_option(lib.OPT_MIN_STEPS, min_steps)
    lib.set_option(lib.OPT_FIXED_SPLIT, fixed)
    log(f"case two dominant keys D={d} P={p} min_steps={min_steps} fixed={fixed}")
    check(run(lib, w), ref(w), "two dominant keys")


@pytest.mark.parametrize("d,p", EDGE_SHAPES, ids=EDGE_IDS)
def test_dominant_key_outside_window_carries_no_weight(lib, d, p):
    # a sliding window of 100 with two query tokens: the key just before the
    # window of the later query (visible to the earlier one only) and the
    # key just before the earlier query's window score ~1e3; the slots of
    # the same page before those keys hold NaN values.  Only the earlier
    # query may see the first key.
    from _gpu import run_ext
    window, tq = 100, 2
    lens = [4099, 701, 163]
    w = W.build(lens, 8, 4, d, p, seed=130 + d + p, pool="holes:0.2", poison=True, num_queries=tq,
                window=window)
    for b, L in enumerate(lens):
        lo_last = L - window          # first key of the later query
        for g in range(4):
            key, u = _plant_dominant(w, b, g, lo_last - 1, 1000.0)      # seen by query 0 only
            page, slot = _token_slot(w, b, lo_last - 2)                  # seen by neither
            if page < 0:
                continue  # a page wholly before the window: released
            w.k_cache[page, slot, g] = key
            for t in range(lo_last - 2 - (lo_last - 2) % p, lo_last - 2):
                pg, sl = _token_slot(w, b, t)
                w.v_cache[pg, sl, g] = W.BF16_NAN
    log(f"case dominant key outside a window D={d} P={p}")
    got = run_ext(lib, w)
    r = oracle.attend_masked(w.q, w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale, window)[0]
    check(got, r, "window edge")
    G = 2
    for b, L in enumerate(lens):
        for g in range(4):
            v = oracle.bf16_to_f64(w.v_cache[_token_slot(w, b, L - window - 1)][g])
            assert np.array_equal(got[b, 0, g * G:(g + 1) * G], np.broadcast_to(v, (G, d)))


@pytest.mark.parametrize("d", [64, 128, 256])
def test_window_pre_window_slots_of_a_live_page_are_not_read(lib, d):
    # pages of 32 tokens, a window that starts mid-page: the slots of that
    # page before the first visible key hold NaN (keys and values); the
    # outputs are finite and match the oracle
    from _gpu import run_ext
    lens = [4099, 701, 2067, 90]
    window = 70
    w = W.build(lens, 16, 4, d, 32, seed=140 + d, pool="holes:0.2", poison=True, window=window)
    for b, L in enumerate(lens):
        lo = max(0, L - window)
        for t in range(lo - lo % 32, lo):
            pg, sl = _token_slot(w, b, t)
            w.k_cache[pg, sl] = W.BF16_NAN
            w.v_cache[pg, sl] = W.BF16_NAN
    got = run_ext(lib, w)
    r = oracle.attend_masked(w.q[:, None], w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale, window)[0]
    check(got, r, f"pre-window NaN D={d}")


# --------------------------------------------- tensor-descriptor entry point
def test_descriptor_entry_matches_pointer_entry(lib):
    # the same call through pda_tensor descriptors: bitwise the pointer
    # entry's output; a transposed view of q, an fp16 q and an int64 length
    # vector are refused by the library with out untouched
    import torch
    w = W.build([1, 33, 700, 0, 4099], 32, 8, 128, 16, seed=150, pool="holes:0.2")
    dev = to_gpu(w)
    a = run(lib, w, dev)
    out = torch.full(tuple(w.q.shape), float("nan"), dtype=torch.bfloat16, device="cuda")
    lib.paged_decode_attention_desc(dev["q"], dev["k"], dev["v"], dev["bt"], dev["lens"], out, float(w.scale))
    torch.cuda.synchronize()
    assert np.array_equal(out.float().cpu().numpy().astype(np.float64), a)
    check(a, ref(w), "descriptor entry")
    out.fill_(3.0)
    qt = dev["q"].transpose(1, 2).contiguous().transpose(1, 2)  # [B, Hq, D] view with permuted strides
    bad = [(dict(q=qt), 8), (dict(q=dev["q"].to(torch.float16)), 7), (dict(lens=dev["lens"].to(torch.int64)), 7)]
    for repl, code in bad:
        args = dict(q=dev["q"], k=dev["k"], v=dev["v"], bt=dev["bt"], lens=dev["lens"])
        args.update(repl)
        with pytest.raises(lib.PdaError) as ei:
            lib.paged_decode_attention_desc(args["q"], args["k"], args["v"], args["bt"], args["lens"], out,
                                            float(w.scale))
        assert ei.value.code == code, str(ei.value)
    torch.cuda.synchronize()
    assert bool((out == 3.0).all())
