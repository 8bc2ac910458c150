"""Property tests of the two work splits of the attention kernel on random
small calls (hypothesis, derandomized so every run draws the same examples).

A latency-bound call takes the fixed split by default (every (sequence,
kv-head group) cut into chunks of whole steps, a workgroup's piece known from
its index, the merge finding a sequence's pieces from its length; a single
chunk per sequence, with no merge, where the stream-K plan has one
workgroup); with PDA_OPT_FIXED_SPLIT = 0 the same call is split stream-K over
the actual lengths.  The draws mix empty and short sequences with longer
ones, windows, several query tokens, every head size and pages of 1 to 32
tokens, so chunks past a sequence's end, single-chunk sequences, empty
sequences and window-shortened step ranges all occur.  Each output is held to
one bf16 spacing of the fp64 oracle (``attend_masked``), under both splits.
"""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
import workloads as W
from _gpu import check, log, q4, run_ext

pytestmark = pytest.mark.gpu

SETTINGS = dict(deadline=None, derandomize=True, database=None,
                suppress_health_check=[HealthCheck.too_slow, HealthCheck.function_scoped_fixture])

HEADS = [(8, 2), (16, 4), (32, 8), (12, 4), (40, 8), (16, 1)]


@st.composite
def small_calls(draw):
    hq, hkv = draw(st.sampled_from(HEADS))
    group = hq // hkv
    d = draw(st.sampled_from([64, 128, 256]))
    p = draw(st.sampled_from([1, 4, 16, 32]))
    nq = draw(st.sampled_from([q for q in (1, 2, 4) if q * group <= 16]))
    batch = draw(st.integers(1, 6))
    lens = draw(st.lists(st.one_of(st.just(0), st.integers(1, 40), st.integers(41, 3000)),
                         min_size=batch, max_size=batch))
    window = draw(st.one_of(st.just(0), st.integers(1, 2000)))
    seed = draw(st.integers(0, 2 ** 16))
    return hq, hkv, d, p, nq, lens, window, seed


@settings(max_examples=40, **SETTINGS)
@given(call=small_calls(), min_steps=st.sampled_from([0, 1, 2]))
def test_fixed_and_stream_k_splits_match_oracle(gpu_lib, call, min_steps):
    hq, hkv, d, p, nq, lens, window, seed = call
    w = W.build(lens, hq, hkv, d, p, seed=seed, pool="holes:0.1", num_queries=nq, window=window)
    ref = oracle.attend_masked(q4(w), w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale,
                               w.window)[0]
    try:
        gpu_lib.set_option(gpu_lib.OPT_MIN_STEPS, min_steps)
        for fixed in (1, 0):
            gpu_lib.set_option(gpu_lib.OPT_FIXED_SPLIT, fixed)
            log(f"split property case lens={lens} {hq}:{hkv} D={d} P={p} Tq={nq} W={window} "
                f"seed={seed} min_steps={min_steps} fixed={fixed}")
            check(run_ext(gpu_lib, w), ref, f"fixed split {fixed}")
    finally:
        gpu_lib.set_option(gpu_lib.OPT_FIXED_SPLIT, 1)
        gpu_lib.set_option(gpu_lib.OPT_MIN_STEPS, 0)
