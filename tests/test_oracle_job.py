"""The fanned-out oracle used by the full-size GPU parity checks assembles
the same array as the plain oracle called on the whole batch (CPU)."""
import dataclasses

import numpy as np

import _oracle_job as J
import oracle
import workloads as W


def test_pairs_assembly_matches_attend():
    w = W.build([0, 5, 40, 300], 12, 4, 64, 16, seed=3, pool="holes:0.2")
    ref = oracle.attend(w.q, w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale)[0]
    assert np.array_equal(J.full_reference(w, 1), ref)


def test_masked_assembly_matches_attend_masked():
    w = W.build([1, 3, 40, 300], 8, 2, 64, 16, seed=4, pool="holes:0.2")
    q4 = W._normal_bf16(np.random.default_rng(5), (4, 3, 8, 64))
    w = dataclasses.replace(w, q=q4, window=17)
    ref = oracle.attend_masked(q4, w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale, 17)[0]
    assert np.array_equal(J.full_reference(w, 1), ref)


def test_job_in_fresh_process(tmp_path):
    # the subprocess path the GPU tests use, with two forked workers
    job = J.start("tiny", str(tmp_path), workers=2)
    got = job.result(timeout=300)
    w = W.make("tiny")
    ref = oracle.attend(w.q, w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale)[0]
    assert np.array_equal(got, ref)
