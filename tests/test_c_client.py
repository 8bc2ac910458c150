"""The library from a plain C program (tests/c/pda_client.c), with no Python
between the caller and the C ABI: include/pda.h compiles as C11 with warnings
as errors, the argument checks return the documented codes (CPU), and a
decode-attention call made with device memory and a stream from the HIP
runtime's C API matches the fp64 oracle (GPU)."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
import workloads as W
from paper_2606_07665_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c", "pda_client.c")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


@pytest.fixture(scope="module")
def client(tmp_path_factory):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc is not installed")
    if not os.path.exists(B.LIB_PATH):
        raise RuntimeError(f"HIP library not built: {B.LIB_PATH}")
    lib_dir = os.path.dirname(B.LIB_PATH)
    exe = str(tmp_path_factory.mktemp("c_client") / "pda_client")
    cmd = [gcc, "-std=c11", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"), SRC, "-o", exe,
           "-L", lib_dir, "-lpda", f"-Wl,-rpath,{lib_dir}",
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}", "-lm"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stdout + res.stderr
    return exe


def test_c_client_argument_checks(client):
    res = subprocess.run([client, "errors"], capture_output=True, text=True, timeout=60)
    assert res.returncode == 0, res.stdout + res.stderr
    for what in ("null q", "head_dim 96", "misaligned q", "nan scale", "empty batch", "version", "plan shape"):
        assert f"ok {what}" in res.stdout, res.stdout
    # every validation error of the descriptor entry point, forced from C
    for what in ("null descriptor", "null data", "fp16 q", "int64 lengths", "q rank", "block_table rows",
                 "heads not a multiple", "head_dim 96", "page_size 24", "transposed q", "padded block_table",
                 "nan scale"):
        assert f"ok desc {what}" in res.stdout, res.stdout


@pytest.mark.gpu
def test_c_client_decode_matches_oracle(client, tmp_path, gpu_lib):
    from _gpu import check, log
    # ragged lengths (one token, a partial page, an empty sequence, several
    # steps) in a pool with NaN-poisoned holes
    w = W.build([1, 17, 300, 0, 2049], 32, 8, 128, 16, seed=21, pool="holes:0.3", poison=True)
    batch, hq, d = w.q.shape
    num_pages, page, hkv, _ = w.k_cache.shape
    maxp = w.block_table.shape[1]
    (tmp_path / "meta.txt").write_text(
        f"{batch} {hq} {hkv} {d} {page} {num_pages} {maxp} {float(np.float32(w.scale)):.9g}\n")
    for name, arr in (("q", w.q), ("k", w.k_cache), ("v", w.v_cache), ("bt", w.block_table),
                      ("lens", w.context_lens)):
        np.ascontiguousarray(arr).tofile(tmp_path / f"{name}.bin")
    log(f"C client: batch {batch} {hq}:{hkv} D={d} P={page} lens={[int(x) for x in w.context_lens]}")
    res = subprocess.run([client, "run", str(tmp_path)], capture_output=True, text=True, timeout=120)
    log(res.stdout)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "ok outputs bitwise equal across streams" in res.stdout
    assert "ok graph replays bitwise equal" in res.stdout
    out = np.fromfile(tmp_path / "out.bin", dtype=np.uint16).reshape(w.q.shape)
    got = W.bf16_bits_to_f32(out).astype(np.float64)
    ref = oracle.attend(w.q, w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale)[0]
    check(got, ref, "C client")
