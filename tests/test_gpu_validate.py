"""The host-side validation of page tables and lengths (debugging aid)."""
import os
import subprocess
import sys

import numpy as np
import pytest

import workloads as W
from _gpu import to_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib(gpu_lib):
    return gpu_lib


def test_validate_accepts_a_good_table_and_names_the_first_bad_entry(lib):
    import torch
    w = W.build([40, 0, 17], 8, 2, 64, 16, seed=90)
    dev = to_gpu(w)
    lib.validate_paging(dev["bt"], dev["lens"], w.num_pages, 16)
    bad = dev["bt"].clone()
    bad[2, 1] = w.num_pages               # sequence 2 uses pages 0 and 1
    with pytest.raises(lib.PdaError, match=r"block_table\[2\]\[1\]"):
        lib.validate_paging(bad, dev["lens"], w.num_pages, 16)
    bad_lens = dev["lens"].clone()
    bad_lens[0] = w.max_pages * 16 + 1
    with pytest.raises(lib.PdaError, match=r"context_lens\[0\]"):
        lib.validate_paging(dev["bt"], bad_lens, w.num_pages, 16)
    # entries past a sequence's pages are not looked at
    unused = dev["bt"].clone()
    unused[1, :] = -7
    lib.validate_paging(unused, dev["lens"], w.num_pages, 16)
    torch.cuda.synchronize()


def test_debug_validate_env_rejects_a_bad_call():
    code = (
        "import sys, torch, numpy as np\n"
        "sys.path.insert(0, '.'); sys.path.insert(0, 'tests')\n"
        "import workloads as W\n"
        "from _gpu import to_gpu\n"
        "from paper_2606_07665_amd import binding as B\n"
        "w = W.build([40, 17], 8, 2, 64, 16, seed=91)\n"
        "d = to_gpu(w)\n"
        "out = torch.empty((2, 8, 64), dtype=torch.bfloat16, device='cuda')\n"
        "B.paged_decode_attention(d['q'], d['k'], d['v'], d['bt'], d['lens'], out, 0.125)\n"
        "d['bt'][0, 1] = -3\n"
        "try:\n"
        "    B.paged_decode_attention(d['q'], d['k'], d['v'], d['bt'], d['lens'], out, 0.125)\n"
        "    print('NO ERROR')\n"
        "except B.PdaError as e:\n"
        "    print('REJECTED', e)\n"
    )
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    env = dict(os.environ, PDA_DEBUG_VALIDATE="1")
    r = subprocess.run([sys.executable, "-c", code], cwd=root, env=env, capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    assert "REJECTED" in r.stdout and "block_table[0][1]" in r.stdout, r.stdout
