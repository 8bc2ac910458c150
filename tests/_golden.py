"""Loader for the hand-derived closed-form cases in tests/golden/."""
import json
import math
import os

import numpy as np

from workloads import Workload, f32_to_bf16_bits

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "closed_forms.json")


def _bits(x):
    return f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


def cases():
    with open(GOLDEN) as f:
        doc = json.load(f)
    out = []
    for c in doc["cases"]:
        q = np.asarray(c["q"], dtype=np.float32)
        b, hq, d = q.shape
        p, hkv, n = c["page_size"], c["num_kv_heads"], c["num_pages"]
        k = np.full((n, p, hkv, d), np.nan, dtype=np.float32)
        v = np.full((n, p, hkv, d), np.nan, dtype=np.float32)
        for pid, slots in c["pages"].items():
            k[int(pid), : len(slots)] = np.asarray(slots, dtype=np.float32)
        for pid, slots in c["v_pages"].items():
            v[int(pid), : len(slots)] = np.asarray(slots, dtype=np.float32)
        kb = _bits(np.nan_to_num(k))
        vb = _bits(np.nan_to_num(v))
        kb[np.isnan(k)] = 0x7FC0
        vb[np.isnan(v)] = 0x7FC0
        w = Workload(q=_bits(q), k_cache=kb, v_cache=vb,
                     block_table=np.asarray(c["block_table"], dtype=np.int32),
                     context_lens=np.asarray(c["context_lens"], dtype=np.int32),
                     scale=np.float32(c["scale"]), name=c["name"])
        env = {"e": math.e, "__builtins__": {}}
        expected = np.array([[[eval(x, env) for x in row] for row in head] for head in c["expected"]],
                            dtype=np.float64)
        out.append((c["name"], w, expected))
    return out
