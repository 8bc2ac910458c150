"""Helpers for GPU tests: move a workload to the device, run the library,
compare with the oracle."""
import sys

import numpy as np

MAX_ABS = 1e-2   # required tolerance vs the fp64 oracle (absolute, on bf16 outputs)
MEAN_ABS = 1e-3


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_gpu(w, device="cuda"):
    import torch

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(device)

    return dict(q=bf(w.q), k=bf(w.k_cache), v=bf(w.v_cache),
                bt=torch.from_numpy(np.ascontiguousarray(w.block_table)).to(device),
                lens=torch.from_numpy(np.ascontiguousarray(w.context_lens)).to(device))


def run(lib, w, dev=None, out=None, stream=None, fill=float("nan")):
    """Run the library on workload w; returns out as float64 numpy [B, Hq, D]."""
    import torch
    if dev is None:
        dev = to_gpu(w)
    if out is None:
        out = torch.full(tuple(w.q.shape), fill, dtype=torch.bfloat16, device=dev["q"].device)
    lib.paged_decode_attention(dev["q"], dev["k"], dev["v"], dev["bt"], dev["lens"], out, float(w.scale),
                               stream=stream)
    torch.cuda.synchronize()
    return out.float().cpu().numpy().astype(np.float64)


def q4(w):
    """q of a workload as [B, Tq, Hq, D]."""
    return w.q if w.q.ndim == 4 else w.q[:, None]


def run_ext(lib, w, dev=None, stream=None):
    """paged_decode_attention_ext on workload w (its query tokens and
    window); returns out as float64 numpy [B, Tq, Hq, D]."""
    import torch
    if dev is None:
        dev = to_gpu(w)
    q = dev["q"] if dev["q"].dim() == 4 else dev["q"].unsqueeze(1)
    out = torch.full(tuple(q.shape), float("nan"), dtype=torch.bfloat16, device="cuda")
    lib.paged_decode_attention_ext(q.contiguous(), dev["k"], dev["v"], dev["bt"], dev["lens"], out,
                                   float(w.scale), window=w.window, stream=stream)
    torch.cuda.synchronize()
    return out.float().cpu().numpy().astype(np.float64)


def bf16_round(x):
    import workloads as W
    return W.bf16_bits_to_f32(W.f32_to_bf16_bits(np.asarray(x, dtype=np.float32))).astype(np.float64)


def bf16_ulps(got, ref, floor=2.0 ** -6):
    """|got - ref| in bf16 spacings at max(|ref|, floor)."""
    ulp = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(ref), floor))) - 7)
    return np.abs(got - ref) / ulp


def check(got, ref, what="", max_ulps=1.0):
    """Required tolerance (max 1e-2, mean 1e-3 absolute), and the stronger
    property this path has: every bf16 output is within one bf16 spacing of
    the fp64 value (the only rounding left is the output's own)."""
    err = np.abs(got - ref)
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    mx, mean = float(err.max()) if err.size else 0.0, float(err.mean()) if err.size else 0.0
    ulps = float(bf16_ulps(got, ref).max()) if err.size else 0.0
    log(f"  {what}: max|err|={mx:.3e} mean|err|={mean:.3e} max={ulps:.2f} bf16 ulp (n={err.size})")
    assert mx <= MAX_ABS and mean <= MEAN_ABS, f"{what}: max {mx:.3e} mean {mean:.3e}"
    if max_ulps is not None:
        assert ulps <= max_ulps, f"{what}: {ulps:.2f} bf16 ulps"
    return mx, mean


def check_full(name, run_fn, tmpdir, max_ulps=1.0):
    """Every output of the named workload against the fp64 oracle.

    The oracle runs in a fresh interpreter (tests/_oracle_job.py) fanned out
    over the host cores, started before this process builds the same seeded
    workload and runs `run_fn(w)` (which returns the GPU output as float64),
    so the two overlap.  Checks the required tolerance (max and mean over all
    outputs) and one bf16 spacing everywhere."""
    import _oracle_job
    import workloads as W
    job = _oracle_job.start(name, str(tmpdir))
    try:
        log(f"workload {name}: generating")
        w = W.make(name)
        log(f"workload {name}: running")
        got = run_fn(w)
        del w
        log(f"workload {name}: waiting for the oracle over every output")
        r = job.result().reshape(got.shape)
    finally:
        if job.proc.poll() is None:
            job.proc.kill()
            job.proc.wait()
    check(got, r, f"{name} (every output)", max_ulps)
    rb = bf16_round(r)
    log(f"  {name}: {100 * float((got == rb).mean()):.2f}% bitwise equal to RN(oracle)")
    return got, r
