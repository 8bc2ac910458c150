"""ctypes binding of libpda.so (argument marshalling only).

Every step of paged decode attention runs in the HIP kernels of the library;
this module only checks tensor metadata, extracts device pointers and sizes
and forwards them, with torch's current HIP stream, to the C ABI declared in
include/pda.h.  There is no fallback: if the library cannot be loaded, every
call raises.
"""
from __future__ import annotations

import ctypes
import functools
import os
import re
from typing import Optional, Tuple

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "_lib", "libpda.so")
HEADER = os.path.join(os.path.dirname(_PKG), "include", "pda.h")

PDA_OK = 0
ERRORS = {1: "PDA_ERR_NULL", 2: "PDA_ERR_SHAPE", 3: "PDA_ERR_UNSUPPORTED", 4: "PDA_ERR_SCALE",
          5: "PDA_ERR_ALIGN", 6: "PDA_ERR_HIP", 7: "PDA_ERR_DTYPE", 8: "PDA_ERR_LAYOUT"}

_lib: Optional[ctypes.CDLL] = None


class PdaError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


class PreludeDims(ctypes.Structure):
    """pda_prelude_dims of include/pda.h."""
    _fields_ = [("batch", ctypes.c_int32), ("hidden", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("rotary_dim", ctypes.c_int32),
                ("interleaved", ctypes.c_int32), ("rope_theta", ctypes.c_float), ("eps", ctypes.c_float)]


DTYPE_BF16, DTYPE_F16, DTYPE_F32, DTYPE_I32, DTYPE_I64 = range(5)  # pda_dtype
MAX_DIMS = 4


class Tensor(ctypes.Structure):
    """pda_tensor of include/pda.h: device pointer, dtype, rank, extents and
    strides in elements."""
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("shape", ctypes.c_int64 * MAX_DIMS), ("stride", ctypes.c_int64 * MAX_DIMS)]


def tensor_desc(data_ptr, dtype: int, shape, stride=None) -> Tensor:
    """A descriptor from a raw pointer; ``stride`` defaults to dense row-major."""
    shape = [int(x) for x in shape]
    if stride is None:
        stride, acc = [], 1
        for n in reversed(shape):
            stride.insert(0, acc)
            acc *= n
    t = Tensor()
    t.data = data_ptr
    t.dtype = int(dtype)
    t.ndim = len(shape)
    for i, (n, st) in enumerate(zip(shape, stride)):
        t.shape[i] = n
        t.stride[i] = int(st)
    return t


def describe(t) -> Tensor:
    """The descriptor of a torch tensor as it is (dtype, shape and strides
    unchanged; the library decides whether it can read them)."""
    import torch
    codes = {torch.bfloat16: DTYPE_BF16, torch.float16: DTYPE_F16, torch.float32: DTYPE_F32,
             torch.int32: DTYPE_I32, torch.int64: DTYPE_I64}
    if t.dtype not in codes:
        raise TypeError(f"no pda_dtype for {t.dtype}")
    if t.dim() > MAX_DIMS:
        raise ValueError(f"a descriptor holds at most {MAX_DIMS} dimensions")
    return tensor_desc(t.data_ptr(), codes[t.dtype], t.shape, t.stride())


def _declare(lib: ctypes.CDLL) -> None:
    i32, i64, f32, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p
    lib.paged_decode_attention.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, f32, vp]
    lib.paged_decode_attention.restype = ctypes.c_int
    lib.paged_decode_attention_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, f32,
                                                   vp]
    lib.paged_decode_attention_noalloc.restype = ctypes.c_int
    tp = ctypes.POINTER(Tensor)
    lib.paged_decode_attention_desc.argtypes = [tp] * 6 + [f32, vp]
    lib.paged_decode_attention_desc.restype = ctypes.c_int
    lib.paged_decode_attention_ext.argtypes = [vp] * 6 + [i32] * 9 + [f32, vp]
    lib.paged_decode_attention_ext.restype = ctypes.c_int
    dims_p = ctypes.POINTER(PreludeDims)
    lib.pda_pack_weights.argtypes = [vp, vp, i32, i32, vp]
    lib.pda_pack_weights.restype = ctypes.c_int
    lib.pda_attention_prelude.argtypes = [vp] * 9 + [dims_p, vp]
    lib.pda_attention_prelude.restype = ctypes.c_int
    lib.pda_attention_prelude_append.argtypes = [vp] * 10 + [i32, i32, i32, dims_p, vp]
    lib.pda_attention_prelude_append.restype = ctypes.c_int
    lib.pda_prelude_workspace_reserve.argtypes = [dims_p, vp]
    lib.pda_prelude_workspace_reserve.restype = ctypes.c_int
    lib.pda_o_proj_residual_norm.argtypes = [vp] * 6 + [i32, i32, i32, f32, vp]
    lib.pda_o_proj_residual_norm.restype = ctypes.c_int
    lib.pda_o_proj_workspace_reserve.argtypes = [i32, i32, i32, vp]
    lib.pda_o_proj_workspace_reserve.restype = ctypes.c_int
    lib.pda_kv_append.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, vp]
    lib.pda_kv_append_n.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, vp]
    lib.pda_kv_append_n.restype = ctypes.c_int
    lib.pda_validate_paging.argtypes = [vp, vp, i32, i32, i32, i32, vp]
    lib.pda_validate_paging.restype = ctypes.c_int
    lib.pda_kv_append.restype = ctypes.c_int
    lib.paged_decode_attention_append.argtypes = [vp] * 8 + [i32] * 7 + [f32, vp]
    lib.paged_decode_attention_append.restype = ctypes.c_int
    lib.pda_plan.argtypes = [i32, i32, i32, i32, i32, i32, i32, ctypes.POINTER(i32), ctypes.POINTER(i32),
                             ctypes.POINTER(i64)]
    lib.pda_plan.restype = ctypes.c_int
    lib.pda_workspace_reserve.argtypes = [i32, i32, i32, i32, i32, i32, vp]
    lib.pda_workspace_reserve.restype = ctypes.c_int
    lib.pda_release_workspaces.argtypes = []
    lib.pda_release_workspaces.restype = ctypes.c_int
    lib.pda_last_error.argtypes = []
    lib.pda_last_error.restype = ctypes.c_char_p
    lib.pda_version.argtypes = []
    lib.pda_version.restype = i32
    lib.pda_set_option.argtypes = [i32, i32]
    lib.pda_set_option.restype = ctypes.c_int
    lib.pda_get_option.argtypes = [i32]
    lib.pda_get_option.restype = i32
    lib.pda_profile_enable.argtypes = [i32]
    lib.pda_profile_enable.restype = ctypes.c_int
    lib.pda_profile_read.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                     ctypes.POINTER(i64)]
    lib.pda_profile_read.restype = ctypes.c_int
    lib.pda_profile_read_prelude.argtypes = lib.pda_profile_read.argtypes
    lib.pda_profile_read_prelude.restype = ctypes.c_int
    lib.pda_profile_read_o_proj.argtypes = lib.pda_profile_read.argtypes
    lib.pda_profile_read_o_proj.restype = ctypes.c_int
    lib.pda_stream_read.argtypes = [vp, i64, vp, i32, i32, vp]
    lib.pda_stream_read.restype = ctypes.c_int


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the built library (raises if it is missing: build it first with
    ``python -m paper_2606_07665_amd.build``)."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise RuntimeError(f"HIP library not built: {path} is missing "
                               "(run python -m paper_2606_07665_amd.build)")
        lib = ctypes.CDLL(path)
        _declare(lib)
        _lib = lib
    return _lib


def declared_symbols(header: str = HEADER):
    """Function names declared in include/pda.h."""
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[A-Za-z_][\w\s\*]*?\b([a-z_][a-z0-9_]*)\s*\(", text, flags=re.M)))


def _check(rc: int) -> None:
    if rc != PDA_OK:
        raise PdaError(rc, load().pda_last_error().decode())


def last_error() -> str:
    return load().pda_last_error().decode()


def version() -> int:
    return int(load().pda_version())


def raw_call(q_ptr, k_ptr, v_ptr, bt_ptr, lens_ptr, out_ptr, batch, hq, hkv, d, page_size, num_pages,
             max_pages, scale, stream_ptr=None) -> int:
    """Direct C call with integer pointers; returns the status code."""
    return load().paged_decode_attention(q_ptr, k_ptr, v_ptr, bt_ptr, lens_ptr, out_ptr, batch, hq, hkv, d,
                                         page_size, num_pages, max_pages, ctypes.c_float(scale), stream_ptr)


def _stream_ptr(stream, device=None):
    """The HIP stream handle of ``stream``, or of torch's current stream on
    ``device`` (default: the current device)."""
    import torch
    if stream is None:
        # the raw handle without building a Stream object (~3 us a call)
        return ctypes.c_void_p(torch._C._cuda_getCurrentRawStream(
            torch.cuda.current_device() if device is None else device))
    return ctypes.c_void_p(stream.cuda_stream)


@functools.lru_cache(maxsize=None)
def _parsed_dims(dims):
    """dims string -> tuple of (kind, value): 0 any, 1 number, 2 symbol."""
    out = []
    for sym in dims.split():
        if sym == "*":
            out.append((0, None))
        elif sym.isdigit():
            out.append((1, int(sym)))
        else:
            out.append((2, sym))
    return tuple(out)


def _validate(specs, known=None):
    """Argument checks of a wrapper, before any launch.  ``specs``: (name,
    tensor or None, torch dtype, dims) with dims a space-separated list of
    extents -- a number, ``*`` (any), or a symbol bound by the first tensor
    that has it (or by ``known``) and checked on every other.  All shapes are
    checked first, then dtypes, then that every tensor is on one GPU, then
    contiguity, so a bad argument raises whichever it is.  Returns the
    bound sizes.  The usual case (every check passes) reads each property of
    a tensor once; any failure reruns the checks in that order to raise."""
    sizes = dict(known or {})
    dev = None
    ok = True
    for _, t, dt, dims in specs:
        if t is None:
            continue
        shape = t.shape
        pd = _parsed_dims(dims)
        if len(shape) != len(pd):
            ok = False
            break
        for (kind, val), ext in zip(pd, shape):
            if kind == 1:
                if ext != val:
                    ok = False
            elif kind == 2:
                want = sizes.get(val)
                if want is None:
                    sizes[val] = int(ext)
                elif ext != want:
                    ok = False
        d = t.get_device()
        if dev is None:
            dev = d
        if not ok or t.dtype != dt or d < 0 or d != dev or not t.is_contiguous():
            ok = False
            break
    if ok:
        return sizes
    return _validate_raise(specs, known)


def _validate_raise(specs, known=None):
    """The checks of _validate one kind at a time, raising the first failure."""
    sizes = dict(known or {})
    present = [sp for sp in specs if sp[1] is not None]
    for name, t, _, dims in present:
        syms = dims.split()
        if t.dim() != len(syms):
            raise ValueError(f"{name} must be [{', '.join(syms)}], got shape {tuple(t.shape)}")
        for sym, ext in zip(syms, t.shape):
            if sym == "*":
                continue
            if sym.isdigit():
                want = int(sym)
            elif sym in sizes:
                want = sizes[sym]
            else:
                sizes[sym] = int(ext)
                continue
            if int(ext) != want:
                raise ValueError(f"{name} must be [{', '.join(syms)}] with {sym} = {want}, got shape {tuple(t.shape)}")
    for name, t, dt, _ in present:
        if t.dtype != dt:
            raise TypeError(f"{name} must be {dt}, got {t.dtype}")
    for name, t, _, _ in present:
        if not t.is_cuda:
            raise ValueError(f"{name} must be a GPU tensor")
    if len({t.device for _, t, _, _ in present}) > 1:
        raise ValueError("all tensors must be on one GPU")
    for name, t, _, _ in present:
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    return sizes


def _cache_specs(k_cache, v_cache, block_table, context_lens):
    import torch
    return [("k_cache", k_cache, torch.bfloat16, "N P Hkv D"), ("v_cache", v_cache, torch.bfloat16, "N P Hkv D"),
            ("block_table", block_table, torch.int32, "B M"), ("context_lens", context_lens, torch.int32, "B")]


def _check_attention_args(q, k_cache, v_cache, block_table, context_lens, out):
    """Checks of a one-query attention call; returns (B, Hq, D, num_pages,
    page_size, Hkv, device).  The usual case (every check passes) reads each
    property once; otherwise _validate runs the full checks and raises the
    specific error."""
    import torch
    bf, i32 = torch.bfloat16, torch.int32
    qs, ks = q.shape, k_cache.shape
    if (len(qs) == 3 and len(ks) == 4 and out.shape == qs and v_cache.shape == ks and ks[3] == qs[2]
            and block_table.dim() == 2 and block_table.shape[0] == qs[0] and context_lens.shape == (qs[0],)
            and q.dtype is bf and out.dtype is bf and k_cache.dtype is bf and v_cache.dtype is bf
            and block_table.dtype is i32 and context_lens.dtype is i32):
        dev = q.get_device()
        if (dev >= 0 and out.get_device() == dev and k_cache.get_device() == dev and v_cache.get_device() == dev
                and block_table.get_device() == dev and context_lens.get_device() == dev
                and q.is_contiguous() and out.is_contiguous() and k_cache.is_contiguous()
                and v_cache.is_contiguous() and block_table.is_contiguous() and context_lens.is_contiguous()):
            return qs[0], qs[1], qs[2], ks[0], ks[1], ks[2], dev
    sz = _validate([("q", q, torch.bfloat16, "B Hq D"), *_cache_specs(k_cache, v_cache, block_table, context_lens),
                    ("out", out, torch.bfloat16, "B Hq D")])
    return sz["B"], sz["Hq"], sz["D"], sz["N"], sz["P"], sz["Hkv"], q.get_device()


def paged_decode_attention(q, k_cache, v_cache, block_table, context_lens, out, scale, stream=None):
    """out[b, h] = softmax(scale * q[b, h] . K_b^T) V_b over the paged cache.

    q, out: bf16 [B, Hq, D]; k_cache, v_cache: bf16 [N, P, Hkv, D];
    block_table: int32 [B, maxp]; context_lens: int32 [B]; all contiguous on
    one GPU.  Launches on ``stream`` (default: torch's current stream).
    """
    b, hq, d, n, p, hkv, dev = _check_attention_args(q, k_cache, v_cache, block_table, context_lens, out)
    _check(raw_call(q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), block_table.data_ptr(),
                    context_lens.data_ptr(), out.data_ptr(), b, hq, hkv, d, p, n, block_table.shape[1],
                    float(scale), _stream_ptr(stream, dev)))
    return out


def paged_decode_attention_noalloc(q, k_cache, v_cache, block_table, context_lens, out, scale, stream=None):
    """:func:`paged_decode_attention` through the entry point that allocates
    nothing: its partials go to the library's fixed per-device scratch
    (NOALLOC_SCRATCH_BYTES).  Calls on one device must not overlap in time."""
    b, hq, d, n, p, hkv, dev = _check_attention_args(q, k_cache, v_cache, block_table, context_lens, out)
    _check(load().paged_decode_attention_noalloc(
        q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), block_table.data_ptr(), context_lens.data_ptr(),
        out.data_ptr(), b, hq, hkv, d, p, n, block_table.shape[1], ctypes.c_float(float(scale)),
        _stream_ptr(stream, dev)))
    return out


NOALLOC_SCRATCH_BYTES = 64 * 1024 * 1024  # PDA_NOALLOC_SCRATCH_BYTES of include/pda.h


def desc_call(q, k_cache, v_cache, block_table, context_lens, out, scale, stream_ptr=None) -> int:
    """paged_decode_attention_desc on six descriptors (Tensor or None);
    returns the status code."""
    ref = [None if t is None else ctypes.byref(t) for t in (q, k_cache, v_cache, block_table, context_lens, out)]
    return load().paged_decode_attention_desc(*ref, ctypes.c_float(scale), stream_ptr)


def paged_decode_attention_desc(q, k_cache, v_cache, block_table, context_lens, out, scale, stream=None):
    """:func:`paged_decode_attention` through the descriptor entry point:
    the tensors are passed as they are (dtype, shape, strides) and the
    library checks them (PDA_ERR_DTYPE, PDA_ERR_SHAPE, PDA_ERR_LAYOUT)."""
    _check(desc_call(*(describe(t) for t in (q, k_cache, v_cache, block_table, context_lens, out)), float(scale),
                     _stream_ptr(stream)))
    return out


def paged_decode_attention_ext(q, k_cache, v_cache, block_table, context_lens, out, scale, window=0,
                               stream=None):
    """Several causal query tokens per sequence and an optional sliding window.

    q, out: bf16 [B, Tq, Hq, D] (the sequence's last Tq tokens; query j sits
    at position L - Tq + j and sees keys up to it); ``window`` 0 = none, W > 0
    = the last W keys up to the query's position.  Other arguments as for
    :func:`paged_decode_attention`.
    """
    import torch
    sz = _validate([("q", q, torch.bfloat16, "B T Hq D"), *_cache_specs(k_cache, v_cache, block_table, context_lens),
                    ("out", out, torch.bfloat16, "B T Hq D")])
    _check(load().paged_decode_attention_ext(
        q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), block_table.data_ptr(), context_lens.data_ptr(),
        out.data_ptr(), sz["B"], sz["Hq"], sz["Hkv"], sz["D"], sz["P"], sz["N"], sz["M"], sz["T"], int(window),
        ctypes.c_float(float(scale)), _stream_ptr(stream)))
    return out


def kv_append(k_new, v_new, k_cache, v_cache, block_table, context_lens, stream=None):
    """Scatter each sequence's new key/value ([B, Hkv, D] bf16) into its page
    slot at position context_lens[b] - 1 (the length counts the new token)."""
    import torch
    sz = _validate([("k_new", k_new, torch.bfloat16, "B Hkv D"), ("v_new", v_new, torch.bfloat16, "B Hkv D"),
                    *_cache_specs(k_cache, v_cache, block_table, context_lens)])
    _check(load().pda_kv_append(k_new.data_ptr(), v_new.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(),
                                block_table.data_ptr(), context_lens.data_ptr(), sz["B"], sz["Hkv"], sz["D"], sz["P"],
                                sz["N"], sz["M"], _stream_ptr(stream)))


def kv_append_n(k_new, v_new, k_cache, v_cache, block_table, context_lens, stream=None):
    """Scatter T new tokens per sequence ([B, T, Hkv, D] bf16) to positions
    context_lens[b] - T + j (the lengths count all of them)."""
    import torch
    sz = _validate([("k_new", k_new, torch.bfloat16, "B T Hkv D"), ("v_new", v_new, torch.bfloat16, "B T Hkv D"),
                    *_cache_specs(k_cache, v_cache, block_table, context_lens)])
    _check(load().pda_kv_append_n(k_new.data_ptr(), v_new.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(),
                                  block_table.data_ptr(), context_lens.data_ptr(), sz["B"], sz["T"], sz["Hkv"],
                                  sz["D"], sz["P"], sz["N"], sz["M"], _stream_ptr(stream)))


def paged_decode_attention_append(q, k_new, v_new, k_cache, v_cache, block_table, context_lens, out, scale,
                                  stream=None):
    """kv_append then paged_decode_attention on the same stream."""
    import torch
    sz = _validate([("q", q, torch.bfloat16, "B Hq D"), ("k_new", k_new, torch.bfloat16, "B Hkv D"),
                    ("v_new", v_new, torch.bfloat16, "B Hkv D"),
                    *_cache_specs(k_cache, v_cache, block_table, context_lens),
                    ("out", out, torch.bfloat16, "B Hq D")])
    _check(load().paged_decode_attention_append(
        q.data_ptr(), k_new.data_ptr(), v_new.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(),
        block_table.data_ptr(), context_lens.data_ptr(), out.data_ptr(), sz["B"], sz["Hq"], sz["Hkv"], sz["D"],
        sz["P"], sz["N"], sz["M"], ctypes.c_float(float(scale)), _stream_ptr(stream)))
    return out


def _ptr(t):
    return None if t is None else t.data_ptr()


def pack_weights(w, stream=None):
    """Pack a bf16 [rows, cols] weight into the prelude's tile order; returns
    a new tensor of the same shape holding the packed data."""
    import torch
    _validate([("w", w, torch.bfloat16, "R C")])
    out = torch.empty_like(w)
    _check(load().pda_pack_weights(w.data_ptr(), out.data_ptr(), w.shape[0], w.shape[1], _stream_ptr(stream)))
    return out


def prelude_dims(batch, hidden, hq, hkv, d, rotary_dim, interleaved, theta, eps) -> PreludeDims:
    return PreludeDims(int(batch), int(hidden), int(hq), int(hkv), int(d), int(rotary_dim), int(bool(interleaved)),
                       float(theta), float(eps))


def _prelude_specs(x, w_packed, context_lens, q_out, bias, q_norm, k_norm):
    import torch
    if (q_norm is None) != (k_norm is None):
        raise ValueError("q_norm and k_norm must both be given or both be None")
    bf = torch.bfloat16
    return [("x", x, bf, "B H"), ("w_packed", w_packed, bf, "N H"), ("context_lens", context_lens, torch.int32, "B"),
            ("q_out", q_out, bf, "B Hq D"), ("bias", bias, bf, "N"), ("q_norm", q_norm, bf, "D"),
            ("k_norm", k_norm, bf, "D")]


def attention_prelude(x, w_packed, context_lens, q_out, k_out, v_out, *, num_q_heads, num_kv_heads, head_dim,
                      rope_theta, rotary_dim=None, interleaved=False, bias=None, q_norm=None, k_norm=None,
                      eps=1e-6, stream=None):
    """QKV projection + optional per-head Q/K RMSNorm + RoPE of this step's
    token (x: bf16 [B, H]; w_packed [(Hq + 2 Hkv) D, H] from
    :func:`pack_weights`; context_lens int32 [B]; q_out [B, Hq, D]; k_out,
    v_out [B, Hkv, D]; bias [(Hq + 2 Hkv) D]; q_norm, k_norm [D])."""
    import torch
    known = dict(Hq=int(num_q_heads), Hkv=int(num_kv_heads), D=int(head_dim),
                 N=(int(num_q_heads) + 2 * int(num_kv_heads)) * int(head_dim))
    sz = _validate(_prelude_specs(x, w_packed, context_lens, q_out, bias, q_norm, k_norm) +
                   [("k_out", k_out, torch.bfloat16, "B Hkv D"), ("v_out", v_out, torch.bfloat16, "B Hkv D")],
                   known)
    dims = prelude_dims(sz["B"], sz["H"], num_q_heads, num_kv_heads, head_dim,
                        head_dim if rotary_dim is None else rotary_dim, interleaved, rope_theta, eps)
    _check(load().pda_attention_prelude(x.data_ptr(), w_packed.data_ptr(), _ptr(bias), _ptr(q_norm), _ptr(k_norm),
                                        context_lens.data_ptr(), q_out.data_ptr(), k_out.data_ptr(),
                                        v_out.data_ptr(), ctypes.byref(dims), _stream_ptr(stream)))


def attention_prelude_append(x, w_packed, context_lens, q_out, k_cache, v_cache, block_table, *, num_q_heads,
                             num_kv_heads, head_dim, rope_theta, rotary_dim=None, interleaved=False, bias=None,
                             q_norm=None, k_norm=None, eps=1e-6, stream=None):
    """The prelude with the KV append fused in: k, v go straight to their
    page slot at position context_lens[b] - 1 (caches [N, P, Hkv, D],
    block_table int32 [B, maxp]; other arguments as for
    :func:`attention_prelude`)."""
    import torch
    known = dict(Hq=int(num_q_heads), Hkv=int(num_kv_heads), D=int(head_dim),
                 N=(int(num_q_heads) + 2 * int(num_kv_heads)) * int(head_dim))
    sz = _validate(_prelude_specs(x, w_packed, context_lens, q_out, bias, q_norm, k_norm) +
                   [("k_cache", k_cache, torch.bfloat16, "Np P Hkv D"), ("v_cache", v_cache, torch.bfloat16, "Np P Hkv D"),
                    ("block_table", block_table, torch.int32, "B M")], known)
    dims = prelude_dims(sz["B"], sz["H"], num_q_heads, num_kv_heads, head_dim,
                        head_dim if rotary_dim is None else rotary_dim, interleaved, rope_theta, eps)
    _check(load().pda_attention_prelude_append(
        x.data_ptr(), w_packed.data_ptr(), _ptr(bias), _ptr(q_norm), _ptr(k_norm), context_lens.data_ptr(),
        q_out.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), block_table.data_ptr(), sz["P"], sz["Np"],
        sz["M"], ctypes.byref(dims), _stream_ptr(stream)))


def prelude_workspace_reserve(dims: PreludeDims, stream=None) -> None:
    _check(load().pda_prelude_workspace_reserve(ctypes.byref(dims), _stream_ptr(stream)))


def plan(batch, hq, hkv, d, page_size, max_pages, num_cus=256) -> Tuple[int, int, int]:
    """(grid blocks, waves, workspace bytes) the split planner picks."""
    g, w, ws = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int64()
    _check(load().pda_plan(batch, hq, hkv, d, page_size, max_pages, num_cus,
                           ctypes.byref(g), ctypes.byref(w), ctypes.byref(ws)))
    return g.value, w.value, ws.value


def workspace_reserve(batch, hq, hkv, d, page_size, max_pages, stream=None) -> None:
    _check(load().pda_workspace_reserve(batch, hq, hkv, d, page_size, max_pages, _stream_ptr(stream)))


def release_workspaces() -> None:
    _check(load().pda_release_workspaces())


OPT_BLOCKS_PER_CU = 1
OPT_MIN_STEPS = 2     # fewest 32-token steps per wave (0 = the planner's choice, the default)
OPT_COMPUTE_PATH = 3  # 0 = matrix cores (default), 1 = vector ALU (the measured alternative)
OPT_FUSED_MERGE = 4   # 0 = merge kernel (default), 1 = fused merge for small plans, 2 = every multi-workgroup plan
OPT_KV_GROUP = 5      # most kv heads per attention workgroup (0 = the planner's choice)
OPT_FIXED_SPLIT = 6   # 1 = fixed split for latency-bound calls (default), 0 = stream-K for every call


def set_option(option: int, value: int) -> None:
    _check(load().pda_set_option(option, value))


def get_option(option: int) -> int:
    return int(load().pda_get_option(option))


def stream_read(buf, sink, unroll: int = 0, blocks_per_cu: int = 0, stream=None) -> None:
    """The streaming-read reference kernel over a whole contiguous GPU tensor
    (any dtype, 16-byte aligned, a multiple of 16 bytes); sink: an int32 GPU
    tensor of at least one element."""
    import torch
    if not buf.is_cuda or not buf.is_contiguous() or not sink.is_cuda or sink.dtype != torch.int32:
        raise ValueError("buf must be a contiguous GPU tensor and sink an int32 GPU tensor")
    _check(load().pda_stream_read(buf.data_ptr(), buf.numel() * buf.element_size(), sink.data_ptr(), unroll,
                                  blocks_per_cu, _stream_ptr(stream)))


def profile_enable(on: bool = True) -> None:
    _check(load().pda_profile_enable(1 if on else 0))


def profile_read() -> Tuple[float, float, int]:
    """(split kernel ms, merge kernel ms, calls) summed since the last read."""
    s, m, n = ctypes.c_double(), ctypes.c_double(), ctypes.c_int64()
    _check(load().pda_profile_read(ctypes.byref(s), ctypes.byref(m), ctypes.byref(n)))
    return s.value, m.value, n.value


def profile_read_prelude() -> Tuple[float, float, int]:
    """(GEMV kernel ms, epilogue kernel ms, prelude calls) summed since the last read."""
    s, m, n = ctypes.c_double(), ctypes.c_double(), ctypes.c_int64()
    _check(load().pda_profile_read_prelude(ctypes.byref(s), ctypes.byref(m), ctypes.byref(n)))
    return s.value, m.value, n.value



def o_proj_residual_norm(attn, w_packed, residual, norm_w, residual_out, normed_out, eps=1e-5, stream=None):
    """z = W_o attn + residual -> residual_out (bf16); RMSNorm(z) * norm_w ->
    normed_out.  attn [B, K], w_packed [H, K] from :func:`pack_weights`,
    residual / outputs [B, H], norm_w [H]; residual_out may be residual."""
    import torch
    bf = torch.bfloat16
    sz = _validate([("attn", attn, bf, "B K"), ("w_packed", w_packed, bf, "H K"), ("residual", residual, bf, "B H"),
                    ("norm_w", norm_w, bf, "H"), ("residual_out", residual_out, bf, "B H"),
                    ("normed_out", normed_out, bf, "B H")])
    _check(load().pda_o_proj_residual_norm(attn.data_ptr(), w_packed.data_ptr(), residual.data_ptr(),
                                           norm_w.data_ptr(), residual_out.data_ptr(), normed_out.data_ptr(), sz["B"],
                                           sz["K"], sz["H"], ctypes.c_float(float(eps)), _stream_ptr(stream)))


def o_proj_workspace_reserve(batch, in_features, hidden, stream=None) -> None:
    _check(load().pda_o_proj_workspace_reserve(batch, in_features, hidden, _stream_ptr(stream)))


def profile_read_o_proj() -> Tuple[float, float, int]:
    """(GEMV kernel ms, epilogue kernel ms, o_proj calls) summed since the last read."""
    s, m, n = ctypes.c_double(), ctypes.c_double(), ctypes.c_int64()
    _check(load().pda_profile_read_o_proj(ctypes.byref(s), ctypes.byref(m), ctypes.byref(n)))
    return s.value, m.value, n.value



def validate_paging(block_table, context_lens, num_pages, page_size, stream=None) -> None:
    """Check the device page table and lengths on the host (synchronises);
    raises PdaError naming the first bad entry."""
    import torch
    _validate([("block_table", block_table, torch.int32, "B M"), ("context_lens", context_lens, torch.int32, "B")])
    _check(load().pda_validate_paging(block_table.data_ptr(), context_lens.data_ptr(), block_table.shape[0],
                                      block_table.shape[1], page_size, num_pages, _stream_ptr(stream)))
