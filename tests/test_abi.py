"""The C-ABI library on the CPU: it loads, exports every function its header
declares, and rejects bad arguments with the documented codes before making
any HIP call (none of these calls touches a device)."""
import ctypes
import re
import math

import pytest

from paper_2606_07665_amd import binding as B

OK, NULL, SHAPE, UNSUPPORTED, SCALE, ALIGN = 0, 1, 2, 3, 4, 5


@pytest.fixture(scope="module")
def lib():
    return B.load()


def test_exports_every_declared_symbol(lib):
    names = B.declared_symbols()
    assert {"paged_decode_attention", "pda_plan", "pda_workspace_reserve", "pda_last_error"} <= set(names)
    for n in names:
        assert hasattr(lib, n), f"{n} declared in include/pda.h but not exported"
    assert B.version() == 1


def call(ptr=16, batch=2, hq=32, hkv=8, d=128, p=16, n=64, maxp=8, scale=0.088, ptrs=None):
    ptrs = ptrs or [ptr] * 6
    return B.raw_call(*ptrs, batch, hq, hkv, d, p, n, maxp, scale)


@pytest.mark.parametrize("kwargs,code,text", [
    (dict(ptr=0), NULL, "NULL"),
    (dict(batch=-1), SHAPE, "batch"),
    (dict(hkv=7), SHAPE, "multiple"),
    (dict(hq=0), SHAPE, "positive"),
    (dict(hq=2048, hkv=2048), UNSUPPORTED, "num_kv_heads"),
    (dict(hq=64, hkv=2), UNSUPPORTED, "group"),
    (dict(d=96), UNSUPPORTED, "head_dim"),
    (dict(p=24), UNSUPPORTED, "page_size"),
    (dict(p=2048), UNSUPPORTED, "page_size"),
    (dict(p=0), SHAPE, "positive"),
    (dict(maxp=0), SHAPE, "positive"),
    (dict(batch=8193), UNSUPPORTED, "batch"),
    (dict(batch=4097, d=256), UNSUPPORTED, "head_dim 256"),
    (dict(d=512), UNSUPPORTED, "head_dim"),
    (dict(n=0), SHAPE, "num_pages"),
    (dict(scale=float("inf")), SCALE, "finite"),
    (dict(scale=float("nan")), SCALE, "finite"),
    (dict(ptrs=[16, 16, 24, 16, 16, 16]), ALIGN, "16-byte"),
    (dict(ptrs=[16, 16, 16, 18, 16, 16]), ALIGN, "4-byte"),
    (dict(maxp=1 << 27, p=16), SHAPE, "too large"),
])
def test_argument_errors(lib, kwargs, code, text):
    rc = call(**kwargs)
    assert rc == code, B.last_error()
    assert text in B.last_error()


def test_empty_batch_is_a_noop(lib):
    # batch 0 returns before any pointer is used or any HIP call is made
    assert call(ptr=0, batch=0) == OK
    assert B.last_error() == ""


def test_planner_fills_the_device_and_sizes_the_workspace(lib):
    # long context: one workgroup per CU, 8 waves each, workspace covers the slots
    g, w, ws = B.plan(4, 64, 8, 128, 16, 8192, num_cus=256)
    assert g == 256 and w == 256 * 8
    slots = g + 4 * 1  # one kv-head group of 8 per sequence
    assert ws >= slots * 8 * 8 * (128 + 2) * 4
    # tiny problem: fewer workgroups than CUs (each wave gets >= 2 steps)
    g, w, ws = B.plan(1, 8, 2, 64, 16, 16, num_cus=256)
    assert g == 1 and w == 8
    # kv-head group: largest divisor of Hkv <= 8, phases up to 8 waves
    g, w, _ = B.plan(3, 12, 3, 64, 16, 10, num_cus=256)
    assert w % 6 == 0
    g, w, _ = B.plan(2, 16, 16, 128, 16, 100, num_cus=256)
    assert w == 8 * g
    # head_dim 256: at most 4 waves per workgroup (one per SIMD), 4 kv heads
    # of a group read together, phases making up 4 waves when Hkv is smaller
    g, w, _ = B.plan(16, 12, 4, 256, 16, 2048, num_cus=256)
    assert g == 256 and w == 4 * g
    g, w, _ = B.plan(16, 16, 8, 256, 16, 2048, num_cus=256)
    assert w == 4 * g
    g, w, _ = B.plan(16, 8, 1, 256, 16, 2048, num_cus=256)
    assert w == 4 * g
    assert B.plan(4096, 12, 4, 256, 16, 4, num_cus=256)[0] >= 1
    with pytest.raises(B.PdaError):
        B.plan(1, 8, 3, 64, 16, 16)
    with pytest.raises(B.PdaError):
        B.plan(1, 8, 2, 64, 16, 16, num_cus=0)


def test_small_calls_take_one_step_per_wave(lib):
    """Planner's choice (min steps 0): a call whose K/V fit in 128 MB and
    whose two-step plan splits the work but leaves CUs idle gets one step
    per wave (twice the workgroups); a caller's fixed value is kept; large
    calls and single-workgroup calls are unchanged."""
    assert B.get_option(B.OPT_MIN_STEPS) == 0
    assert B.plan(1, 32, 8, 128, 16, 256, num_cus=256)[0] == 128   # 1 x 4096 tokens
    assert B.plan(4, 32, 8, 128, 16, 64, num_cus=256)[0] == 128    # 4 x 1024
    assert B.plan(4, 64, 8, 128, 16, 8192, num_cus=256)[0] == 256  # long70b
    assert B.plan(1, 8, 2, 64, 16, 16, num_cus=256)[0] == 1        # one workgroup: no merge
    try:
        B.set_option(B.OPT_MIN_STEPS, 2)
        assert B.plan(1, 32, 8, 128, 16, 256, num_cus=256)[0] == 64
    finally:
        B.set_option(B.OPT_MIN_STEPS, 0)


def test_fixed_split_option(lib):
    """Latency-bound calls take the fixed split by default: every
    (sequence, kv-head group) is cut into the same number of whole-step
    chunks (2 x 3000 tokens at D = 256: 2 sequences x 4 groups x 24 chunks
    of 4 steps = 192 workgroups, against 188 for the stream-K split over
    the same step count); large calls, and calls with more sequences than
    half the device's workgroups, keep the stream-K split."""
    assert B.get_option(B.OPT_FIXED_SPLIT) == 1
    assert B.plan(2, 16, 4, 256, 32, 94, num_cus=256)[0] == 192
    assert B.plan(4, 64, 8, 128, 16, 8192, num_cus=256)[0] == 256  # long70b: stream-K
    # a call the stream-K split gives one workgroup: one chunk per sequence,
    # whole sequences on separate workgroups (2 x 128 tokens, 8:2 heads)
    assert B.plan(2, 8, 2, 64, 16, 8, num_cus=256)[0] == 2
    try:
        B.set_option(B.OPT_FIXED_SPLIT, 0)
        assert B.get_option(B.OPT_FIXED_SPLIT) == 0
        assert B.plan(2, 16, 4, 256, 32, 94, num_cus=256)[0] == 188
        assert B.plan(2, 8, 2, 64, 16, 8, num_cus=256)[0] == 1
        with pytest.raises(B.PdaError):
            B.set_option(B.OPT_FIXED_SPLIT, 2)
        with pytest.raises(B.PdaError):
            B.set_option(B.OPT_FIXED_SPLIT, -1)
    finally:
        B.set_option(B.OPT_FIXED_SPLIT, 1)


def test_planner_grid_scales_with_options(lib):
    try:
        B.set_option(B.OPT_BLOCKS_PER_CU, 2)
        assert B.plan(4, 64, 8, 128, 16, 8192, num_cus=256)[0] == 512
        B.set_option(B.OPT_BLOCKS_PER_CU, 1)
        B.set_option(B.OPT_MIN_STEPS, 1 << 20)
        assert B.plan(4, 64, 8, 128, 16, 8192, num_cus=256)[0] == 1
    finally:
        B.set_option(B.OPT_BLOCKS_PER_CU, 1)
        B.set_option(B.OPT_MIN_STEPS, 0)
    assert B.get_option(B.OPT_MIN_STEPS) == 0
    with pytest.raises(B.PdaError):
        B.set_option(B.OPT_MIN_STEPS, -1)
    with pytest.raises(B.PdaError):
        B.set_option(B.OPT_BLOCKS_PER_CU, 0)
    with pytest.raises(B.PdaError):
        B.set_option(99, 1)
    assert B.get_option(99) == -1


def test_compute_path_option(lib):
    assert B.get_option(B.OPT_COMPUTE_PATH) == 0
    with pytest.raises(B.PdaError):
        B.set_option(B.OPT_COMPUTE_PATH, 2)
    try:
        B.set_option(B.OPT_COMPUTE_PATH, 1)
        assert B.get_option(B.OPT_COMPUTE_PATH) == 1
        # shapes outside the vector-ALU path fail before any device work
        for kw in (dict(d=64), dict(p=8), dict(hq=64, hkv=4)):
            assert call(**kw) == UNSUPPORTED and "vector-ALU" in B.last_error()
        assert ext_call(tq=3) == UNSUPPORTED and "vector-ALU" in B.last_error()  # 12 columns
        assert call(batch=4000) == UNSUPPORTED and "LDS" in B.last_error()
        f = B.load().paged_decode_attention_append
        rc = f(16, 16, 16, 16, 16, 16, 16, 16, 2, 32, 8, 64, 16, 64, 8, ctypes.c_float(0.1), None)
        assert rc == UNSUPPORTED and "vector-ALU" in B.last_error()
        # up to 8 columns per kv head are taken (batch 0: no device work)
        assert call(batch=0) == OK and ext_call(batch=0, tq=2) == OK
    finally:
        B.set_option(B.OPT_COMPUTE_PATH, 0)
    assert call(d=64, batch=0) == OK


def test_stream_read_argument_errors(lib):
    f = B.load().pda_stream_read
    assert f(16, 0, 16, 0, 0, None) == SHAPE and "multiple of 16" in B.last_error()
    assert f(16, 24, 16, 0, 0, None) == SHAPE
    assert f(16, 1024, 16, 3, 0, None) == UNSUPPORTED and "unroll" in B.last_error()
    assert f(16, 1024, 16, 8, 33, None) == UNSUPPORTED and "blocks_per_cu" in B.last_error()
    assert f(0, 1024, 16, 8, 8, None) == NULL
    assert f(16, 1024, 0, 8, 8, None) == NULL
    assert f(8, 1024, 16, 8, 8, None) == ALIGN
    assert f(16, 1024, 18, 8, 8, None) == ALIGN


def test_profile_read_null_pointer(lib):
    assert lib.pda_profile_read(None, None, None) == NULL
    s, m, n = B.profile_read()
    assert n == 0 and s == 0.0 and m == 0.0


def append_call(ptr=16, batch=2, hkv=8, d=128, p=16, n=64, maxp=8, ptrs=None):
    ptrs = ptrs or [ptr] * 6
    return B.load().pda_kv_append(*ptrs, batch, hkv, d, p, n, maxp, None)


@pytest.mark.parametrize("kwargs,code,text", [
    (dict(ptr=0), NULL, "NULL"),
    (dict(ptrs=[16, 16, 16, 16, 0, 16]), NULL, "NULL"),
    (dict(batch=-1), SHAPE, "batch"),
    (dict(hkv=0), SHAPE, "positive"),
    (dict(d=96), UNSUPPORTED, "head_dim"),
    (dict(hkv=1025), UNSUPPORTED, "num_kv_heads"),
    (dict(p=24), UNSUPPORTED, "page_size"),
    (dict(maxp=0), SHAPE, "positive"),
    (dict(n=0), SHAPE, "num_pages"),
    (dict(batch=8193), UNSUPPORTED, "batch"),
    (dict(ptrs=[16, 24, 16, 16, 16, 16]), ALIGN, "16-byte"),
    (dict(ptrs=[16, 16, 16, 40, 16, 16]), ALIGN, "16-byte"),
    (dict(ptrs=[16, 16, 16, 16, 16, 18]), ALIGN, "4-byte"),
])
def test_kv_append_argument_errors(lib, kwargs, code, text):
    rc = append_call(**kwargs)
    assert rc == code, B.last_error()
    assert text in B.last_error()


def test_kv_append_empty_batch_is_a_noop(lib):
    assert append_call(ptr=0, batch=0) == OK
    assert B.last_error() == ""


def test_append_then_attend_validates_attention_arguments_first(lib):
    # the attention arguments are checked before the append kernel could run
    f = B.load().paged_decode_attention_append
    rc = f(16, 16, 16, 16, 16, 16, 16, 16, 2, 32, 7, 128, 16, 64, 8, ctypes.c_float(0.1), None)
    assert rc == SHAPE and "multiple" in B.last_error()
    rc = f(16, 16, 16, 16, 16, 16, 16, 16, 2, 32, 8, 128, 16, 64, 8, ctypes.c_float(math.inf), None)
    assert rc == SCALE
    rc = f(0, 16, 16, 16, 16, 16, 16, 16, 2, 32, 8, 128, 16, 64, 8, ctypes.c_float(0.1), None)
    assert rc == NULL
    rc = f(16, 16, 16, 16, 16, 16, 16, 24, 2, 32, 8, 128, 16, 64, 8, ctypes.c_float(0.1), None)
    assert rc == ALIGN
    rc = f(16, 0, 16, 16, 16, 16, 16, 16, 2, 32, 8, 128, 16, 64, 8, ctypes.c_float(0.1), None)
    assert rc == NULL
    assert f(0, 0, 0, 0, 0, 0, 0, 0, 0, 32, 8, 128, 16, 64, 8, ctypes.c_float(0.1), None) == OK


def ext_call(batch=2, hq=32, hkv=8, tq=1, window=0, ptrs=None):
    ptrs = ptrs or [16] * 6
    return B.load().paged_decode_attention_ext(*ptrs, batch, hq, hkv, 128, 16, 64, 8, tq, window,
                                               ctypes.c_float(0.1), None)


@pytest.mark.parametrize("kwargs,code,text", [
    (dict(tq=0), SHAPE, "num_queries"),
    (dict(window=-1), SHAPE, "window"),
    (dict(tq=5), UNSUPPORTED, "exceeds 16"),          # 5 x group 4 = 20 columns
    (dict(hq=16, hkv=1, tq=2), UNSUPPORTED, "exceeds 16"),
    (dict(hq=8, hkv=8, tq=17), UNSUPPORTED, "exceeds 16"),
    (dict(ptrs=[0, 16, 16, 16, 16, 16]), NULL, "NULL"),
    (dict(hkv=7), SHAPE, "multiple"),
])
def test_ext_argument_errors(lib, kwargs, code, text):
    rc = ext_call(**kwargs)
    assert rc == code, B.last_error()
    assert text in B.last_error()


def test_ext_accepts_the_full_column_budget(lib):
    # 4 query tokens x group 4 and 16 x group 1 both fill the 16 columns; batch 0 is a no-op
    assert ext_call(batch=0, tq=4) == OK and ext_call(batch=0, hq=8, hkv=8, tq=16, window=3) == OK


def test_workspace_covers_every_num_queries(lib):
    _, _, ws = B.plan(4, 32, 8, 128, 16, 512, num_cus=256)
    g, _, _ = B.plan(4, 32, 8, 128, 16, 512, num_cus=256)
    assert ws >= (g + 4) * 8 * 16 * (128 + 2) * 4


# ------------------------------------------------------------------ prelude
def dims(**kw):
    d = dict(batch=2, hidden=512, hq=8, hkv=2, d=128, rotary_dim=128, interleaved=0, theta=1e4, eps=1e-6)
    d.update(kw)
    return B.PreludeDims(d["batch"], d["hidden"], d["hq"], d["hkv"], d["d"], d["rotary_dim"], d["interleaved"],
                         d["theta"], d["eps"])


def prelude_call(ptrs=None, **kw):
    p = ptrs or [16] * 9
    return B.load().pda_attention_prelude(*p, ctypes.byref(dims(**kw)), None)


@pytest.mark.parametrize("kwargs,code,text", [
    (dict(batch=-1), SHAPE, "batch"),
    (dict(batch=257), UNSUPPORTED, "batch"),
    (dict(batch=65, hq=5, hkv=1, d=64, rotary_dim=64), UNSUPPORTED, "multiple of 128"),   # 7 x 64 rows
    (dict(hidden=300), UNSUPPORTED, "hidden"),
    (dict(hidden=0), SHAPE, "positive"),
    (dict(hkv=3), SHAPE, "multiple"),
    (dict(d=96), UNSUPPORTED, "head_dim"),
    (dict(rotary_dim=7), SHAPE, "rotary_dim"),
    (dict(rotary_dim=130), SHAPE, "rotary_dim"),
    (dict(interleaved=2), SHAPE, "interleaved"),
    (dict(theta=0.0), SCALE, "rope_theta"),
    (dict(theta=float("inf")), SCALE, "rope_theta"),
    (dict(eps=-1.0), SCALE, "eps"),
    (dict(ptrs=[0] + [16] * 8), NULL, "NULL"),
    (dict(ptrs=[16, 16, 0, 16, 0, 16, 16, 16, 16]), NULL, "both"),   # q_norm without k_norm
    (dict(ptrs=[16, 16, 0, 0, 0, 16, 16, 16, 24]), ALIGN, "16-byte"),
    (dict(ptrs=[24, 16, 0, 0, 0, 16, 16, 16, 16]), ALIGN, "16-byte"),
])
def test_prelude_argument_errors(lib, kwargs, code, text):
    rc = prelude_call(**kwargs)
    assert rc == code, B.last_error()
    assert text in B.last_error()


def test_prelude_dims_null_and_empty_batch(lib):
    assert B.load().pda_attention_prelude(*[16] * 9, None, None) == NULL
    assert prelude_call(ptrs=[0] * 9, batch=0) == OK


def test_prelude_append_checks_the_cache_arguments(lib):
    f = B.load().pda_attention_prelude_append
    d = dims()
    assert f(*[16] * 10, 24, 64, 8, ctypes.byref(d), None) == UNSUPPORTED          # page size
    assert f(*[16] * 10, 16, 0, 8, ctypes.byref(d), None) == SHAPE                 # num_pages
    assert f(*[16] * 7, 0, 16, 16, 16, 64, 8, ctypes.byref(d), None) == NULL       # k_cache
    assert f(*[16] * 7, 24, 16, 16, 16, 64, 8, ctypes.byref(d), None) == ALIGN


@pytest.mark.parametrize("rows,cols,code", [(15, 64, SHAPE), (16, 48, SHAPE), (0, 64, SHAPE)])
def test_pack_argument_errors(lib, rows, cols, code):
    assert B.load().pda_pack_weights(16, 1 << 20, rows, cols, None) == code


def test_pack_rejects_overlap_and_null(lib):
    assert B.load().pda_pack_weights(4096, 4096 + 512, 16, 64, None) == SHAPE
    assert B.load().pda_pack_weights(0, 4096, 16, 64, None) == NULL


# ------------------------------------------------------------------ o_proj
def oproj_call(ptrs=None, batch=2, k=256, h=512, eps=1e-5):
    p = ptrs or [16] * 6
    return B.load().pda_o_proj_residual_norm(*p, batch, k, h, ctypes.c_float(eps), None)


@pytest.mark.parametrize("kwargs,code,text", [
    (dict(batch=-1), SHAPE, "batch"),
    (dict(batch=257), UNSUPPORTED, "batch"),
    (dict(batch=65, h=1040), UNSUPPORTED, "multiple of 128"),
    (dict(k=0), SHAPE, "positive"),
    (dict(k=100), UNSUPPORTED, "in_features"),
    (dict(h=24), UNSUPPORTED, "hidden"),
    (dict(h=32768 + 16), UNSUPPORTED, "hidden"),
    (dict(eps=float("nan")), SCALE, "eps"),
    (dict(ptrs=[16, 16, 0, 16, 16, 32]), NULL, "NULL"),
    (dict(ptrs=[24, 16, 16, 16, 16, 32]), ALIGN, "16-byte"),
    (dict(ptrs=[16, 16, 16, 16, 17, 32]), ALIGN, "2-byte"),
    (dict(ptrs=[16, 16, 16, 16, 32, 32]), SHAPE, "normed_out"),
])
def test_oproj_argument_errors(lib, kwargs, code, text):
    rc = oproj_call(**kwargs)
    assert rc == code, B.last_error()
    assert text in B.last_error()


def test_oproj_empty_batch_is_a_noop(lib):
    assert oproj_call(ptrs=[0] * 6, batch=0) == OK


def test_kv_append_n_token_count_errors(lib):
    f = B.load().pda_kv_append_n
    assert f(*[16] * 6, 2, 0, 8, 128, 16, 64, 8, None) == SHAPE and "num_tokens" in B.last_error()
    assert f(*[16] * 6, 2, 1025, 8, 128, 16, 64, 8, None) == SHAPE
    assert f(*[0] * 6, 0, 4, 8, 128, 16, 64, 8, None) == OK


def test_validate_paging_argument_errors(lib):
    f = B.load().pda_validate_paging
    assert f(16, 16, -1, 8, 16, 64, None) == SHAPE
    assert f(16, 16, 2, 0, 16, 64, None) == SHAPE
    assert f(0, 16, 2, 8, 16, 64, None) == NULL
    assert f(0, 0, 0, 8, 16, 64, None) == OK


# ------------------------------------------------- tensor-descriptor entry
DTYPE, LAYOUT = 7, 8
BF, F16, F32, I32, I64 = B.DTYPE_BF16, B.DTYPE_F16, B.DTYPE_F32, B.DTYPE_I32, B.DTYPE_I64


def _descs(batch=2, hq=32, hkv=8, d=128, p=16, n=64, maxp=8, ptr=0x1000):
    T = B.tensor_desc
    return dict(q=T(ptr, BF, (batch, hq, d)), k=T(ptr, BF, (n, p, hkv, d)), v=T(ptr, BF, (n, p, hkv, d)),
                bt=T(ptr, I32, (batch, maxp)), lens=T(ptr, I32, (batch,)), out=T(ptr, BF, (batch, hq, d)))


def desc_call(scale=0.088, **replace):
    ds = _descs(**{k: replace.pop(k) for k in list(replace) if k in ("batch", "hq", "hkv", "d", "p", "n", "maxp")})
    ds.update(replace)
    return B.desc_call(ds["q"], ds["k"], ds["v"], ds["bt"], ds["lens"], ds["out"], scale)


T = B.tensor_desc
DESC_ERRORS = [
    # a missing descriptor, or a non-empty tensor without data
    (dict(q=None), NULL, "q: descriptor is NULL"),
    (dict(lens=None), NULL, "context_lens: descriptor is NULL"),
    (dict(k=T(0, BF, (64, 16, 8, 128))), NULL, "k_cache: data is NULL"),
    # element types: nothing is converted
    (dict(q=T(0x1000, F16, (2, 32, 128))), DTYPE, "q: dtype fp16"),
    (dict(v=T(0x1000, F32, (64, 16, 8, 128))), DTYPE, "v_cache: dtype fp32"),
    (dict(lens=T(0x1000, I64, (2,))), DTYPE, "context_lens: dtype int64"),
    (dict(bt=T(0x1000, BF, (2, 8))), DTYPE, "block_table: dtype bf16"),
    (dict(out=T(0x1000, 99, (2, 32, 128))), DTYPE, "out: dtype unknown"),
    # ranks, extents and their agreement
    (dict(q=T(0x1000, BF, (2, 4096))), SHAPE, "q: 2 dimensions"),
    (dict(q=T(0x1000, BF, (2, -32, 128))), SHAPE, "out of range"),
    (dict(out=T(0x1000, BF, (2, 32, 64))), SHAPE, "out must have the shape of q"),
    (dict(v=T(0x1000, BF, (64, 16, 4, 128))), SHAPE, "v_cache must have the shape of k_cache"),
    (dict(k=T(0x1000, BF, (64, 16, 8, 64)), v=T(0x1000, BF, (64, 16, 8, 64))), SHAPE, "head_dim"),
    (dict(bt=T(0x1000, I32, (3, 8))), SHAPE, "one row per sequence"),
    (dict(lens=T(0x1000, I32, (1,))), SHAPE, "one row per sequence"),
    (dict(hq=30), SHAPE, "multiple"),
    (dict(n=0), SHAPE, "num_pages"),
    # supported set
    (dict(d=96), UNSUPPORTED, "head_dim"),
    (dict(p=24), UNSUPPORTED, "page_size"),
    (dict(hq=64, hkv=2), UNSUPPORTED, "group"),
    # layouts: transposed, sliced and padded views
    (dict(q=T(0x1000, BF, (2, 32, 128), (4096, 1, 32))), LAYOUT, "q: stride"),
    (dict(k=T(0x1000, BF, (64, 16, 8, 128), (16 * 8 * 128, 128, 16 * 128, 1))), LAYOUT, "k_cache: stride"),
    (dict(bt=T(0x1000, I32, (2, 8), (16, 1))), LAYOUT, "block_table: stride"),
    (dict(lens=T(0x1000, I32, (2,), (2,))), LAYOUT, "context_lens: stride"),
    (dict(out=T(0x1000, BF, (2, 32, 128), (8192, 256, 1))), LAYOUT, "out: stride"),
    # the rest of the pointer entry point's checks
    (dict(scale=float("nan")), SCALE, "finite"),
    (dict(q=T(0x1008, BF, (2, 32, 128))), ALIGN, "16-byte"),
]


@pytest.mark.parametrize("kwargs,code,text", DESC_ERRORS, ids=[f"{e[1]}-{e[2]}" for e in DESC_ERRORS])
def test_descriptor_errors(lib, kwargs, code, text):
    rc = desc_call(**kwargs)
    assert rc == code, B.last_error()
    assert text in B.last_error()


def test_descriptor_extent_one_and_empty_tensors_have_no_layout(lib):
    # the stride of an extent-1 dimension is not looked at, and an empty
    # batch (no data pointers needed) returns before any HIP call
    q = T(0x1000, BF, (1, 32, 128), (999, 128, 1))
    assert desc_call(batch=1, q=q, out=T(0x1000, BF, (1, 32, 128), (7, 128, 1)), scale=float("nan")) == SCALE
    e = _descs(batch=0, ptr=0)
    e["k"], e["v"] = T(0x1000, BF, (64, 16, 8, 128)), T(0x1000, BF, (64, 16, 8, 128))
    assert B.desc_call(e["q"], e["k"], e["v"], e["bt"], e["lens"], e["out"], 0.088) == OK
    assert B.last_error() == ""


# ------------------------------------------- binding argument checks (CPU)
# CPU tensors: with every shape and dtype right, a wrapper stops at "must be
# a GPU tensor"; a wrong shape or dtype is reported before that, so each bad
# argument raises before any launch whichever it is.
def _t(*shape, dtype=None):
    import torch
    return torch.zeros(shape, dtype=dtype or torch.bfloat16)


def _i32(*shape):
    import torch
    return torch.zeros(shape, dtype=torch.int32)


def _prelude_args(**over):
    # B 2, H 64, Hq 4, Hkv 2, D 64: N = (4 + 4) * 64 = 512
    a = dict(x=_t(2, 64), w_packed=_t(512, 64), context_lens=_i32(2), q_out=_t(2, 4, 64), k_out=_t(2, 2, 64),
             v_out=_t(2, 2, 64), bias=_t(512), q_norm=_t(64), k_norm=_t(64))
    a.update(over)
    return a


PRELUDE_BAD = [
    (dict(w_packed=_t(448, 64)), "w_packed must be [N, H] with N = 512"),
    (dict(x=_t(2, 96)), "w_packed must be [N, H] with H = 96"),
    (dict(q_out=_t(2, 4, 32)), "q_out must be [B, Hq, D] with D = 64"),
    (dict(k_out=_t(2, 3, 64)), "k_out must be [B, Hkv, D] with Hkv = 2"),
    (dict(v_out=_t(3, 2, 64)), "v_out must be [B, Hkv, D] with B = 2"),
    (dict(context_lens=_i32(3)), "context_lens must be [B] with B = 2"),
    (dict(bias=_t(500)), "bias must be [N] with N = 512"),
    (dict(q_norm=_t(32)), "q_norm must be [D] with D = 64"),
    (dict(x=_t(2, 1, 64)), "x must be [B, H]"),
]


@pytest.mark.parametrize("over,text", PRELUDE_BAD, ids=[t for _, t in PRELUDE_BAD])
def test_prelude_binding_shape_checks(over, text):
    a = _prelude_args(**over)
    with pytest.raises(ValueError, match=re.escape(text)):
        B.attention_prelude(**a, num_q_heads=4, num_kv_heads=2, head_dim=64, rope_theta=1e4)


def test_prelude_binding_dtype_device_and_norm_pair_checks():
    import torch
    kw = dict(num_q_heads=4, num_kv_heads=2, head_dim=64, rope_theta=1e4)
    with pytest.raises(TypeError, match="context_lens must be torch.int32"):
        B.attention_prelude(**_prelude_args(context_lens=torch.zeros(2, dtype=torch.int64)), **kw)
    with pytest.raises(TypeError, match="bias must be torch.bfloat16"):
        B.attention_prelude(**_prelude_args(bias=torch.zeros(512)), **kw)
    with pytest.raises(ValueError, match="both be given"):
        B.attention_prelude(**_prelude_args(k_norm=None), **kw)
    with pytest.raises(ValueError, match="must be a GPU tensor"):
        B.attention_prelude(**_prelude_args(), **kw)


def test_prelude_append_binding_checks_the_caches():
    kw = dict(num_q_heads=4, num_kv_heads=2, head_dim=64, rope_theta=1e4)

    def call(**over):
        a = _prelude_args()
        del a["k_out"], a["v_out"]
        a.update(k_cache=_t(10, 16, 2, 64), v_cache=_t(10, 16, 2, 64), block_table=_i32(2, 5))
        a.update(over)
        B.attention_prelude_append(**a, **kw)
    with pytest.raises(ValueError, match=re.escape("k_cache must be [Np, P, Hkv, D] with Hkv = 2")):
        call(k_cache=_t(10, 16, 4, 64))
    with pytest.raises(ValueError, match=re.escape("v_cache must be [Np, P, Hkv, D] with P = 16")):
        call(v_cache=_t(10, 8, 2, 64))
    with pytest.raises(ValueError, match=re.escape("block_table must be [B, M] with B = 2")):
        call(block_table=_i32(3, 5))
    with pytest.raises(ValueError, match="must be a GPU tensor"):
        call()


def test_append_then_attend_binding_checks():
    def call(**over):
        a = dict(q=_t(2, 8, 64), k_new=_t(2, 2, 64), v_new=_t(2, 2, 64), k_cache=_t(10, 16, 2, 64),
                 v_cache=_t(10, 16, 2, 64), block_table=_i32(2, 5), context_lens=_i32(2), out=_t(2, 8, 64))
        a.update(over)
        B.paged_decode_attention_append(**a, scale=0.125)
    with pytest.raises(ValueError, match=re.escape("block_table must be [B, M] with B = 2")):
        call(block_table=_i32(3, 5))
    with pytest.raises(ValueError, match=re.escape("context_lens must be [B] with B = 2")):
        call(context_lens=_i32(1))
    with pytest.raises(ValueError, match=re.escape("q must be [B, Hq, D]")):
        call(q=_t(2, 1, 8, 64))
    with pytest.raises(ValueError, match=re.escape("k_new must be [B, Hkv, D] with D = 64")):
        call(k_new=_t(2, 2, 32))
    with pytest.raises(ValueError, match="must be a GPU tensor"):
        call()


def test_o_proj_and_kv_append_binding_checks():
    def oproj(**over):
        a = dict(attn=_t(2, 64), w_packed=_t(32, 64), residual=_t(2, 32), norm_w=_t(32), residual_out=_t(2, 32),
                 normed_out=_t(2, 32))
        a.update(over)
        B.o_proj_residual_norm(**a)
    with pytest.raises(ValueError, match=re.escape("w_packed must be [H, K] with K = 64")):
        oproj(w_packed=_t(32, 96))
    with pytest.raises(ValueError, match=re.escape("norm_w must be [H] with H = 32")):
        oproj(norm_w=_t(16))
    with pytest.raises(ValueError, match="must be a GPU tensor"):
        oproj()
    with pytest.raises(ValueError, match=re.escape("v_new must be [B, Hkv, D] with Hkv = 2")):
        B.kv_append(_t(2, 2, 64), _t(2, 1, 64), _t(10, 16, 2, 64), _t(10, 16, 2, 64), _i32(2, 5), _i32(2))


def test_fused_merge_option(lib):
    assert B.get_option(B.OPT_FUSED_MERGE) == 0
    with pytest.raises(B.PdaError):
        B.set_option(B.OPT_FUSED_MERGE, 3)
    try:
        for v in (1, 2, 0):
            B.set_option(B.OPT_FUSED_MERGE, v)
            assert B.get_option(B.OPT_FUSED_MERGE) == v
        # the reserve bound covers every kv-head grouping the planner may pick
        # (a single request takes one kv head per workgroup with the fused merge)
        _, _, ws = B.plan(1, 32, 8, 128, 16, 256, num_cus=256)
        assert ws >= (64 + 8) * 1 * 16 * (128 + 2) * 4
    finally:
        B.set_option(B.OPT_FUSED_MERGE, 0)
