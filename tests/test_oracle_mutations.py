"""The oracle's pins are sharp: plant a plausible mistake in (a copy of) the
oracle's arithmetic, on the CPU, and check that at least one pin fails."""
import functools

import numpy as np
import pytest

import oracle
import test_oracle as pins
from _golden import cases as golden_cases


def make_one_group(slot_swap=False, no_scale=False, no_shift=False, short=False,
                   no_norm=False, neg=False, kv_swap=False, head_mod=False):
    def _one_group(q_bits, k_bits, v_bits, bt_row, length, page_size, g, group, sigma):
        d = q_bits.shape[-1]
        if length == 0:
            return np.zeros((group, d)), np.full(group, -np.inf), np.zeros((group, 0))
        n = length - 1 if short else length
        t = np.arange(n)
        if slot_swap:
            pages = np.asarray(bt_row)[np.minimum(t % page_size, len(bt_row) - 1)].astype(np.int64)
            slots = np.minimum(t // page_size, page_size - 1)
        else:
            pages = np.asarray(bt_row)[t // page_size].astype(np.int64)
            slots = t % page_size
        kt = oracle.bf16_to_f64(k_bits[pages, slots, g, :])
        vt = oracle.bf16_to_f64(v_bits[pages, slots, g, :])
        if kv_swap:
            kt, vt = vt, kt
        hkv = k_bits.shape[2]
        rows = q_bits[g::hkv] if head_mod else q_bits[g * group:(g + 1) * group]
        qg = oracle.bf16_to_f64(rows)
        s = (1.0 if no_scale else sigma) * (qg @ kt.T)
        if neg:
            s = -s
        with np.errstate(over="ignore", invalid="ignore"):
            m = np.zeros((group, 1)) if no_shift else s.max(axis=1, keepdims=True)
            e = np.exp(s - m)
            den = e.sum(axis=1, keepdims=True)
            w = e if no_norm else e / den
            return w @ vt, (m + np.log(den))[:, 0], w
    return _one_group


MUTANTS = {
    "page/slot swapped": dict(slot_swap=True),
    "scale dropped": dict(no_scale=True),
    "no max shift": dict(no_shift=True),
    "one token short": dict(short=True),
    "weights not normalised": dict(no_norm=True),
    "score sign flipped": dict(neg=True),
    "K and V swapped": dict(kv_swap=True),
    "head h -> kv head h % Hkv": dict(head_mod=True),
}

PIN_FUNCS = [
    pins.test_length_one_returns_v_exactly,
    pins.test_constant_v_returns_constant,
    pins.test_zero_query_gives_mean_of_values,
    pins.test_brute_force_dense_independent_gather,
    pins.test_matches_torch_sdpa_fp64,
    pins.test_gqa_mapping_probe,
    pins.test_dominant_token_no_overflow,
    pins.test_brute_force_fsum_tiny,
]


def test_unmutated_oracle_passes_every_pin():
    for f in PIN_FUNCS:
        f()


@pytest.mark.parametrize("name", list(MUTANTS))
def test_each_mutant_is_caught(name, monkeypatch):
    monkeypatch.setattr(oracle, "_one_group", make_one_group(**MUTANTS[name]))
    failed = []
    for f in PIN_FUNCS:
        try:
            with np.errstate(all="ignore"):
                f()
        except (AssertionError, ValueError, IndexError, FloatingPointError):
            failed.append(f.__name__)
    for gname, w, expected in golden_cases():
        try:
            with np.errstate(all="ignore"):
                pins.test_golden_closed_forms(gname, w, expected)
        except (AssertionError, ValueError, IndexError):
            failed.append("golden:" + gname)
    assert failed, f"mutant '{name}' passed every pin"


def make_kv_append(at_len=False, slot_swap=False, kv_swap=False, write_empty=False):
    def kv_append(k_cache, v_cache, k_new, v_new, block_table, context_lens):
        k = np.array(k_cache, copy=True)
        v = np.array(v_cache, copy=True)
        p = k.shape[1]
        for b in range(len(context_lens)):
            length = int(context_lens[b])
            if length == 0 and not write_empty:
                continue
            t = length if at_len else length - 1
            j, r = (t % p, t // p) if slot_swap else (t // p, t % p)
            j = min(j, block_table.shape[1] - 1)
            r = min(r, p - 1)
            page = int(block_table[b][j])
            k[page, r], v[page, r] = (v_new[b], k_new[b]) if kv_swap else (k_new[b], v_new[b])
        return k, v
    return kv_append


APPEND_MUTANTS = {
    "position L instead of L-1": dict(at_len=True),
    "page/slot swapped": dict(slot_swap=True),
    "K and V swapped": dict(kv_swap=True),
    "empty sequences written": dict(write_empty=True),
}
APPEND_PINS = [pins.test_kv_append_writes_exactly_the_new_slot,
               pins.test_append_then_attend_equals_attend_on_the_full_cache]


@pytest.mark.parametrize("name", list(APPEND_MUTANTS))
def test_each_append_mutant_is_caught(name, monkeypatch):
    monkeypatch.setattr(oracle, "kv_append", make_kv_append(**APPEND_MUTANTS[name]))
    failed = []
    for f in APPEND_PINS:
        try:
            with np.errstate(all="ignore"):
                f()
        except (AssertionError, ValueError, IndexError):
            failed.append(f.__name__)
    assert failed, f"mutant '{name}' passed every pin"


def make_visible_range(window_off=False, causal_off=False, from_start=False):
    def visible_range(length, num_queries, j, window):
        p = int(j) if from_start else int(length) - int(num_queries) + int(j)
        hi = p if causal_off else p + 1
        if window > 0:
            lo = max(0, hi - int(window) + (1 if window_off else 0))
        else:
            lo = 0
        return lo, max(hi, lo)
    return visible_range


def reversed_queries(orig):
    def attend_masked(q, *args, **kw):
        return orig(np.ascontiguousarray(q[:, ::-1]), *args, **kw)
    return attend_masked


MASK_PINS = [
    pins.test_masked_single_query_without_window_is_attend,
    pins.test_masked_queries_are_causal_prefixes,
    *[functools.partial(pins.test_masked_matches_torch_sdpa_with_boolean_mask, tq, wdw)
      for tq, wdw in [(1, 5), (2, 16), (4, 1), (3, 40), (2, 0)]],
    pins.test_window_of_one_returns_the_own_value,
    pins.test_window_released_pages_are_never_read,
    pins.test_queries_before_the_first_token_are_zero,
]
MASK_MUTANTS = {
    "window one token short": ("visible_range", make_visible_range(window_off=True)),
    "query sees its own token excluded": ("visible_range", make_visible_range(causal_off=True)),
    "query positions from the start": ("visible_range", make_visible_range(from_start=True)),
    "query tokens in reverse order": ("attend_masked", reversed_queries(oracle.attend_masked)),
}


@pytest.mark.parametrize("name", list(MASK_MUTANTS))
def test_each_masked_mutant_is_caught(name, monkeypatch):
    attr, fn = MASK_MUTANTS[name]
    monkeypatch.setattr(oracle, attr, fn)
    failed = []
    for f in MASK_PINS:
        try:
            with np.errstate(all="ignore"):
                f()
        except (AssertionError, ValueError, IndexError):
            failed.append(getattr(f, "__name__", str(f)))
    assert failed, f"mutant '{name}' passed every pin"


# ------------------------------------------------------------------ prelude
import test_oracle_prelude as ppins  # noqa: E402

_rope, _rms, _prelude = oracle.rope, oracle.rms_norm, oracle.prelude


def rope_mutant(sign=1.0, swap_pairs=False, exponent=2.0):
    def rope(t, positions, theta, rotary_dim, interleaved=False):
        t = np.array(t, dtype=np.float64, copy=True)
        half = rotary_dim // 2
        inter = (not interleaved) if swap_pairs else interleaved
        for i in range(half):
            a, b = (2 * i, 2 * i + 1) if inter else (i, i + half)
            ang = np.asarray(positions, dtype=np.float64) * float(np.float32(theta)) ** (-exponent * i / rotary_dim)
            c, s_ = np.cos(ang)[:, None], sign * np.sin(ang)[:, None]
            xa, xb = t[..., a].copy(), t[..., b].copy()
            t[..., a] = xa * c - xb * s_
            t[..., b] = xb * c + xa * s_
        return t
    return rope


def rms_mutant(t, weight_bits, eps):
    t = np.asarray(t, dtype=np.float64)
    return t / np.sqrt(np.sum(t * t, axis=-1, keepdims=True) + float(np.float32(eps))) * oracle.bf16_to_f64(weight_bits)


def prelude_kv_swapped(*a, **kw):
    q, k, v = _prelude(*a, **kw)
    return q, v, k


def prelude_norm_after_rope(x, w, hq, hkv, d, lens, theta, **kw):
    qn, kn, eps = kw.pop("q_norm", None), kw.pop("k_norm", None), kw.get("eps", 1e-6)
    q, k, v = _prelude(x, w, hq, hkv, d, lens, theta, **kw)
    if qn is not None:
        q, k = _rms(q, qn, eps), _rms(k, kn, eps)
    return q, k, v


PRELUDE_PINS = [
    ppins.test_integer_projection_is_exact_and_blocks_are_ordered_q_k_v,
    ppins.test_bias_adds_to_every_row,
    *[functools.partial(ppins.test_rope_is_complex_multiplication, i, rd) for i in (False, True) for rd in (16, 8)],
    ppins.test_rope_scores_depend_only_on_relative_position,
    ppins.test_rope_at_position_zero_is_identity_and_keeps_pair_norms,
    ppins.test_rms_norm_matches_torch,
    *[functools.partial(ppins.test_prelude_matches_independent_torch_formulation, kw)
      for kw in (dict(), dict(qk_norm=True), dict(bias=True, rotary_dim=8, interleaved=True),
                 dict(qk_norm=True, rotary_dim=8))],
    ppins.test_position_is_length_minus_one_and_empty_slots_use_zero,
]
PRELUDE_MUTANTS = {
    "rotation the other way": ("rope", rope_mutant(sign=-1.0)),
    "pairs of the other convention": ("rope", rope_mutant(swap_pairs=True)),
    "frequency exponent halved": ("rope", rope_mutant(exponent=1.0)),
    "norm by the sum of squares": ("rms_norm", rms_mutant),
    "k and v blocks swapped": ("prelude", prelude_kv_swapped),
    "norm applied after the rotation": ("prelude", prelude_norm_after_rope),
}


@pytest.mark.parametrize("name", list(PRELUDE_MUTANTS))
def test_each_prelude_mutant_is_caught(name, monkeypatch):
    attr, fn = PRELUDE_MUTANTS[name]
    monkeypatch.setattr(oracle, attr, fn)
    failed = []
    for f in PRELUDE_PINS:
        try:
            with np.errstate(all="ignore"):
                f()
        except (AssertionError, ValueError, IndexError):
            failed.append(getattr(f, "__name__", str(f)))
    assert failed, f"mutant '{name}' passed every pin"


# ------------------------------------------------------------------ o_proj
import test_oracle_oproj as opins  # noqa: E402

_oproj = oracle.o_proj_residual_norm


def oproj_no_residual(attn, w_o, residual, norm_w, eps):
    z = oracle.bf16_to_f64(attn) @ oracle.bf16_to_f64(w_o).T
    return z, oracle.rms_norm(z, norm_w, eps)


def oproj_norm_before_residual(attn, w_o, residual, norm_w, eps):
    y = oracle.bf16_to_f64(attn) @ oracle.bf16_to_f64(w_o).T
    z = y + oracle.bf16_to_f64(residual)
    return z, oracle.rms_norm(y, norm_w, eps) + 0 * z


def oproj_transposed(attn, w_o, residual, norm_w, eps):
    a = oracle.bf16_to_f64(attn)
    wt = oracle.bf16_to_f64(w_o)
    z = (a @ wt.reshape(wt.shape[1], wt.shape[0])).reshape(len(a), -1)[:, :wt.shape[0]] + oracle.bf16_to_f64(residual)
    return z, oracle.rms_norm(z, norm_w, eps)


OPROJ_PINS = [opins.test_integer_projection_plus_residual_is_exact,
              opins.test_norm_output_has_unit_rms_and_ignores_scale,
              *[functools.partial(opins.test_matches_torch_linear_and_rms_norm, e) for e in (1e-6, 1e-5, 0.5)]]
OPROJ_MUTANTS = {"residual dropped": oproj_no_residual, "norm of the projection alone": oproj_norm_before_residual,
                 "weights read transposed": oproj_transposed}


@pytest.mark.parametrize("name", list(OPROJ_MUTANTS))
def test_each_oproj_mutant_is_caught(name, monkeypatch):
    monkeypatch.setattr(oracle, "o_proj_residual_norm", OPROJ_MUTANTS[name])
    failed = []
    for f in OPROJ_PINS:
        try:
            with np.errstate(all="ignore"):
                f()
        except (AssertionError, ValueError, IndexError):
            failed.append(getattr(f, "__name__", str(f)))
    assert failed, f"mutant '{name}' passed every pin"
