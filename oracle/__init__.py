"""fp64 CPU oracle for paged decode attention -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP library
(no kernels, headers, helpers or constants) and never calls it.

What it computes.  The paper's kernel family (iv) (Method, "Principle-Driven
LLM Kernel Generator") is single-token decode attention over a paged KV cache:
an online-softmax pass over the cached keys and values of each sequence, split
across workgroups and finished by a merge of the per-split results.  Split
plus online softmax plus merge reaches, in exact arithmetic, plain softmax
attention of one query row over the sequence's cached tokens, so
:func:`attend` is that plain definition written out:

    for sequence b with L_b cached tokens and query head h, with kv head
    g = h // G (G = Hq / Hkv, consecutive query heads share a kv head),
        k_t = K[page(b, t), t mod P, g, :],  v_t likewise,
        page(b, t) = block_table[b, t // P],
        s_t = sigma * <q[b, h, :], k_t>          (sigma = the fp32 scale)
        w_t = exp(s_t - max s) / sum_u exp(s_u - max s)
        out[b, h, :] = sum_t w_t v_t,   lse = max s + log sum_u exp(s_u - max s)

with every bf16 input widened exactly to fp64 and all arithmetic in fp64.
A sequence with L_b = 0 yields a zero row (lse = -inf).

:func:`split_merge` follows the algorithm instead: per-chunk running max,
denominator and unnormalised accumulator, then the log-sum-exp merge of the
chunks.  It is pinned against :func:`attend` for arbitrary chunkings.

:func:`kv_append` is the step before attention in the paper's decode loop:
the new token's key and value are scattered into their page slot and the
length already counts that token.

:func:`prelude` is the attention prelude that produces this step's q, k and
v (Method, "Principle-Driven LLM Kernel Generator", kernel family (i): QKV
projection plus rotary position embedding, optionally with a per-head
RMSNorm of q and k).

:func:`o_proj_residual_norm` is the step after attention (kernel family (v)
of the same section: the output projection fused with the residual add and
the RMSNorm that follows it).

:func:`attend_masked` is the same definition with a key range per query:
several query tokens per sequence (the decode steps that the paper's engine
mixes with chunked prefill, each seeing only keys up to its own position)
and an optional sliding window (the Mistral adaptation in the paper's table
of model-specific adaptations).

Readings where the paper is silent (it prints no attention formula, page
size, layout or tolerance): standard scaled dot-product softmax with no other
mask than the length, KV pool layout [num_pages, P, Hkv, D], lengths that
include the token appended for the current step, and zero output for an
empty sequence.
"""
from __future__ import annotations

import math
from typing import Iterable, List, Optional, Sequence, Tuple

import numpy as np

__all__ = ["bf16_to_f64", "attend", "attend_pairs", "weights", "split_merge",
           "brute_force_tiny", "kv_append", "attend_masked", "visible_range",
           "prelude", "rms_norm", "rope", "o_proj_residual_norm"]


def bf16_to_f64(bits) -> np.ndarray:
    """Exact value of bf16 bit patterns as float64 (bits are the top half of
    an IEEE float32)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def _sigma(scale) -> float:
    # the kernel receives the scale as fp32; use exactly that number
    return float(np.float32(scale))


def _gather(cache_bits, block_table_row, length, page_size, g, start=0) -> np.ndarray:
    """[L - start, D] fp64 rows of kv head g for tokens start..L-1 of one
    sequence."""
    t = np.arange(start, length)
    pages = np.asarray(block_table_row)[t // page_size].astype(np.int64)
    slots = t % page_size
    return bf16_to_f64(cache_bits[pages, slots, g, :])


def _one_group(q_bits, k_bits, v_bits, bt_row, length, page_size, g, group, sigma):
    """Outputs [G, D] and lse [G] for kv head g of one sequence."""
    d = q_bits.shape[-1]
    if length == 0:
        return np.zeros((group, d)), np.full(group, -np.inf), np.zeros((group, 0))
    kt = _gather(k_bits, bt_row, length, page_size, g)
    vt = _gather(v_bits, bt_row, length, page_size, g)
    qg = bf16_to_f64(q_bits[g * group:(g + 1) * group, :])
    s = sigma * (qg @ kt.T)                      # [G, L]
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    den = e.sum(axis=1, keepdims=True)
    w = e / den
    return w @ vt, (m + np.log(den))[:, 0], w


def attend(q, k_cache, v_cache, block_table, context_lens, scale):
    """Plain fp64 decode attention over the whole batch.

    q: uint16 [B, Hq, D]; k_cache, v_cache: uint16 [N, P, Hkv, D];
    block_table: int [B, maxp]; context_lens: int [B]; scale: float.
    Returns (out float64 [B, Hq, D], lse float64 [B, Hq]).
    """
    bsz, hq, d = q.shape
    _, page_size, hkv, _ = k_cache.shape
    group = hq // hkv
    sigma = _sigma(scale)
    out = np.zeros((bsz, hq, d))
    lse = np.full((bsz, hq), -np.inf)
    for b in range(bsz):
        length = int(context_lens[b])
        for g in range(hkv):
            o, l_, _ = _one_group(q[b], k_cache, v_cache, block_table[b], length,
                                  page_size, g, group, sigma)
            out[b, g * group:(g + 1) * group] = o
            lse[b, g * group:(g + 1) * group] = l_
    return out, lse


def attend_pairs(q, k_cache, v_cache, block_table, context_lens, scale,
                 pairs: Iterable[Tuple[int, int]]):
    """Same definition for selected (sequence b, kv head g) pairs only.

    Returns {(b, g): (out [G, D], lse [G])}; used to check full-size runs on
    sampled outputs.
    """
    hq = q.shape[1]
    _, page_size, hkv, _ = k_cache.shape
    group = hq // hkv
    sigma = _sigma(scale)
    res = {}
    for b, g in pairs:
        o, l_, _ = _one_group(q[b], k_cache, v_cache, block_table[b],
                              int(context_lens[b]), page_size, g, group, sigma)
        res[(int(b), int(g))] = (o, l_)
    return res


def weights(q, k_cache, block_table, context_lens, scale, b, h) -> np.ndarray:
    """Softmax weights w_t (fp64, length L_b) of query head h of sequence b."""
    hq = q.shape[1]
    _, page_size, hkv, _ = k_cache.shape
    group = hq // hkv
    g = h // group
    length = int(context_lens[b])
    _, _, w = _one_group(q[b], k_cache, k_cache, block_table[b], length,
                         page_size, g, group, _sigma(scale))
    return w[h - g * group]


def split_merge(q, k_cache, v_cache, block_table, context_lens, scale,
                bounds: Sequence[Sequence[int]]):
    """Split-then-merge form of the same attention, in fp64.

    ``bounds[b]`` is an increasing list of token offsets 0 = c_0 <= c_1 <= ...
    <= c_n = L_b; chunk j covers tokens [c_j, c_{j+1}) and may be empty.
    Per chunk (and query head): m_j = max s, l_j = sum exp(s - m_j),
    a_j = sum exp(s - m_j) v.  Merge: M = max over non-empty chunks of m_j,
    out = sum_j exp(m_j - M) a_j / sum_j exp(m_j - M) l_j; empty chunks carry
    no weight.  Returns out float64 [B, Hq, D].
    """
    bsz, hq, d = q.shape
    _, page_size, hkv, _ = k_cache.shape
    group = hq // hkv
    sigma = _sigma(scale)
    out = np.zeros((bsz, hq, d))
    for b in range(bsz):
        length = int(context_lens[b])
        cuts = list(bounds[b])
        assert cuts[0] == 0 and cuts[-1] == length and all(
            x <= y for x, y in zip(cuts, cuts[1:]))
        if length == 0:
            continue
        for g in range(hkv):
            kt = _gather(k_cache, block_table[b], length, page_size, g)
            vt = _gather(v_cache, block_table[b], length, page_size, g)
            qg = bf16_to_f64(q[b, g * group:(g + 1) * group, :])
            parts = []
            for lo, hi in zip(cuts, cuts[1:]):
                if hi == lo:
                    continue
                s = sigma * (qg @ kt[lo:hi].T)          # [G, n]
                m = s.max(axis=1, keepdims=True)
                e = np.exp(s - m)
                parts.append((m[:, 0], e.sum(axis=1), e @ vt[lo:hi]))
            big_m = np.max(np.stack([p[0] for p in parts]), axis=0)       # [G]
            num = np.zeros((group, d))
            den = np.zeros(group)
            for m_j, l_j, a_j in parts:
                f = np.exp(m_j - big_m)
                num += f[:, None] * a_j
                den += f * l_j
            out[b, g * group:(g + 1) * group] = num / den[:, None]
    return out


def brute_force_tiny(q, k_cache, v_cache, block_table, context_lens, scale):
    """Pure-Python loops with exactly rounded sums (math.fsum); for tiny
    inputs only.  Returns a nested list out[b][h][d] of floats."""
    bsz, hq, d = q.shape
    _, page_size, hkv, _ = k_cache.shape
    group = hq // hkv
    sigma = _sigma(scale)
    qf = bf16_to_f64(q)
    kf = bf16_to_f64(k_cache)
    vf = bf16_to_f64(v_cache)
    result: List[List[List[float]]] = []
    for b in range(bsz):
        rows = []
        length = int(context_lens[b])
        for h in range(hq):
            g = h // group
            if length == 0:
                rows.append([0.0] * d)
                continue
            scores = []
            for t in range(length):
                page = int(block_table[b][t // page_size])
                slot = t % page_size
                scores.append(sigma * math.fsum(
                    float(qf[b, h, i]) * float(kf[page, slot, g, i]) for i in range(d)))
            top = max(scores)
            ex = [math.exp(s - top) for s in scores]
            den = math.fsum(ex)
            row = []
            for i in range(d):
                acc = []
                for t in range(length):
                    page = int(block_table[b][t // page_size])
                    slot = t % page_size
                    acc.append(ex[t] * float(vf[page, slot, g, i]))
                row.append(math.fsum(acc) / den)
            rows.append(row)
        result.append(rows)
    return result


def kv_append(k_cache, v_cache, k_new, v_new, block_table, context_lens):
    """The KV append that precedes decode attention (Method, "Kernel
    Customization and Multi-Request Adaptation": a scatter kernel writes the
    new key and value vectors, and attention then runs with the sequence
    length advanced by one).

    ``context_lens`` already counts the new token, so sequence b's new key
    and value (``k_new[b]``, ``v_new[b]``: [Hkv, D] bf16 bits) land at
    position L_b - 1: page ``block_table[b, (L_b - 1) // P]``, slot
    ``(L_b - 1) % P``, every kv head.  Sequences with L_b = 0 write nothing.

    With several new tokens per sequence (``k_new``: [B, T, Hkv, D]), the
    lengths count all of them and token j lands at position L_b - T + j;
    positions below 0 (L_b < T) write nothing.
    Returns new (k_cache, v_cache) arrays; the inputs are not modified.
    """
    k = np.array(k_cache, copy=True)
    v = np.array(v_cache, copy=True)
    page_size = k.shape[1]
    kn = np.asarray(k_new)
    vn = np.asarray(v_new)
    if kn.ndim == 3:
        kn, vn = kn[:, None], vn[:, None]
    tokens = kn.shape[1]
    for b in range(len(context_lens)):
        length = int(context_lens[b])
        for j in range(tokens):
            t = length - tokens + j
            if t < 0:
                continue
            page = int(block_table[b][t // page_size])
            k[page, t % page_size] = kn[b, j]
            v[page, t % page_size] = vn[b, j]
    return k, v



def visible_range(length, num_queries, j, window):
    """Keys [lo, hi) that query j of ``num_queries`` sees in a sequence of
    ``length`` cached tokens (readings where the paper is silent):

    * the queries are the sequence's last ``num_queries`` tokens, so query j
      sits at position p = length - num_queries + j and sees keys t <= p
      (causal, as in a decode step or a chunk of prefill);
    * a sliding window of W > 0 tokens keeps keys p - W < t <= p (W keys
      counting the query's own token); W = 0 means no window.

    A query at a negative position (length < num_queries) sees nothing.
    """
    p = int(length) - int(num_queries) + int(j)
    hi = p + 1
    lo = max(0, hi - int(window)) if window > 0 else 0
    return lo, max(hi, lo)


def attend_masked(q, k_cache, v_cache, block_table, context_lens, scale, window=0):
    """Decode attention with several query tokens per sequence and an
    optional sliding window, in fp64.

    q: uint16 [B, Tq, Hq, D] (Tq query tokens per sequence, in position
    order); caches, block_table, context_lens, scale as for :func:`attend`.
    For sequence b, query j and head h (kv head g = h // G), the softmax runs
    over the keys of :func:`visible_range`; a query that sees no key gets a
    zero row (lse = -inf).  Returns (out float64 [B, Tq, Hq, D], lse [B, Tq, Hq]).
    """
    bsz, tq, hq, d = q.shape
    _, page_size, hkv, _ = k_cache.shape
    group = hq // hkv
    sigma = _sigma(scale)
    out = np.zeros((bsz, tq, hq, d))
    lse = np.full((bsz, tq, hq), -np.inf)
    for b in range(bsz):
        length = int(context_lens[b])
        for j in range(tq):
            lo, hi = visible_range(length, tq, j, window)
            if hi == lo:
                continue
            for g in range(hkv):
                kt = _gather(k_cache, block_table[b], hi, page_size, g, start=lo)
                vt = _gather(v_cache, block_table[b], hi, page_size, g, start=lo)
                qg = bf16_to_f64(q[b, j, g * group:(g + 1) * group, :])
                s = sigma * (qg @ kt.T)
                m = s.max(axis=1, keepdims=True)
                e = np.exp(s - m)
                den = e.sum(axis=1, keepdims=True)
                out[b, j, g * group:(g + 1) * group] = (e / den) @ vt
                lse[b, j, g * group:(g + 1) * group] = (m + np.log(den))[:, 0]
    return out, lse


def rms_norm(t, weight_bits, eps):
    """RMSNorm over the last axis: t / sqrt(mean(t^2) + eps) * w, in fp64
    (w: bf16 bits; eps: the fp32 value the kernel receives)."""
    t = np.asarray(t, dtype=np.float64)
    ms = np.mean(t * t, axis=-1, keepdims=True)
    return t / np.sqrt(ms + float(np.float32(eps))) * bf16_to_f64(weight_bits)


def rope(t, positions, theta, rotary_dim, interleaved=False):
    """Rotary position embedding of the last axis, in fp64.

    t: [B, H, D]; positions: [B].  Pair i < rotary_dim / 2 turns by the angle
    p * theta^(-2i / rotary_dim): the pair is (i, i + rotary_dim / 2) in the
    rotate-half convention, or (2i, 2i + 1) when ``interleaved``; dimensions
    at or beyond ``rotary_dim`` pass through.  (x_a, x_b) becomes
    (x_a cos - x_b sin, x_b cos + x_a sin).  ``theta`` is the fp32 value the
    kernel receives.
    """
    t = np.array(t, dtype=np.float64, copy=True)
    half = rotary_dim // 2
    base = float(np.float32(theta))
    for i in range(half):
        a, b = (2 * i, 2 * i + 1) if interleaved else (i, i + half)
        ang = np.asarray(positions, dtype=np.float64) * base ** (-2.0 * i / rotary_dim)
        c = np.cos(ang)[:, None]
        s_ = np.sin(ang)[:, None]
        xa, xb = t[..., a].copy(), t[..., b].copy()
        t[..., a] = xa * c - xb * s_
        t[..., b] = xb * c + xa * s_
    return t


def prelude(x, w_qkv, num_q_heads, num_kv_heads, head_dim, context_lens, theta, *, bias=None,
            q_norm=None, k_norm=None, eps=1e-6, rotary_dim=None, interleaved=False):
    """Attention prelude of one decode step, in fp64 (kernel family (i) of
    Method, "Principle-Driven LLM Kernel Generator").

    x: bf16 bits [B, H] (the normalised hidden state of the new token);
    w_qkv: bf16 bits [N, H] with N = (Hq + 2 Hkv) D, rows ordered q heads,
    then k heads, then v heads; bias: bf16 bits [N] or None; q_norm, k_norm:
    bf16 bits [D] or None (per-head RMSNorm weights, applied before the
    rotation).  The new token of sequence b sits at position
    max(context_lens[b] - 1, 0) (the length counts it).
    y = W x (+ bias); q, k, v are its head blocks; q and k are normalised
    (when weights are given) and rotated; v is left as is.
    Returns (q [B, Hq, D], k [B, Hkv, D], v [B, Hkv, D]) as float64.
    """
    hq, hkv, d = int(num_q_heads), int(num_kv_heads), int(head_dim)
    xf = bf16_to_f64(x)
    wf = bf16_to_f64(w_qkv)
    y = xf @ wf.T
    if bias is not None:
        y = y + bf16_to_f64(bias)[None, :]
    bsz = y.shape[0]
    q = y[:, :hq * d].reshape(bsz, hq, d)
    k = y[:, hq * d:(hq + hkv) * d].reshape(bsz, hkv, d)
    v = y[:, (hq + hkv) * d:].reshape(bsz, hkv, d)
    if q_norm is not None:
        q = rms_norm(q, q_norm, eps)
    if k_norm is not None:
        k = rms_norm(k, k_norm, eps)
    pos = np.maximum(np.asarray(context_lens, dtype=np.int64) - 1, 0)
    rd = d if rotary_dim is None else int(rotary_dim)
    q = rope(q, pos, theta, rd, interleaved)
    k = rope(k, pos, theta, rd, interleaved)
    return q, k, v.copy()


def o_proj_residual_norm(attn, w_o, residual, norm_w, eps):
    """Output projection + residual add + RMSNorm of one decode step, in fp64
    (kernel family (v) of Method, "Principle-Driven LLM Kernel Generator").

    attn: bf16 bits [B, K] (the attention output, heads concatenated);
    w_o: bf16 bits [H, K]; residual: bf16 bits [B, H]; norm_w: bf16 bits [H].
    z = W_o attn + residual is the new residual stream; h = RMSNorm(z) * w
    over the H features is the next sublayer's input (z not rounded first).
    Returns (z, h), float64 [B, H] each.
    """
    z = bf16_to_f64(attn) @ bf16_to_f64(w_o).T + bf16_to_f64(residual)
    return z, rms_norm(z, norm_w, eps)
