"""Seeded synthetic inputs for paged decode attention.

This module only builds inputs: bf16 bit patterns for q and the paged K/V
pools, the per-sequence page tables and context lengths.  It holds none of
the attention arithmetic, so both the fp64 oracle and the GPU path can be fed
from it without sharing any of the method's code.

Storage conventions (the contract of the library's entry point):

* ``q``            uint16 bf16 bits, ``[B, Hq, D]`` contiguous.
* ``k_cache``      uint16 bf16 bits, ``[num_pages, P, Hkv, D]`` contiguous.
* ``v_cache``      same shape and layout as ``k_cache``.
* ``block_table``  int32 ``[B, max_pages]``; row ``b`` lists the physical pages
  of sequence ``b`` in token order.  Columns at or beyond ``ceil(L_b / P)`` are
  filled with -1 (never valid page ids).
* ``context_lens`` int32 ``[B]``; ``L_b`` counts every cached token of the
  sequence, including the one appended for the current decode step.

The paper's serving runtime keeps KV in fixed-size blocks of a shared pool
(Method, "Kernel Customization and Multi-Request Adaptation") and advances each
sequence length by one after the append (same section, the ``kv_append``
paragraph).  Page size, layout and distributions are not printed in the paper;
the five named workloads below are synthetic stand-ins shaped like the model
families it evaluates (Experiments, Setup).

Generation recipe, fixed for reproducibility: one ``numpy.random.Generator``
(PCG64) per workload; draw order lengths -> pool permutation -> q -> K -> V.
Normal deviates come from the inverse CDF of a uniform 16-bit draw: the draw
i indexes a 65536-entry table whose entry is the standard-normal quantile at
(i + 0.5) / 65536, times the requested standard deviation, rounded to bf16
with round-to-nearest-even.  This is a bf16 N(0, std^2) sample with tails cut
at about 4.2 std, and it is ~20x faster than float normals, which matters for
the multi-GB pools.
"""
from __future__ import annotations

import dataclasses
import functools
import math
import statistics
from typing import Dict, Optional, Sequence

import numpy as np

BF16_NAN = np.uint16(0x7FC0)
_CHUNK = 1 << 24  # values per draw call; part of the recipe (do not change)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round-to-nearest-even), return uint16 bits.

    Inputs here are finite normals; NaN/inf handling is not needed.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@functools.lru_cache(maxsize=8)
def _quantile_table(std: float) -> np.ndarray:
    nd = statistics.NormalDist(0.0, 1.0)
    z = np.array([nd.inv_cdf((i + 0.5) / 65536.0) for i in range(65536)], dtype=np.float64)
    return f32_to_bf16_bits((z * std).astype(np.float32))


def _normal_bf16(rng: np.random.Generator, shape, std: float = 1.0) -> np.ndarray:
    table = _quantile_table(float(std))
    n = int(np.prod(shape, dtype=np.int64))
    out = np.empty(n, dtype=np.uint16)
    for s in range(0, n, _CHUNK):
        e = min(n, s + _CHUNK)
        idx = rng.integers(0, 65536, size=e - s, dtype=np.uint16)
        np.take(table, idx, out=out[s:e])
    return out.reshape(shape)


@dataclasses.dataclass(frozen=True)
class Config:
    """One synthetic decode-attention workload."""

    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    seed: int
    lengths: str            # "fixed:<L>", "uniform:<lo>:<hi>", "zipf:<s>:<lo>:<hi>"
    pool: str               # "perm:<pool_pages>", "exact", "holes:<frac>"
    q_std: float = 1.0
    description: str = ""
    num_queries: int = 1    # query tokens per sequence (causal among them)
    window: int = 0         # sliding window in tokens, 0 = none

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads


CONFIGS: Dict[str, Config] = {
    "tiny": Config(
        "tiny", 1, 8, 2, 64, 16, 0, "fixed:256", "perm:64",
        description="batch 1, 8:2 heads (G=4), D=64, L=256, P=16, 16 pages "
                    "drawn from a shuffled pool of 64"),
    "llama8b": Config(
        "llama8b", 1, 32, 8, 128, 16, 1, "fixed:4096", "perm:4096",
        description="Llama-3-8B-shaped layer, batch 1, 32:8 heads, D=128, "
                    "L=4096, P=16, 256 pages scattered over a 4096-page pool"),
    "batched": Config(
        "batched", 64, 32, 8, 128, 16, 2, "uniform:128:8192", "exact",
        description="batch 64, 32:8 heads, D=128, L~U[128,8192], P=16, one "
                    "shuffled pool sized to the total tokens"),
    "long70b": Config(
        "long70b", 4, 64, 8, 128, 16, 3, "fixed:131072", "exact", q_std=0.5,
        description="70B-shaped long-context layer, batch 4, 64:8 heads (G=8), "
                    "D=128, L=131072, P=16, shuffled pool, q~N(0,0.5^2)"),
    "ragged": Config(
        "ragged", 256, 40, 8, 128, 32, 4, "zipf:1.2:16:32768", "holes:0.1",
        description="batch 256, 40:8 heads (G=5), D=128, L~Zipf(1.2) clipped "
                    "to [16,32768] and never a multiple of 32, P=32, shuffled "
                    "pool with 10% unused holes"),
    # variants of the same path (not among the five workloads above)
    "window": Config(
        "window", 64, 32, 8, 128, 16, 5, "fixed:16384", "exact", window=4096,
        description="Mistral-7B-shaped layer with a 4096-token sliding window, "
                    "batch 64, 32:8 heads, D=128, L=16384, P=16"),
    "multiq": Config(
        "multiq", 64, 32, 8, 128, 16, 6, "uniform:128:8192", "exact", num_queries=4,
        description="batch 64, 32:8 heads, D=128, L~U[128,8192], P=16, four "
                    "causal query tokens per sequence (G x 4 = 16 columns)"),
    "gqa16": Config(
        "gqa16", 32, 32, 2, 128, 16, 7, "fixed:32768", "exact",
        description="GLM-4-shaped 32:2 heads (G=16), batch 32, D=128, "
                    "L=32768, P=16"),
    "falcon3": Config(
        "falcon3", 16, 12, 4, 256, 16, 8, "uniform:16:32768", "exact",
        description="Falcon3-7B-shaped layer with head_dim 256, batch 16, 12:4 heads "
                    "(G=3), L~U[16,32768], P=16"),
    "tokenpage": Config(
        "tokenpage", 64, 32, 8, 128, 1, 9, "uniform:128:8192", "exact",
        description="batched with pages of one token (a token-granular cache), "
                    "batch 64, 32:8 heads, D=128, L~U[128,8192], P=1, shuffled pool"),
}
CONFIG_ORDER = ["tiny", "llama8b", "batched", "long70b", "ragged"]
VARIANT_ORDER = ["window", "multiq", "gqa16", "falcon3", "tokenpage"]


def window_start(length: int, num_queries: int, window: int) -> int:
    """First token any query of the sequence can see: with a window W > 0
    the earliest query (position L - Tq) sees keys from L - Tq + 1 - W on."""
    if window <= 0:
        return 0
    return max(0, int(length) - int(num_queries) + 1 - int(window))


@dataclasses.dataclass
class Workload:
    """Inputs of one paged decode-attention call (host numpy arrays)."""

    q: np.ndarray             # uint16 [B, Hq, D], or [B, Tq, Hq, D] with several query tokens
    k_cache: np.ndarray       # uint16 [N, P, Hkv, D]
    v_cache: np.ndarray       # uint16 [N, P, Hkv, D]
    block_table: np.ndarray   # int32 [B, maxp]
    context_lens: np.ndarray  # int32 [B]
    scale: np.float32
    name: str = "custom"
    window: int = 0           # sliding window in tokens, 0 = none

    @property
    def batch(self) -> int:
        return self.q.shape[0]

    @property
    def num_queries(self) -> int:
        return self.q.shape[1] if self.q.ndim == 4 else 1

    @property
    def num_q_heads(self) -> int:
        return self.q.shape[-2]

    @property
    def head_dim(self) -> int:
        return self.q.shape[-1]

    @property
    def num_kv_heads(self) -> int:
        return self.k_cache.shape[2]

    @property
    def page_size(self) -> int:
        return self.k_cache.shape[1]

    @property
    def num_pages(self) -> int:
        return self.k_cache.shape[0]

    @property
    def max_pages(self) -> int:
        return self.block_table.shape[1]

    def algorithmic_bytes(self) -> int:
        """Bytes the operation must move at minimum: each K and V element
        that some query sees once (shared by the GQA group and the query
        tokens), q in, out out, the page ids of those tokens and the lengths."""
        lens = self.context_lens.astype(np.int64)
        d, hkv, hq, b = self.head_dim, self.num_kv_heads, self.num_q_heads, self.batch
        p, tq = self.page_size, self.num_queries
        start = np.array([window_start(x, tq, self.window) for x in lens], dtype=np.int64)
        live = np.maximum(lens - start, 0)
        pages = int(np.sum(np.where(lens > 0, (lens + p - 1) // p - start // p, 0)))
        return int(4 * d * hkv * int(live.sum()) + 2 * 2 * b * tq * hq * d + 4 * pages + 4 * b)


def _draw_lengths(cfg: Config, rng: np.random.Generator) -> np.ndarray:
    kind, *args = cfg.lengths.split(":")
    if kind == "fixed":
        return np.full(cfg.batch, int(args[0]), dtype=np.int64)
    if kind == "uniform":
        lo, hi = int(args[0]), int(args[1])
        return rng.integers(lo, hi + 1, size=cfg.batch, dtype=np.int64)
    if kind == "zipf":
        s, lo, hi = float(args[0]), int(args[1]), int(args[2])
        lens = np.clip(rng.zipf(s, size=cfg.batch).astype(np.int64), lo, hi)
        # every sequence ends in a partly filled page
        lens = np.where(lens % cfg.page_size == 0, lens - 1, lens)
        return lens
    raise ValueError(f"unknown length spec {cfg.lengths!r}")


def build(
    lengths: Sequence[int],
    num_q_heads: int,
    num_kv_heads: int,
    head_dim: int,
    page_size: int,
    seed: int,
    *,
    pool: str = "exact",
    q_std: float = 1.0,
    scale: Optional[float] = None,
    poison: bool = True,
    max_pages: Optional[int] = None,
    name: str = "custom",
    rng: Optional[np.random.Generator] = None,
    num_queries: int = 1,
    window: int = 0,
) -> Workload:
    """Build a workload for explicit lengths.

    ``pool``: ``"exact"`` (pool = pages needed, shuffled), ``"perm:<N>"``
    (pool of N pages, the used ones drawn by a random permutation) or
    ``"holes:<f>"`` (pool = ceil(needed / (1-f)), pages handed out in
    sequence order from a random permutation, the rest unused).
    With ``poison`` every pool slot that no live token uses (unused pages
    and the tail slots of each last page) holds bf16 NaN.

    ``num_queries`` > 1 makes q ``[B, Tq, Hq, D]``.  With a sliding
    ``window`` and ``poison``, pages that lie wholly before the first token
    any query sees are released: their page-table entries become -1 and,
    unless another sequence uses them, their contents NaN (a serving engine
    may hand such pages to other requests).
    """
    if rng is None:
        rng = np.random.Generator(np.random.PCG64(seed))
    lens = np.asarray(lengths, dtype=np.int64)
    b = lens.shape[0]
    if num_q_heads % num_kv_heads:
        raise ValueError("num_q_heads must be a multiple of num_kv_heads")
    npages = (lens + page_size - 1) // page_size
    need = int(npages.sum())
    kind, *args = pool.split(":")
    if kind == "exact":
        n_pool = max(need, 1)
    elif kind == "perm":
        n_pool = int(args[0])
    elif kind == "holes":
        n_pool = max(int(math.ceil(need / (1.0 - float(args[0])))), 1)
    else:
        raise ValueError(f"unknown pool spec {pool!r}")
    if n_pool < need:
        raise ValueError("pool smaller than the pages needed")
    perm = rng.permutation(n_pool).astype(np.int64)
    maxp = int(npages.max()) if b else 0
    if max_pages is not None:
        if max_pages < maxp:
            raise ValueError("max_pages below the longest sequence")
        maxp = max_pages
    maxp = max(maxp, 1)
    bt = np.full((b, maxp), -1, dtype=np.int32)
    cursor = 0
    for i in range(b):
        bt[i, : npages[i]] = perm[cursor: cursor + npages[i]]
        cursor += int(npages[i])
    qshape = (b, num_q_heads, head_dim) if num_queries == 1 else (b, num_queries, num_q_heads, head_dim)
    q = _normal_bf16(rng, qshape, q_std)
    k = _normal_bf16(rng, (n_pool, page_size, num_kv_heads, head_dim))
    v = _normal_bf16(rng, (n_pool, page_size, num_kv_heads, head_dim))
    if poison:
        if window > 0:
            for i in range(b):
                first = window_start(int(lens[i]), num_queries, window) // page_size
                bt[i, :first] = -1
        used = np.zeros(n_pool, dtype=bool)
        for i in range(b):
            row = bt[i, : npages[i]]
            used[row[row >= 0]] = True
            tail = int(lens[i] % page_size)
            if tail:
                last = bt[i, npages[i] - 1]
                k[last, tail:] = BF16_NAN
                v[last, tail:] = BF16_NAN
        k[~used] = BF16_NAN
        v[~used] = BF16_NAN
    if scale is None:
        scale = 1.0 / math.sqrt(head_dim)
    return Workload(q=q, k_cache=k, v_cache=v, block_table=bt,
                    context_lens=lens.astype(np.int32), scale=np.float32(scale), name=name,
                    window=int(window))


def make(name: str, *, poison: bool = True, seed: Optional[int] = None) -> Workload:
    """Build one of the five named workloads with its fixed seed."""
    cfg = CONFIGS[name]
    rng = np.random.Generator(np.random.PCG64(cfg.seed if seed is None else seed))
    lens = _draw_lengths(cfg, rng)
    return build(lens, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, cfg.page_size,
                 cfg.seed, pool=cfg.pool, q_std=cfg.q_std, poison=poison, name=name, rng=rng,
                 num_queries=cfg.num_queries, window=cfg.window)


def lengths_of(name: str, seed: Optional[int] = None) -> np.ndarray:
    """The context lengths a named workload draws (cheap: no KV generated)."""
    cfg = CONFIGS[name]
    rng = np.random.Generator(np.random.PCG64(cfg.seed if seed is None else seed))
    return _draw_lengths(cfg, rng)


def permute_pages(w: Workload, seed: int) -> Workload:
    """Move every physical page to a new slot of the pool and remap the page
    table accordingly.  The logical KV of every sequence is unchanged."""
    rng = np.random.Generator(np.random.PCG64(seed))
    n = w.num_pages
    new_of_old = rng.permutation(n)
    k = np.empty_like(w.k_cache)
    v = np.empty_like(w.v_cache)
    k[new_of_old] = w.k_cache
    v[new_of_old] = w.v_cache
    bt = w.block_table.copy()
    live = bt >= 0
    bt[live] = new_of_old[bt[live]].astype(np.int32)
    return dataclasses.replace(w, k_cache=k, v_cache=v, block_table=bt)



# ------------------------------------------------------------------ prelude
@dataclasses.dataclass(frozen=True)
class PreludeConfig:
    """One synthetic attention-prelude workload (QKV projection + RoPE)."""

    name: str
    batch: int
    hidden: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    seed: int
    lengths: str                 # as for Config: the new token sits at L - 1
    theta: float
    qk_norm: bool = False
    bias: bool = False
    rotary_dim: Optional[int] = None   # None = head_dim, 0 = no rotation
    interleaved: bool = False
    description: str = ""


PRELUDE_CONFIGS: Dict[str, PreludeConfig] = {
    "prelude_qwen3_4b": PreludeConfig(
        "prelude_qwen3_4b", 1, 2560, 32, 8, 128, 10, "fixed:4096", 1.0e6, qk_norm=True,
        description="Qwen3-4B-shaped prelude, batch 1, hidden 2560, 32:8 heads, D=128, "
                    "per-head Q/K RMSNorm, theta 1e6"),
    "prelude_llama8b": PreludeConfig(
        "prelude_llama8b", 64, 4096, 32, 8, 128, 11, "uniform:128:8192", 5.0e5,
        description="Llama-3-8B-shaped prelude, batch 64, hidden 4096, 32:8 heads, D=128, "
                    "theta 5e5"),
    "prelude_70b": PreludeConfig(
        "prelude_70b", 4, 8192, 64, 8, 128, 12, "fixed:131072", 5.0e5,
        description="70B-shaped prelude, batch 4, hidden 8192, 64:8 heads, D=128, theta 5e5, "
                    "positions 131071"),
    "prelude_glm4": PreludeConfig(
        "prelude_glm4", 8, 4096, 32, 2, 128, 13, "uniform:16:32768", 1.0e4, bias=True,
        rotary_dim=64, interleaved=True,
        description="GLM-4-9B-shaped prelude, batch 8, hidden 4096, 32:2 heads, D=128, QKV "
                    "bias, rotary on the first 64 dims in interleaved pairs, theta 1e4"),
    "prelude_falcon3": PreludeConfig(
        "prelude_falcon3", 16, 3072, 12, 4, 256, 14, "uniform:16:32768", 1000042.0,
        description="Falcon3-7B-shaped prelude, batch 16, hidden 3072, 12:4 heads, D=256, "
                    "theta 1000042"),
    "prelude_ragged": PreludeConfig(
        "prelude_ragged", 256, 5120, 40, 8, 128, 15, "zipf:1.2:16:32768", 1.0e6,
        description="prelude of the ragged serving batch, batch 256, hidden 5120, 40:8 heads, "
                    "D=128, positions Zipf(1.2) in [16, 32768], theta 1e6"),
}


@dataclasses.dataclass
class PreludeWorkload:
    """Inputs of one attention-prelude call (host numpy arrays, bf16 bits)."""

    x: np.ndarray                 # [B, H]
    w_qkv: np.ndarray             # [(Hq + 2 Hkv) D, H], rows: q heads, k heads, v heads
    bias: Optional[np.ndarray]    # [N] or None
    q_norm: Optional[np.ndarray]  # [D] or None
    k_norm: Optional[np.ndarray]  # [D] or None
    context_lens: np.ndarray      # int32 [B]; the new token sits at L - 1
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    theta: np.float32
    eps: np.float32
    rotary_dim: int
    interleaved: bool
    name: str = "custom"

    @property
    def batch(self) -> int:
        return self.x.shape[0]

    @property
    def hidden(self) -> int:
        return self.x.shape[1]

    @property
    def rows(self) -> int:
        return self.w_qkv.shape[0]

    def algorithmic_bytes(self) -> int:
        """Weights once, x in, q/k/v out, bias and norm weights, lengths."""
        n, h, b = self.rows, self.hidden, self.batch
        extra = (2 * n if self.bias is not None else 0) + 2 * self.head_dim * (
            (self.q_norm is not None) + (self.k_norm is not None))
        return int(2 * n * h + 2 * b * h + 2 * b * n + extra + 4 * b)


def build_prelude(batch, hidden, num_q_heads, num_kv_heads, head_dim, seed, *, lengths=None,
                  theta=1.0e4, qk_norm=False, bias=False, rotary_dim=None, interleaved=False,
                  eps=1e-6, name="custom", rng=None) -> PreludeWorkload:
    """Seeded prelude inputs.  Draw order: lengths (by the caller), x, W,
    bias, q_norm, k_norm.  x ~ N(0, 1) (a normalised hidden state); W ~
    N(0, 1/hidden) so that q, k, v are O(1); bias ~ N(0, 0.1^2); norm
    weights ~ 1 + N(0, 0.1^2).  ``rotary_dim`` None means the whole head,
    0 no rotation."""
    if rng is None:
        rng = np.random.Generator(np.random.PCG64(seed))
    n = (num_q_heads + 2 * num_kv_heads) * head_dim
    if lengths is None:
        lengths = np.full(batch, 1, dtype=np.int64)
    x = _normal_bf16(rng, (batch, hidden), 1.0)
    w = _normal_bf16(rng, (n, hidden), 1.0 / math.sqrt(hidden))
    bvec = _normal_bf16(rng, (n,), 0.1) if bias else None
    qn = kn = None
    if qk_norm:
        one = bf16_bits_to_f32(_normal_bf16(rng, (2, head_dim), 0.1)) + np.float32(1.0)
        qn, kn = f32_to_bf16_bits(one[0]), f32_to_bf16_bits(one[1])
    return PreludeWorkload(x=x, w_qkv=w, bias=bvec, q_norm=qn, k_norm=kn,
                           context_lens=np.asarray(lengths, dtype=np.int32), num_q_heads=num_q_heads,
                           num_kv_heads=num_kv_heads, head_dim=head_dim, theta=np.float32(theta),
                           eps=np.float32(eps), rotary_dim=head_dim if rotary_dim is None else int(rotary_dim),
                           interleaved=bool(interleaved), name=name)


def make_prelude(name: str, seed: Optional[int] = None) -> PreludeWorkload:
    """Build one of the named prelude workloads with its fixed seed."""
    cfg = PRELUDE_CONFIGS[name]
    rng = np.random.Generator(np.random.PCG64(cfg.seed if seed is None else seed))
    shim = Config(cfg.name, cfg.batch, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, 16, cfg.seed,
                  cfg.lengths, "exact")
    lens = _draw_lengths(shim, rng)
    return build_prelude(cfg.batch, cfg.hidden, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, cfg.seed,
                         lengths=lens, theta=cfg.theta, qk_norm=cfg.qk_norm, bias=cfg.bias,
                         rotary_dim=cfg.rotary_dim, interleaved=cfg.interleaved, name=name, rng=rng)



# ------------------------------------------------------------------ o_proj
@dataclasses.dataclass(frozen=True)
class OProjConfig:
    """One synthetic output-projection workload (o_proj + residual + RMSNorm)."""

    name: str
    batch: int
    in_features: int   # Hq * D
    hidden: int
    seed: int
    description: str = ""


OPROJ_CONFIGS: Dict[str, OProjConfig] = {
    "oproj_qwen3_4b": OProjConfig("oproj_qwen3_4b", 1, 4096, 2560, 20,
                                  "Qwen3-4B-shaped o_proj, batch 1, 32 x 128 -> 2560"),
    "oproj_llama8b": OProjConfig("oproj_llama8b", 64, 4096, 4096, 21,
                                 "Llama-3-8B-shaped o_proj, batch 64, 4096 -> 4096"),
    "oproj_70b": OProjConfig("oproj_70b", 4, 8192, 8192, 22, "70B-shaped o_proj, batch 4, 8192 -> 8192"),
    "oproj_falcon3": OProjConfig("oproj_falcon3", 16, 3072, 3072, 23,
                                 "Falcon3-7B-shaped o_proj, batch 16, 12 x 256 -> 3072"),
    "oproj_ragged": OProjConfig("oproj_ragged", 256, 5120, 5120, 24,
                                "o_proj of the ragged serving batch, batch 256, 40 x 128 -> 5120"),
}


@dataclasses.dataclass
class OProjWorkload:
    """Inputs of one o_proj + residual + RMSNorm call (host bf16 bits)."""

    attn: np.ndarray      # [B, K]
    w_o: np.ndarray       # [H, K]
    residual: np.ndarray  # [B, H]
    norm_w: np.ndarray    # [H]
    eps: np.float32
    name: str = "custom"

    @property
    def batch(self) -> int:
        return self.attn.shape[0]

    @property
    def in_features(self) -> int:
        return self.attn.shape[1]

    @property
    def hidden(self) -> int:
        return self.w_o.shape[0]

    def algorithmic_bytes(self) -> int:
        """Weights once, attention output and residual in, residual and
        normed outputs out, the norm weights."""
        b, k, h = self.batch, self.in_features, self.hidden
        return int(2 * h * k + 2 * b * k + 2 * b * h * 3 + 2 * h)


def build_oproj(batch, in_features, hidden, seed, *, eps=1e-5, name="custom", rng=None) -> OProjWorkload:
    """Seeded o_proj inputs.  Draw order: attn, W_o, residual, norm weights.
    attn ~ N(0, 1); W_o ~ N(0, 1/K); residual ~ N(0, 1); weights ~ 1 + N(0, 0.1^2)."""
    if rng is None:
        rng = np.random.Generator(np.random.PCG64(seed))
    attn = _normal_bf16(rng, (batch, in_features), 1.0)
    w = _normal_bf16(rng, (hidden, in_features), 1.0 / math.sqrt(in_features))
    res = _normal_bf16(rng, (batch, hidden), 1.0)
    nw = f32_to_bf16_bits(bf16_bits_to_f32(_normal_bf16(rng, (hidden,), 0.1)) + np.float32(1.0))
    return OProjWorkload(attn=attn, w_o=w, residual=res, norm_w=nw, eps=np.float32(eps), name=name)


def make_oproj(name: str, seed: Optional[int] = None) -> OProjWorkload:
    cfg = OPROJ_CONFIGS[name]
    return build_oproj(cfg.batch, cfg.in_features, cfg.hidden, cfg.seed if seed is None else seed, name=name)
