"""Seeded synthetic workloads for EG-MLA decode.

This module draws inputs and nothing else: it holds none of the method's
arithmetic, so both the fp64 oracle (``oracle/``) and the HIP path consume
exactly the same arrays.  Values are drawn in float32 with
``numpy.random.default_rng(seed)`` and, for bf16 storage, rounded to bf16 with
round-to-nearest-even; bf16 arrays are returned as their raw ``uint16`` bit
patterns.

Shapes follow the paper's model family (App. A hyper-parameter table: 1.2B
class = n_emb 2048, 128-dim heads, 64-dim decoupled RoPE key, kv_lora 128;
vocabulary 50304 as implied by the embedding-parameter counts) and a
128-head, d_c=512 layer for the paged stress case.  The paper's own
training/eval corpora are not available; these synthetic draws stand in for
them.

Draw order for one workload (fixed, so every consumer sees the same values):
seq_lens, page permutation, token ids, latents, RoPE keys, queries, W_UK,
W_UV, gate table.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass
from typing import Optional, Tuple

import numpy as np


# --------------------------------------------------------------------------
# bf16 storage helpers (data conversion only)
# --------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round-to-nearest-even) and return the bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


# --------------------------------------------------------------------------
# Workload description
# --------------------------------------------------------------------------
@dataclass(frozen=True)
class Workload:
    """One decode workload: layer shapes, cache layout, value recipe and seed."""

    name: str
    batch: int
    heads: int
    head_dim: int          # d_h: non-RoPE part of each query/key head
    v_head_dim: int        # d_v
    latent_dim: int        # d_c: cached latent width
    rope_dim: int          # d_r: decoupled RoPE key width, shared by all heads
    gate_dim: int          # width of a gate-table row (equals d_c: gate applied in latent space)
    vocab: int
    dtype: str             # "fp32" or "bf16" storage
    seq_len: Optional[int] = None                    # every sequence at this context
    seq_len_range: Optional[Tuple[int, int]] = None  # ragged: uniform in [lo, hi]
    page_size: int = 64
    paged: bool = False    # random page table (True) or contiguous per-sequence rows (False)
    seed: int = 0
    hidden: int = 2048     # model width, used by the append step
    recipe: str = "layer"  # "tiny": latents/queries ~ N(0, 1/sqrt(last dim)); "layer": N(0, 1)
    gate_all_ones: bool = False
    description: str = ""

    @property
    def qk_dim(self) -> int:
        return self.head_dim + self.rope_dim

    @property
    def row_dim(self) -> int:
        return self.latent_dim + self.rope_dim

    @property
    def max_seq_len(self) -> int:
        if self.seq_len is not None:
            return self.seq_len
        return self.seq_len_range[1]

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "fp32" else 2

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five decode workloads.  Index 0 is the tiny fp32 case, 1 is the
# ~1B-model layer at batch 32 / context 4096 (the throughput headline), 2 the
# long-context case, 3 the large-batch case, 4 the ragged paged 128-head case.
WORKLOADS = [
    Workload(name="tiny_fp32_b1_h4_dc32_l128", batch=1, heads=4, head_dim=32, v_head_dim=32,
             latent_dim=32, rope_dim=0, gate_dim=32, vocab=1000, dtype="fp32", seq_len=128,
             page_size=64, seed=0, hidden=128, recipe="tiny",
             description="tiny fp32 single decode step, no RoPE part"),
    Workload(name="layer1b_b32_h16_dc128_dr64_l4096", batch=32, heads=16, head_dim=128, v_head_dim=128,
             latent_dim=128, rope_dim=64, gate_dim=128, vocab=50304, dtype="bf16", seq_len=4096,
             seed=1, hidden=2048, description="~1B-model layer decode, batch 32, context 4096"),
    Workload(name="longctx_b4_h16_dc128_dr64_l32768", batch=4, heads=16, head_dim=128, v_head_dim=128,
             latent_dim=128, rope_dim=64, gate_dim=128, vocab=50304, dtype="bf16", seq_len=32768,
             seed=2, hidden=2048, description="long-context decode, batch 4, context 32768"),
    Workload(name="bigbatch_b256_h16_dc128_dr64_l2048", batch=256, heads=16, head_dim=128, v_head_dim=128,
             latent_dim=128, rope_dim=64, gate_dim=128, vocab=50304, dtype="bf16", seq_len=2048,
             seed=3, hidden=2048, description="large-batch decode, batch 256, context 2048"),
    Workload(name="paged_b64_h128_dc512_dr64_ragged", batch=64, heads=128, head_dim=128, v_head_dim=128,
             latent_dim=512, rope_dim=64, gate_dim=512, vocab=129280, dtype="bf16",
             seq_len_range=(512, 16384), page_size=64, paged=True, seed=4, hidden=7168,
             description="ragged paged stress, 64-token pages, random page table"),
]

# Plain-MLA comparison for the large-batch case: latent 320, all-ones gate.
MLA_DC320_BIGBATCH = WORKLOADS[3].replace(
    name="mla_bigbatch_b256_h16_dc320_dr64_l2048", latent_dim=320, gate_dim=320,
    gate_all_ones=True, description="plain MLA baseline (d_c=320, all-ones gate), batch 256, context 2048")


# --------------------------------------------------------------------------
# Generated inputs
# --------------------------------------------------------------------------
@dataclass
class DecodeInputs:
    """Host arrays for one decode call.  bf16 arrays hold uint16 bit patterns."""

    wl: Workload
    seq_lens: np.ndarray          # [B] int32, includes the current token
    page_table: Optional[np.ndarray]  # [B, max_pages] int32, or None for contiguous rows
    max_pages: int                # pages per sequence (capacity = max_pages * page_size)
    num_rows: int                 # rows in the cache (= pages * page_size)
    latent_cache: np.ndarray      # [num_rows, d_c + d_r]  (latent | RoPE key)
    token_ids: np.ndarray         # [num_rows] int32
    gate_table: np.ndarray        # [V, d_c]
    q: np.ndarray                 # [B, H, d_h + d_r]  (non-RoPE | RoPE, already rotated)
    w_uk: np.ndarray              # [H, d_h, d_c]
    w_uv: np.ndarray              # [H, d_v, d_c]

    def slot(self, b: int, j: int) -> int:
        """Cache row holding token j of sequence b."""
        P = self.wl.page_size
        if self.page_table is None:
            return b * self.max_pages * P + j
        return int(self.page_table[b, j // P]) * P + j % P

    def slots_of(self, b: int) -> np.ndarray:
        """Cache rows of every cached token of sequence b, in order."""
        P = self.wl.page_size
        j = np.arange(int(self.seq_lens[b]), dtype=np.int64)
        if self.page_table is None:
            return b * self.max_pages * P + j
        return self.page_table[b, j // P].astype(np.int64) * P + j % P

    def total_tokens(self) -> int:
        return int(self.seq_lens.astype(np.int64).sum())

    def unique_ids(self) -> int:
        """Distinct token ids over every cached token of the batch."""
        ids = np.concatenate([self.token_ids[self.slots_of(b)] for b in range(self.wl.batch)])
        return int(np.unique(ids).size)


def _store(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "fp32":
        return np.ascontiguousarray(x, dtype=np.float32)
    return f32_to_bf16_bits(x)


def generate(wl: Workload, seq_lens: Optional[np.ndarray] = None) -> DecodeInputs:
    """Draw every input of one decode call for workload ``wl``.

    ``seq_lens`` overrides the drawn lengths (used by edge-case tests); the
    rest of the draw order is unchanged.
    """
    rng = np.random.default_rng(wl.seed)
    B, H, P = wl.batch, wl.heads, wl.page_size
    # 1. lengths
    if wl.seq_len_range is not None:
        lo, hi = wl.seq_len_range
        drawn = rng.integers(lo, hi + 1, size=B).astype(np.int32)
    else:
        drawn = np.full(B, wl.seq_len, dtype=np.int32)
    if seq_lens is not None:
        drawn = np.asarray(seq_lens, dtype=np.int32).copy()
        assert drawn.shape == (B,)
    lens = drawn
    cap = max(int(lens.max()), 1)
    max_pages = (cap + P - 1) // P
    # 2. pages
    if wl.paged:
        npages = np.maximum((lens.astype(np.int64) + P - 1) // P, 0)
        total_pages = max(int(npages.sum()), 1)
        perm = rng.permutation(total_pages).astype(np.int32)
        page_table = np.zeros((B, max_pages), dtype=np.int32)
        off = 0
        for b in range(B):
            n = int(npages[b])
            page_table[b, :n] = perm[off:off + n]
            off += n
        num_rows = total_pages * P
    else:
        page_table = None
        num_rows = B * max_pages * P
    # 3.-9. values
    token_ids = rng.integers(0, wl.vocab, size=num_rows, dtype=np.int64).astype(np.int32)
    if wl.recipe == "tiny":
        lat_std = 1.0 / math.sqrt(wl.latent_dim)
        q_std = 1.0 / math.sqrt(wl.qk_dim)
        kr_std = 1.0 / math.sqrt(max(wl.rope_dim, 1))
    else:
        lat_std, q_std, kr_std = 1.0, 1.0, 1.0
    latent = rng.standard_normal((num_rows, wl.latent_dim), dtype=np.float32) * np.float32(lat_std)
    krope = rng.standard_normal((num_rows, wl.rope_dim), dtype=np.float32) * np.float32(kr_std)
    q = rng.standard_normal((B, H, wl.qk_dim), dtype=np.float32) * np.float32(q_std)
    w_std = np.float32(1.0 / math.sqrt(wl.latent_dim))
    w_uk = rng.standard_normal((H, wl.head_dim, wl.latent_dim), dtype=np.float32) * w_std
    w_uv = rng.standard_normal((H, wl.v_head_dim, wl.latent_dim), dtype=np.float32) * w_std
    if wl.gate_all_ones:
        gate = np.ones((wl.vocab, wl.gate_dim), dtype=np.float32)
    else:
        gate = np.float32(1.0) + np.float32(0.1) * rng.standard_normal((wl.vocab, wl.gate_dim), dtype=np.float32)
    cache = np.concatenate([latent, krope], axis=1)
    del latent, krope
    return DecodeInputs(
        wl=wl, seq_lens=lens, page_table=page_table, max_pages=max_pages, num_rows=num_rows,
        latent_cache=_store(cache, wl.dtype), token_ids=token_ids, gate_table=_store(gate, wl.dtype),
        q=_store(q, wl.dtype), w_uk=_store(w_uk, wl.dtype), w_uv=_store(w_uv, wl.dtype))


def generate_layer_group(wl: Workload, group_size: int, seq_lens: Optional[np.ndarray] = None) -> list:
    """One layer group of App. H: ``group_size`` layers decoding one shared cache.

    Layer 0 is ``generate(wl, seq_lens)``.  Layer k > 0 draws its own query,
    W_UK, W_UV and gate table from seed ``wl.seed + 7919 k`` and takes layer 0's
    lengths, page table, cache rows and token ids (the same arrays)."""
    base = generate(wl, seq_lens)
    layers = [base]
    for k in range(1, group_size):
        other = generate(wl.replace(seed=wl.seed + 7919 * k), seq_lens=base.seq_lens)
        layers.append(dataclasses.replace(other, seq_lens=base.seq_lens, page_table=base.page_table,
                                          max_pages=base.max_pages, num_rows=base.num_rows,
                                          latent_cache=base.latent_cache, token_ids=base.token_ids))
    return layers


@dataclass
class GateEmbedding:
    """Unfolded gate of Sec. 3.1 Eq. (3)-(4): an embedding table and W^UE.

    Component 0 of every embedding row is 1 and column 0 of W^UE is 1, so
    g = W^UE e = 1 + (a zero-mean term of std 0.1): the same statistics as the
    folded tables the decode workloads draw."""

    emb: np.ndarray    # [V, e]
    w_ue: np.ndarray   # [d_c, e]


def generate_gate_embedding(wl: Workload, emb_dim: int, seed: Optional[int] = None) -> GateEmbedding:
    """Seeded embedding table [V, emb_dim] ~ N(0, 1) and W^UE [d_c, emb_dim] ~ N(0, 0.1 / sqrt(emb_dim - 1))."""
    rng = np.random.default_rng(wl.seed + 2000 if seed is None else seed)
    emb = rng.standard_normal((wl.vocab, emb_dim), dtype=np.float32)
    emb[:, 0] = 1.0
    w_ue = rng.standard_normal((wl.latent_dim, emb_dim), dtype=np.float32) * np.float32(
        0.1 / math.sqrt(max(emb_dim - 1, 1)))
    w_ue[:, 0] = 1.0
    return GateEmbedding(emb=_store(emb, wl.dtype), w_ue=_store(w_ue, wl.dtype))


@dataclass
class LiteralGate:
    """Inputs of the paper-literal gate (Sec. 3.1 Eq. (2)-(5)): a full-width gate
    table and the LayerNorm's affine parameters, all head-major like kv^C =
    W^UKV c (per head: d_h key dims, then d_v value dims)."""

    gate_full: np.ndarray   # [V, H (d_h + d_v)]
    ln_w: np.ndarray        # [H (d_h + d_v)]
    ln_b: np.ndarray        # [H (d_h + d_v)]


def generate_literal_gate(wl: Workload, seed: Optional[int] = None, center: float = 1.0) -> LiteralGate:
    """Seeded gate rows center + 0.1 N(0, 1) (center 1 by default), LayerNorm weight
    1 + 0.1 N(0, 1) and bias 0.1 N(0, 1)."""
    rng = np.random.default_rng(wl.seed + 4000 if seed is None else seed)
    width = wl.heads * (wl.head_dim + wl.v_head_dim)
    g = np.float32(center) + np.float32(0.1) * rng.standard_normal((wl.vocab, width), dtype=np.float32)
    lw = np.float32(1.0) + np.float32(0.1) * rng.standard_normal(width, dtype=np.float32)
    lb = np.float32(0.1) * rng.standard_normal(width, dtype=np.float32)
    return LiteralGate(gate_full=_store(g, wl.dtype), ln_w=_store(lw, wl.dtype), ln_b=_store(lb, wl.dtype))


@dataclass
class AppendInputs:
    """Host arrays for one append call (new tokens written into a cache)."""

    wl: Workload
    x: np.ndarray            # [n, hidden]
    token_ids: np.ndarray    # [n] int32
    positions: np.ndarray    # [n] int32, 0-based position of each token in its sequence
    slots: np.ndarray        # [n] int32 destination cache rows (distinct)
    w_dkv: np.ndarray        # [d_c + d_r, hidden]
    kv_norm_w: Optional[np.ndarray]  # [d_c] or None
    num_rows: int            # rows of the destination cache
    rope_theta: float = 10000.0


def generate_append(wl: Workload, n_tokens: int, num_rows: int, with_norm: bool = True,
                    seed: Optional[int] = None) -> AppendInputs:
    """Draw one append step: hidden states, ids, positions and distinct destination slots."""
    rng = np.random.default_rng(wl.seed + 1000 if seed is None else seed)
    assert n_tokens <= num_rows
    x = rng.standard_normal((n_tokens, wl.hidden), dtype=np.float32)
    ids = rng.integers(0, wl.vocab, size=n_tokens, dtype=np.int64).astype(np.int32)
    positions = rng.integers(0, 32768, size=n_tokens, dtype=np.int64).astype(np.int32)
    slots = rng.permutation(num_rows)[:n_tokens].astype(np.int32)
    w = rng.standard_normal((wl.row_dim, wl.hidden), dtype=np.float32) * np.float32(1.0 / math.sqrt(wl.hidden))
    nw = (np.float32(1.0) + np.float32(0.1) * rng.standard_normal(wl.latent_dim, dtype=np.float32)) if with_norm else None
    return AppendInputs(wl=wl, x=_store(x, wl.dtype), token_ids=ids, positions=positions, slots=slots,
                        w_dkv=_store(w, wl.dtype), kv_norm_w=None if nw is None else _store(nw, wl.dtype),
                        num_rows=num_rows)


@dataclass
class PrefillInputs:
    """Host arrays for one causal prefill over T tokens of a single sequence."""

    wl: Workload
    q: np.ndarray          # [T, H, d_h + d_r]
    latent: np.ndarray     # [T, d_c + d_r]
    token_ids: np.ndarray  # [T] int32
    gate_table: np.ndarray
    w_uk: np.ndarray
    w_uv: np.ndarray


def generate_prefill(wl: Workload, seq_len: int, seed: Optional[int] = None) -> PrefillInputs:
    """Draw one single-sequence prefill of ``seq_len`` tokens with the workload's layer shapes."""
    rng = np.random.default_rng(wl.seed + 2000 if seed is None else seed)
    H = wl.heads
    ids = rng.integers(0, wl.vocab, size=seq_len, dtype=np.int64).astype(np.int32)
    if wl.recipe == "tiny":
        lat_std, q_std, kr_std = 1 / math.sqrt(wl.latent_dim), 1 / math.sqrt(wl.qk_dim), 1 / math.sqrt(max(wl.rope_dim, 1))
    else:
        lat_std, q_std, kr_std = 1.0, 1.0, 1.0
    lat = rng.standard_normal((seq_len, wl.latent_dim), dtype=np.float32) * np.float32(lat_std)
    kr = rng.standard_normal((seq_len, wl.rope_dim), dtype=np.float32) * np.float32(kr_std)
    q = rng.standard_normal((seq_len, H, wl.qk_dim), dtype=np.float32) * np.float32(q_std)
    w_std = np.float32(1.0 / math.sqrt(wl.latent_dim))
    w_uk = rng.standard_normal((H, wl.head_dim, wl.latent_dim), dtype=np.float32) * w_std
    w_uv = rng.standard_normal((H, wl.v_head_dim, wl.latent_dim), dtype=np.float32) * w_std
    if wl.gate_all_ones:
        gate = np.ones((wl.vocab, wl.gate_dim), dtype=np.float32)
    else:
        gate = np.float32(1.0) + np.float32(0.1) * rng.standard_normal((wl.vocab, wl.gate_dim), dtype=np.float32)
    return PrefillInputs(wl=wl, q=_store(q, wl.dtype), latent=_store(np.concatenate([lat, kr], 1), wl.dtype),
                         token_ids=ids, gate_table=_store(gate, wl.dtype), w_uk=_store(w_uk, wl.dtype),
                         w_uv=_store(w_uv, wl.dtype))


@dataclass
class PrefillBatch:
    """Host arrays for a causal prefill of several sequences packed back to back."""

    wl: Workload
    cu_seqlens: np.ndarray  # [B + 1] int32 offsets
    q: np.ndarray           # [T, H, d_h + d_r]
    latent: np.ndarray      # [T, d_c + d_r]
    token_ids: np.ndarray   # [T] int32
    gate_table: np.ndarray
    w_uk: np.ndarray
    w_uv: np.ndarray

    def sequence(self, b: int) -> PrefillInputs:
        """Sequence b alone, as a single-sequence prefill (views of the packed arrays)."""
        lo, hi = int(self.cu_seqlens[b]), int(self.cu_seqlens[b + 1])
        return PrefillInputs(wl=self.wl, q=self.q[lo:hi], latent=self.latent[lo:hi], token_ids=self.token_ids[lo:hi],
                             gate_table=self.gate_table, w_uk=self.w_uk, w_uv=self.w_uv)


def generate_prefill_batch(wl: Workload, seq_lens, seed: Optional[int] = None) -> PrefillBatch:
    """Sequences of the given lengths (zeros allowed) drawn as one prefill of their total, then split."""
    lens = np.asarray(seq_lens, dtype=np.int64)
    cu = np.zeros(len(lens) + 1, dtype=np.int32)
    cu[1:] = np.cumsum(lens)
    one = generate_prefill(wl, int(cu[-1]), seed=seed)
    return PrefillBatch(wl=wl, cu_seqlens=cu, q=one.q, latent=one.latent, token_ids=one.token_ids,
                        gate_table=one.gate_table, w_uk=one.w_uk, w_uv=one.w_uv)


def small_workload(base: Workload, **kw) -> Workload:
    """A reduced copy of ``base`` for parity tests that the oracle finishes in seconds."""
    return base.replace(**kw)
