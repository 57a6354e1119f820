"""Byte and flop accounting for EG-MLA decode.

* ``kv_cache_elements_per_token`` restates the per-token KV-cache element
  counts of the paper's Table 5 (Sec. 5.1): MHA 2 n_h d_h l, GQA 2 n_g d_h l,
  MQA 2 d_h l, MLA (d_c + d_h^R) l, EG-MLA (d_c/r + d_h^R) l.
* ``decode_bytes`` gives the algorithmic HBM bytes of one decode call: every
  cached latent+RoPE row and token id once, every *distinct* gate-table row
  once, and q, W_UK, W_UV and out once.  Repeated gate gathers and split-K
  partials are implementation overhead and are not counted.
* ``decode_flops`` counts the absorbed-form multiply-adds (2 flops each).
"""
from __future__ import annotations

from dataclasses import dataclass


def kv_cache_elements_per_token(mechanism: str, *, layers: int, heads: int = 0, head_dim: int = 0,
                                groups: int = 0, latent_dim: int = 0, rope_dim: int = 0,
                                compression: int = 1, layer_group: int = 1) -> int:
    """Per-token KV-cache elements summed over ``layers`` layers (Table 5).

    ``layer_group`` (App. H, lgz) applies to the latent mechanisms: the layers
    of a group share one cached row, so ``ceil(layers / lgz)`` rows are kept."""
    m = mechanism.lower()
    if layer_group != 1:
        assert layer_group >= 1 and m in ("mla", "eg-mla", "egmla", "eg_mla")
        rows = -(-layers // layer_group)
        return kv_cache_elements_per_token(m, layers=rows, latent_dim=latent_dim, rope_dim=rope_dim,
                                           compression=compression)
    if m == "mha":
        return 2 * heads * head_dim * layers
    if m == "gqa":
        return 2 * groups * head_dim * layers
    if m == "mqa":
        return 2 * head_dim * layers
    if m == "mla":
        return (latent_dim + rope_dim) * layers
    if m in ("eg-mla", "egmla", "eg_mla"):
        assert latent_dim % compression == 0
        return (latent_dim // compression + rope_dim) * layers
    raise ValueError(mechanism)


@dataclass
class DecodeTraffic:
    cache_rows: int      # latent + RoPE rows of every cached token
    token_ids: int
    gate_rows: int       # distinct gate-table rows
    q: int
    w_uk: int
    w_uv: int
    out: int

    @property
    def total(self) -> int:
        return self.cache_rows + self.token_ids + self.gate_rows + self.q + self.w_uk + self.w_uv + self.out

    @property
    def main_kernel(self) -> int:
        """Bytes the token-streaming kernel must move: cache rows, ids, distinct gate rows."""
        return self.cache_rows + self.token_ids + self.gate_rows

    @property
    def main_kernel_absorbing(self) -> int:
        """The same for a token-streaming kernel that also absorbs the query (reads q and W_UK once)."""
        return self.main_kernel + self.q + self.w_uk


def decode_bytes(*, batch: int, heads: int, head_dim: int, v_head_dim: int, latent_dim: int,
                 rope_dim: int, elem_bytes: int, total_tokens: int, distinct_ids: int) -> DecodeTraffic:
    """Algorithmic HBM bytes of one decode call."""
    e = elem_bytes
    return DecodeTraffic(
        cache_rows=total_tokens * (latent_dim + rope_dim) * e,
        token_ids=total_tokens * 4,
        gate_rows=distinct_ids * latent_dim * e,
        q=batch * heads * (head_dim + rope_dim) * e,
        w_uk=heads * head_dim * latent_dim * e,
        w_uv=heads * v_head_dim * latent_dim * e,
        out=batch * heads * v_head_dim * e,
    )


def decode_flops(*, batch: int, heads: int, head_dim: int, v_head_dim: int, latent_dim: int,
                 rope_dim: int, total_tokens: int) -> int:
    """Absorbed-form flops of one decode call (2 per multiply-add)."""
    per_token_head = (latent_dim + rope_dim) + latent_dim      # score dot + latent value accumulate
    absorb = batch * heads * head_dim * latent_dim
    up = batch * heads * v_head_dim * latent_dim
    gate = total_tokens * latent_dim // 2                      # one multiply per latent element
    return 2 * (total_tokens * heads * per_token_head + absorb + up + gate)


def cache_bytes_per_token(*, layers: int, latent_dim: int, rope_dim: int, elem_bytes: int,
                          layer_group: int = 1) -> int:
    """Bytes this library caches per token over ``layers`` layers: per cached
    row (one per group of ``layer_group`` layers, App. H) the latent and RoPE
    key in the storage type and one int32 token id (which Table 5 does not
    count)."""
    rows = -(-layers // layer_group)
    return rows * ((latent_dim + rope_dim) * elem_bytes + 4)
