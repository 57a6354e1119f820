"""fp64 CPU oracle for EG-MLA decode, prefill and append.

TEST INFRASTRUCTURE ONLY.  Only the tests, the package's ``smoke()`` check and
the benchmark's CPU-baseline leg may import this module.  It shares no code
with the HIP path: it widens the stored values itself, computes everything in
float64 with NumPy, and is written to be read against the paper, not to be
fast.

What it computes (EG-MLA, arXiv 2509.16686):

* Latent KV compression, Sec. 3.1 Eq. (1): c_t = W^DKV x_t, plus the decoupled
  RoPE key k^R_t = RoPE(W^KR x_t) of App. C Eq. (C.10), one d_r vector shared
  by all heads.
* Embedding gate, Sec. 3.1 Eq. (3)-(5): e_t = Emb(i_t), g_t = W^UE e_t, applied
  by a Hadamard product (``gate_rows`` computes g for given ids; over the
  whole vocabulary it is the folded table G).  Reading taken here (the paper places the gate in
  the latent space in its abstract, related-work and Sec. 5 text, but after
  the up-projection in Eq. (5) and its listing): the gate multiplies the
  cached latent, c~_t = c_t * G[i_t], where G = Emb W^UE^T is the gate table
  folded offline (the EG-MLA-A variant of Sec. 5.2).  No LayerNorm follows in
  this reading, so an all-ones gate gives back plain MLA.
* Attention, App. C Eq. (C.2), (C.6), (C.11)-(C.13): per head i,
  k_{j,i} = [W_UK[i] c~_j ; k^R_j], v_{j,i} = W_UV[i] c~_j, and
  u_{t,i} = sum_j softmax_j(q_{t,i} . k_{j,i} / sqrt(d_h + d_r)) v_{j,i}.
  The RoPE key is not gated (it is concatenated after gating).
* Absorbed decode: q_lat = W_UK[i]^T q^C, scores q_lat . c~_j + q^R . k^R_j,
  value aggregation in latent space and one W_UV[i] at the end.  This equals
  the explicit form by associativity of the matrix products.

* The paper-literal gate (``literal_kv``, ``decode_literal``): Eq. (2)-(5) as
  printed and the model listing's order, kv^C = W^UKV c, x = kv^C * g (or
  kv^C + g, the ablation), LN over all heads' H (d_h + d_v) dims (or none, the
  other ablation), then attention with the listing's per-head key/value split.

Functions that follow an algorithm step by step rather than a closed
definition: ``append`` (projection, optional RMSNorm, RoPE).  Its RoPE pairing
(adjacent pairs, base 10000, 0-based positions) and RMSNorm epsilon (1e-6)
are readings; the paper does not define them.  ``append`` is pinned only
through closed forms (rotation preserves pair norms, position 0 is the
identity, norm scaling), so its exact RoPE convention is parity unpinned
against the paper.
"""
from __future__ import annotations

import math
from typing import Optional

import numpy as np

RMS_EPS = 1e-6
ROPE_BASE = 10000.0


# ---------------------------------------------------------------------------
# storage -> float64 (exact widening; bf16 arrives as uint16 bit patterns)
# ---------------------------------------------------------------------------
def widen(a: np.ndarray, storage: str) -> np.ndarray:
    """Exact float64 value of a stored array.

    ``storage`` is "fp32" (float32 values), "bf16" (uint16 bit patterns) or
    "f64" (already float64; used by invariant tests that feed exact products).
    """
    if storage == "f64":
        return np.asarray(a, dtype=np.float64)
    if storage == "fp32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    if storage == "bf16":
        bits = np.asarray(a, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    raise ValueError(f"unknown storage {storage!r}")


def softmax_scale(head_dim: int, rope_dim: int) -> float:
    """App. C Eq. (C.13): logits are divided by sqrt(d_h + d_h^R)."""
    return 1.0 / math.sqrt(head_dim + rope_dim)


def cache_rows(seq_len: int, b: int, page_table: Optional[np.ndarray], page_size: int,
               max_pages: int) -> np.ndarray:
    """Rows of the cache holding tokens 0..seq_len-1 of sequence b.

    Paged: token j lives in page page_table[b, j // P] at offset j % P.
    Contiguous (no page table): sequence b owns rows b*max_pages*P ... .
    """
    j = np.arange(seq_len, dtype=np.int64)
    if page_table is None:
        return b * max_pages * page_size + j
    return np.asarray(page_table, dtype=np.int64)[b, j // page_size] * page_size + j % page_size


def _softmax(s: np.ndarray) -> np.ndarray:
    """Softmax over the last axis (max-subtracted; exact up to rounding)."""
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=-1, keepdims=True)


# ---------------------------------------------------------------------------
# gate rows from the token embedding (Sec. 3.1 Eq. (3)-(4))
# ---------------------------------------------------------------------------
def gate_rows(emb, w_ue, ids, *, storage: str) -> np.ndarray:
    """g_i = W^UE e_i with e_i = Emb[ids[i]]; returns [n, d_c] in float64.

    emb [V_e, e], w_ue [d_c, e] ([out, in] like every weight here), ids [n]
    (clamped into [0, V_e) as the library does).  Over ids 0..V-1 this is the
    folded gate table G = Emb W^UE^T of the table-lookup variant (Sec. 5.2).
    """
    ef = widen(emb, storage)
    wf = widen(w_ue, storage)
    idx = np.clip(np.asarray(ids, dtype=np.int64), 0, ef.shape[0] - 1)
    return ef[idx] @ wf.T                                    # row i: W^UE e_{ids[i]}


# ---------------------------------------------------------------------------
# decode (one query row per sequence over its whole cached context)
# ---------------------------------------------------------------------------
def decode(q, cache, token_ids, gate_table, w_uk, w_uv, seq_lens, *, latent_dim: int,
           head_dim: int, rope_dim: int, storage: str, page_table=None, page_size: int = 64,
           max_pages: int = 0, scale: Optional[float] = None, use_gate: bool = True) -> np.ndarray:
    """Absorbed-form EG-MLA decode; returns out [B, H, d_v] in float64.

    Shapes: q [B,H,d_h+d_r] (q^R already rotated), cache [rows, d_c+d_r],
    token_ids [rows], gate_table [V, d_c], w_uk [H,d_h,d_c], w_uv [H,d_v,d_c],
    seq_lens [B] (the current token included).  A sequence of length 0 gives
    zeros.  ``use_gate=False`` skips the Hadamard product (plain MLA).
    """
    qf = widen(q, storage)
    cf = widen(cache, storage)
    gf = widen(gate_table, storage)
    wk = widen(w_uk, storage)
    wv = widen(w_uv, storage)
    B, H, _ = qf.shape
    d_c, d_h, d_r = latent_dim, head_dim, rope_dim
    tau = softmax_scale(d_h, d_r) if scale is None else scale
    out = np.zeros((B, H, wv.shape[1]), dtype=np.float64)
    for b in range(B):
        L = int(seq_lens[b])
        if L == 0:
            continue
        rows = cache_rows(L, b, page_table, page_size, max_pages)
        c = cf[rows, :d_c]                                   # latent c_j
        k_r = cf[rows, d_c:d_c + d_r]                        # RoPE key k^R_j (not gated)
        g = gf[np.asarray(token_ids)[rows].astype(np.int64)]  # gate row G[i_j]
        c_g = c * g if use_gate else c                       # Eq. (5), latent reading
        q_c = qf[b, :, :d_h]
        q_r = qf[b, :, d_h:d_h + d_r]
        q_lat = np.einsum("hk,hkc->hc", q_c, wk)             # W_UK[h]^T q^C  (absorption)
        s = tau * (q_lat @ c_g.T + q_r @ k_r.T)              # [H, L], Eq. (C.11)-(C.13)
        p = _softmax(s)
        o_lat = p @ c_g                                      # value aggregation in latent space
        out[b] = np.einsum("hvc,hc->hv", wv, o_lat)          # W_UV[h] o_lat
    return out


def decode_explicit(q, cache, token_ids, gate_table, w_uk, w_uv, seq_lens, *, latent_dim: int,
                    head_dim: int, rope_dim: int, storage: str, page_table=None, page_size: int = 64,
                    max_pages: int = 0, scale: Optional[float] = None) -> np.ndarray:
    """Same result as ``decode`` through the explicit per-head keys and values of App. C."""
    qf = widen(q, storage)
    cf = widen(cache, storage)
    gf = widen(gate_table, storage)
    wk = widen(w_uk, storage)
    wv = widen(w_uv, storage)
    B, H, _ = qf.shape
    d_c, d_h, d_r = latent_dim, head_dim, rope_dim
    tau = softmax_scale(d_h, d_r) if scale is None else scale
    out = np.zeros((B, H, wv.shape[1]), dtype=np.float64)
    for b in range(B):
        L = int(seq_lens[b])
        if L == 0:
            continue
        rows = cache_rows(L, b, page_table, page_size, max_pages)
        c_g = cf[rows, :d_c] * gf[np.asarray(token_ids)[rows].astype(np.int64)]
        k_r = cf[rows, d_c:d_c + d_r]
        for h in range(H):
            k_c = c_g @ wk[h].T                              # k^C_{j,h} = W_UK[h] c~_j   [L, d_h]
            v_c = c_g @ wv[h].T                              # v^C_{j,h} = W_UV[h] c~_j   [L, d_v]
            k = np.concatenate([k_c, k_r], axis=1)           # Eq. (C.12)
            s = tau * (k @ qf[b, h, :d_h + d_r])             # Eq. (C.13) logits
            out[b, h] = _softmax(s) @ v_c
    return out


def decode_layer_group(cache, token_ids, seq_lens, layers, *, latent_dim: int, head_dim: int, rope_dim: int,
                       storage: str, page_table=None, page_size: int = 64, max_pages: int = 0) -> list:
    """Layer grouping of App. H (lgz consecutive layers share the first half of the
    KV projection and its activations), decoded: the group caches one
    [c | k^R] row and one token id per token, written by its first layer, and
    every layer of the group decodes those rows with its own query, W_UK, W_UV
    and gate table.  ``layers`` holds (q, gate_table, w_uk, w_uv) per layer;
    returns each layer's out [B, H, d_v], the same as ``decode`` of that layer
    over the shared rows."""
    return [decode(q, cache, token_ids, gate, w_uk, w_uv, seq_lens, latent_dim=latent_dim, head_dim=head_dim,
                   rope_dim=rope_dim, storage=storage, page_table=page_table, page_size=page_size,
                   max_pages=max_pages) for (q, gate, w_uk, w_uv) in layers]


# ---------------------------------------------------------------------------
# the paper-literal gate (Sec. 3.1 Eq. (2)-(5) as printed, and the model
# listing of App. E): the gate multiplies the up-projected keys and values of
# every head, and a LayerNorm spans all heads' dims
# ---------------------------------------------------------------------------
LN_EPS = 1e-5  # the listing's nn.LayerNorm default


def literal_kv(cache_rows_c, token_ids, gate_full, w_uk, w_uv, ln_w, ln_b, *, mode: str = "mul",
               use_ln: bool = True) -> np.ndarray:
    """Gated, normalised up-projected rows [n, H (d_h + d_v)] (float64 inputs).

    Eq. (2): kv^C_t = W^UKV c_t, whose per-head blocks are [W_UK[h] c_t ; W_UV[h] c_t]
    (the listing views kv as [n_h, d_nope + d_v] and splits each head into key
    and value parts).  Eq. (3)-(5): x_t = kv^C_t (.) g_t with g_t = G[i_t] (the
    full-width gate row; mode "add" is the ablation's kv^C_t + g_t), then
    kv~_t = LN(x_t) over all H (d_h + d_v) dims with weight ln_w and bias ln_b
    (use_ln False is the other ablation).
    """
    H = w_uk.shape[0]
    kv = np.concatenate([np.concatenate([cache_rows_c @ w_uk[h].T, cache_rows_c @ w_uv[h].T], axis=1)
                         for h in range(H)], axis=1)
    g = gate_full[np.asarray(token_ids).astype(np.int64)]
    x = kv * g if mode == "mul" else kv + g
    if not use_ln:
        return x
    mu = x.mean(axis=1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=1, keepdims=True)
    return (x - mu) / np.sqrt(var + LN_EPS) * ln_w + ln_b


def decode_literal(q, cache, token_ids, gate_full, w_uk, w_uv, ln_w, ln_b, seq_lens, *, latent_dim: int,
                   head_dim: int, rope_dim: int, storage: str, page_table=None, page_size: int = 64,
                   max_pages: int = 0, mode: str = "mul", use_ln: bool = True) -> np.ndarray:
    """Decode with the paper-literal gate; returns out [B, H, d_v] in float64.

    Per head h: k_j = [kv~_j[h, :d_h] ; k^R_j], v_j = kv~_j[h, d_h:] (App. C
    Eq. (C.11)-(C.13) with the listing's split), u = softmax(q . k / sqrt(d_h + d_r)) v.
    gate_full [V, H (d_h + d_v)] is head-major like kv; ln_w, ln_b [H (d_h + d_v)].
    """
    qf = widen(q, storage)
    cf = widen(cache, storage)
    gf = widen(gate_full, storage)
    wk = widen(w_uk, storage)
    wv = widen(w_uv, storage)
    lw = widen(ln_w, storage) if ln_w is not None else None
    lb = widen(ln_b, storage) if ln_b is not None else None
    B, H, _ = qf.shape
    d_c, d_h, d_r = latent_dim, head_dim, rope_dim
    d_v = wv.shape[1]
    tau = softmax_scale(d_h, d_r)
    out = np.zeros((B, H, d_v), dtype=np.float64)
    for b in range(B):
        L = int(seq_lens[b])
        if L == 0:
            continue
        rows = cache_rows(L, b, page_table, page_size, max_pages)
        kvt = literal_kv(cf[rows, :d_c], np.asarray(token_ids)[rows], gf, wk, wv, lw, lb, mode=mode, use_ln=use_ln)
        k_r = cf[rows, d_c:d_c + d_r]
        for h in range(H):
            blk = kvt[:, h * (d_h + d_v):(h + 1) * (d_h + d_v)]
            k = np.concatenate([blk[:, :d_h], k_r], axis=1)
            s = tau * (k @ qf[b, h, :d_h + d_r])
            out[b, h] = _softmax(s) @ blk[:, d_h:]
    return out


# ---------------------------------------------------------------------------
# prefill (causal, explicit form): the reference for eg_mla_prefill_ref
# ---------------------------------------------------------------------------
def prefill(q, latent, token_ids, gate_table, w_uk, w_uv, *, latent_dim: int, head_dim: int,
            rope_dim: int, storage: str, scale: Optional[float] = None) -> np.ndarray:
    """Causal attention for every position t of one sequence: out [T, H, d_v].

    Row t attends to tokens j <= t (App. C Eq. (C.13), sum from j = 1 to t).
    """
    qf = widen(q, storage)
    lf = widen(latent, storage)
    gf = widen(gate_table, storage)
    wk = widen(w_uk, storage)
    wv = widen(w_uv, storage)
    T, H, _ = qf.shape
    d_c, d_h, d_r = latent_dim, head_dim, rope_dim
    tau = softmax_scale(d_h, d_r) if scale is None else scale
    c_g = lf[:, :d_c] * gf[np.asarray(token_ids).astype(np.int64)]
    k_r = lf[:, d_c:d_c + d_r]
    mask = np.tril(np.ones((T, T), dtype=bool))
    out = np.zeros((T, H, wv.shape[1]), dtype=np.float64)
    for h in range(H):
        k = np.concatenate([c_g @ wk[h].T, k_r], axis=1)      # [T, d_h + d_r]
        v = c_g @ wv[h].T                                     # [T, d_v]
        s = tau * (qf[:, h, :d_h + d_r] @ k.T)                # [T(query), T(key)]
        s = np.where(mask, s, -np.inf)
        out[:, h] = _softmax(s) @ v
    return out


# ---------------------------------------------------------------------------
# append (write new tokens into the cache)
# ---------------------------------------------------------------------------
def rope_rotate(r: np.ndarray, positions: np.ndarray, base: float = ROPE_BASE) -> np.ndarray:
    """Rotary embedding on adjacent pairs (2i, 2i+1) with angle pos * base^(-2i/d)."""
    d = r.shape[-1]
    i = np.arange(d // 2, dtype=np.float64)
    inv_freq = base ** (-2.0 * i / d)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv_freq[None, :]
    cos, sin = np.cos(ang), np.sin(ang)
    x0 = r[:, 0::2]
    x1 = r[:, 1::2]
    out = np.empty_like(r)
    out[:, 0::2] = x0 * cos - x1 * sin
    out[:, 1::2] = x0 * sin + x1 * cos
    return out


def append(x, w_dkv, kv_norm_w, positions, *, latent_dim: int, rope_dim: int, storage: str,
           rope_theta: float = ROPE_BASE) -> np.ndarray:
    """Cache rows [n, d_c + d_r] for new tokens: [RMSNorm(c) | RoPE(k^R)].

    Eq. (1) c_t = W^DKV x_t and Eq. (C.10) k^R_t = RoPE(W^KR x_t); W^DKV and
    W^KR are stacked as one [d_c + d_r, hidden] matrix.  With a norm weight
    the latent is RMS-normalised first (the listing's latent norm).
    """
    xf = widen(x, storage)
    wf = widen(w_dkv, storage)
    y = xf @ wf.T
    c = y[:, :latent_dim]
    r = y[:, latent_dim:latent_dim + rope_dim]
    if kv_norm_w is not None:
        gam = widen(kv_norm_w, storage)
        c = c / np.sqrt(np.mean(c * c, axis=1, keepdims=True) + RMS_EPS) * gam
    if rope_dim:
        r = rope_rotate(r, positions, rope_theta)
    return np.concatenate([c, r], axis=1)
