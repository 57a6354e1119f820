"""Pure-Python scalar-loop EG-MLA decode for tiny inputs.

TEST INFRASTRUCTURE ONLY (same import rule as ``eg_mla_oracle``).  This is a
second, independent transcription of App. C Eq. (C.2), (C.6), (C.11)-(C.13)
with the gate of Eq. (3)-(5) applied to the latent: explicit per-head keys
and values built element by element, logits, a direct softmax, and the
weighted sum.  No NumPy arithmetic is used, so a slip in the vectorised
oracle's indexing or einsum strings shows up as a mismatch.
"""
from __future__ import annotations

import math


def decode(q, cache, token_ids, gate, w_uk, w_uv, seq_lens, rows_of, *, latent_dim, head_dim, rope_dim):
    """All arguments are nested Python lists of floats (already widened).

    ``rows_of(b)`` returns the cache rows of sequence b in token order.
    Returns out[b][h][v].
    """
    d_c, d_h, d_r = latent_dim, head_dim, rope_dim
    H = len(w_uk)
    d_v = len(w_uv[0])
    tau = 1.0 / math.sqrt(d_h + d_r)
    out = []
    for b in range(len(seq_lens)):
        per_head = []
        rows = rows_of(b)
        for h in range(H):
            if seq_lens[b] == 0:
                per_head.append([0.0] * d_v)
                continue
            logits = []
            values = []
            for r in rows:
                gated = [cache[r][c] * gate[token_ids[r]][c] for c in range(d_c)]
                key = [sum(w_uk[h][k][c] * gated[c] for c in range(d_c)) for k in range(d_h)]
                key += [cache[r][d_c + i] for i in range(d_r)]
                val = [sum(w_uv[h][v][c] * gated[c] for c in range(d_c)) for v in range(d_v)]
                logits.append(tau * sum(q[b][h][k] * key[k] for k in range(d_h + d_r)))
                values.append(val)
            top = max(logits)
            weights = [math.exp(s - top) for s in logits]
            total = sum(weights)
            per_head.append([sum(weights[j] * values[j][v] for j in range(len(rows))) / total
                             for v in range(d_v)])
        out.append(per_head)
    return out


def gate_rows(emb, w_ue, ids):
    """Eq. (4) element by element: g[i][c] = sum_k W^UE[c][k] Emb[ids[i]][k].

    ``emb`` and ``w_ue`` are nested lists of floats; ids are clamped into the
    table like the library does."""
    out = []
    for i in ids:
        e = emb[min(max(int(i), 0), len(emb) - 1)]
        out.append([sum(w_ue[c][k] * e[k] for k in range(len(e))) for c in range(len(w_ue))])
    return out


def decode_literal(q, cache, token_ids, gate_full, w_uk, w_uv, ln_w, ln_b, seq_lens, rows_of, *, latent_dim,
                   head_dim, rope_dim, mode="mul", use_ln=True, eps=1e-5):
    """Scalar loops for the paper-literal gate (Eq. (2)-(5)): per cached row,
    the up-projected key and value of every head, the gate product (or sum),
    one LayerNorm over all heads' dims, then per-head attention."""
    d_c, d_h, d_r = latent_dim, head_dim, rope_dim
    H = len(w_uk)
    d_v = len(w_uv[0])
    width = H * (d_h + d_v)
    tau = 1.0 / math.sqrt(d_h + d_r)
    out = []
    for b in range(len(seq_lens)):
        rows = rows_of(b)
        normed = []
        for r in rows:
            x = []
            for h in range(H):
                for k in range(d_h):
                    x.append(sum(w_uk[h][k][c] * cache[r][c] for c in range(d_c)))
                for v in range(d_v):
                    x.append(sum(w_uv[h][v][c] * cache[r][c] for c in range(d_c)))
            g = gate_full[token_ids[r]]
            x = [x[i] * g[i] if mode == "mul" else x[i] + g[i] for i in range(width)]
            if use_ln:
                mu = sum(x) / width
                var = sum((xi - mu) ** 2 for xi in x) / width
                x = [(x[i] - mu) / math.sqrt(var + eps) * ln_w[i] + ln_b[i] for i in range(width)]
            normed.append(x)
        per_head = []
        for h in range(H):
            if seq_lens[b] == 0:
                per_head.append([0.0] * d_v)
                continue
            base = h * (d_h + d_v)
            logits = []
            for j, r in enumerate(rows):
                key = normed[j][base:base + d_h] + [cache[r][d_c + i] for i in range(d_r)]
                logits.append(tau * sum(q[b][h][k] * key[k] for k in range(d_h + d_r)))
            top = max(logits)
            wts = [math.exp(s_ - top) for s_ in logits]
            tot = sum(wts)
            per_head.append([sum(wts[j] * normed[j][base + d_h + v] for j in range(len(rows))) / tot
                             for v in range(d_v)])
        out.append(per_head)
    return out
