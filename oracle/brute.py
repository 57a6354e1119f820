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
