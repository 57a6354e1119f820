"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a scalar
brute-force transcription, an algebraic identity (absorbed == explicit),
a special case that reduces to a library routine (torch SDPA in fp64) or to
a closed form, or an invariance the method must have.
"""
import math

import numpy as np
import pytest
import torch

from oracle import brute
from oracle import eg_mla_oracle as orc
from paper_2509_16686_amd import workloads as W


def kw(inp):
    wl = inp.wl
    return dict(latent_dim=wl.latent_dim, head_dim=wl.head_dim, rope_dim=wl.rope_dim, storage=wl.dtype,
                page_table=inp.page_table, page_size=wl.page_size, max_pages=inp.max_pages)


def run(fn, inp, **over):
    args = kw(inp)
    args.update(over)
    return fn(inp.q, inp.latent_cache, inp.token_ids, inp.gate_table, inp.w_uk, inp.w_uv, inp.seq_lens, **args)


def tiny(**over):
    base = W.Workload(name="tiny", batch=2, heads=2, head_dim=3, v_head_dim=3, latent_dim=4, rope_dim=2,
                      gate_dim=4, vocab=7, dtype="fp32", seq_len=6, page_size=4, seed=11, recipe="layer")
    return base.replace(**over)


def rel_err(a, b):
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def to_lists(inp):
    f = lambda a: orc.widen(a, inp.wl.dtype).tolist()
    return dict(q=f(inp.q), cache=f(inp.latent_cache), token_ids=inp.token_ids.tolist(), gate=f(inp.gate_table),
                w_uk=f(inp.w_uk), w_uv=f(inp.w_uv), seq_lens=inp.seq_lens.tolist())


# ---- P1: brute force ------------------------------------------------------
@pytest.mark.parametrize("over", [dict(), dict(paged=True), dict(seq_len=1), dict(rope_dim=0),
                                  dict(dtype="bf16", seed=3), dict(heads=3, head_dim=5, v_head_dim=2)])
def test_brute_force_matches_oracle(over):
    inp = W.generate(tiny(**over))
    L = to_lists(inp)
    wl = inp.wl
    got = brute.decode(L["q"], L["cache"], L["token_ids"], L["gate"], L["w_uk"], L["w_uv"], L["seq_lens"],
                       lambda b: [inp.slot(b, j) for j in range(int(inp.seq_lens[b]))],
                       latent_dim=wl.latent_dim, head_dim=wl.head_dim, rope_dim=wl.rope_dim)
    ref = run(orc.decode, inp)
    assert rel_err(ref, np.array(got)) < 1e-12


def test_brute_force_tiny_fp32_workload():
    inp = W.generate(W.WORKLOADS[0])
    L = to_lists(inp)
    wl = inp.wl
    got = brute.decode(L["q"], L["cache"], L["token_ids"], L["gate"], L["w_uk"], L["w_uv"], L["seq_lens"],
                       lambda b: [inp.slot(b, j) for j in range(int(inp.seq_lens[b]))],
                       latent_dim=wl.latent_dim, head_dim=wl.head_dim, rope_dim=wl.rope_dim)
    assert rel_err(run(orc.decode, inp), np.array(got)) < 1e-12


# ---- gate rows from the token embedding (Eq. (3)-(4)) --------------------
@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_gate_rows_brute_force(dtype):
    wl = tiny(dtype=dtype, vocab=9, latent_dim=5, gate_dim=5)
    ge = W.generate_gate_embedding(wl, emb_dim=6)
    ids = np.array([0, 8, 3, 3, -2, 11, 4], dtype=np.int32)  # out of range: clamped
    f = lambda a: orc.widen(a, dtype).tolist()
    got = np.array(brute.gate_rows(f(ge.emb), f(ge.w_ue), ids.tolist()))
    ref = orc.gate_rows(ge.emb, ge.w_ue, ids, storage=dtype)
    assert ref.shape == (7, 5)
    assert rel_err(ref, got) < 1e-12


def test_gate_rows_identity_projection_returns_embeddings():
    # W^UE = I (e = d_c): the gate is the embedding row itself, exactly
    wl = tiny(vocab=9)
    ge = W.generate_gate_embedding(wl, emb_dim=wl.latent_dim)
    eye = np.eye(wl.latent_dim, dtype=np.float32)
    ids = np.arange(9, dtype=np.int32)
    g = orc.gate_rows(ge.emb, eye, ids, storage="fp32")
    np.testing.assert_array_equal(g, orc.widen(ge.emb, "fp32"))


def test_unfolded_gate_decode_matches_brute_force():
    # EG-MLA with the gate computed from the embedding (Eq. (3)-(5)) through
    # the folded table G = Emb W^UE^T (the table-lookup variant): brute force
    # computes G and the decode with scalar loops, the oracle with NumPy
    wl = tiny(vocab=9, seq_len=7)
    inp = W.generate(wl)
    ge = W.generate_gate_embedding(wl, emb_dim=6)
    f = lambda a: orc.widen(a, wl.dtype).tolist()
    G_brute = brute.gate_rows(f(ge.emb), f(ge.w_ue), list(range(wl.vocab)))
    L = to_lists(inp)
    got = brute.decode(L["q"], L["cache"], L["token_ids"], G_brute, L["w_uk"], L["w_uv"], L["seq_lens"],
                       lambda b: [inp.slot(b, j) for j in range(int(inp.seq_lens[b]))],
                       latent_dim=wl.latent_dim, head_dim=wl.head_dim, rope_dim=wl.rope_dim)
    G = orc.gate_rows(ge.emb, ge.w_ue, np.arange(wl.vocab), storage=wl.dtype)
    ref = orc.decode(
        orc.widen(inp.q, wl.dtype), orc.widen(inp.latent_cache, wl.dtype), inp.token_ids, G,
        orc.widen(inp.w_uk, wl.dtype), orc.widen(inp.w_uv, wl.dtype), inp.seq_lens, latent_dim=wl.latent_dim,
        head_dim=wl.head_dim, rope_dim=wl.rope_dim, storage="f64", page_table=inp.page_table,
        page_size=wl.page_size, max_pages=inp.max_pages)
    assert rel_err(ref, np.array(got)) < 1e-12


def test_gate_embedding_recipe_centres_gates_at_one():
    wl = W.WORKLOADS[1].replace(vocab=4000)
    ge = W.generate_gate_embedding(wl, emb_dim=512)
    G = orc.gate_rows(ge.emb, ge.w_ue, np.arange(4000), storage=wl.dtype)
    assert abs(G.mean() - 1.0) < 0.01 and 0.08 < G.std() < 0.12


# ---- P2: absorbed == explicit --------------------------------------------
@pytest.mark.parametrize("wl", [tiny(), tiny(paged=True, batch=3, seq_len=9), W.WORKLOADS[0],
                                W.WORKLOADS[1].replace(batch=2, seq_len=300),
                                W.WORKLOADS[4].replace(batch=2, heads=4, seq_len_range=(70, 200))])
def test_absorbed_equals_explicit(wl):
    inp = W.generate(wl)
    a = run(orc.decode, inp)
    e = run(orc.decode_explicit, inp)
    assert rel_err(a, e) < 1e-12


# ---- P3 / P4: gate special cases -----------------------------------------
def test_all_ones_gate_is_plain_mla_bitwise():
    inp = W.generate(tiny(gate_all_ones=True, batch=3, seq_len=10))
    with_gate = run(orc.decode, inp)
    mla = run(orc.decode, inp, use_gate=False)
    assert np.array_equal(with_gate, mla)
    # and a non-trivial gate really changes the result
    inp2 = W.generate(tiny(batch=3, seq_len=10))
    assert rel_err(run(orc.decode, inp2), run(orc.decode, inp2, use_gate=False)) > 1e-3


def test_constant_gate_rows_fold_into_weights():
    inp = W.generate(tiny(batch=2, seq_len=8, heads=3))
    wl = inp.wl
    gamma = np.linspace(0.5, 1.7, wl.latent_dim)
    gate = np.tile(gamma, (wl.vocab, 1))
    wk = orc.widen(inp.w_uk, "fp32") * gamma
    wv = orc.widen(inp.w_uv, "fp32") * gamma
    cache = orc.widen(inp.latent_cache, "fp32")
    q = orc.widen(inp.q, "fp32")
    args = kw(inp)
    args["storage"] = "f64"
    gated = orc.decode(q, cache, inp.token_ids, gate, orc.widen(inp.w_uk, "fp32"), orc.widen(inp.w_uv, "fp32"),
                       inp.seq_lens, **args)
    folded = orc.decode(q, cache, inp.token_ids, gate, wk, wv, inp.seq_lens, use_gate=False, **args)
    assert rel_err(gated, folded) < 1e-12


# ---- P5: closed forms -----------------------------------------------------
def test_single_token_is_value_of_that_token():
    inp = W.generate(tiny(seq_len=1, batch=3))
    out = run(orc.decode, inp)
    cf = orc.widen(inp.latent_cache, "fp32")
    g = orc.widen(inp.gate_table, "fp32")
    wv = orc.widen(inp.w_uv, "fp32")
    for b in range(3):
        r = inp.slot(b, 0)
        cg = cf[r, :4] * g[inp.token_ids[r]]
        for h in range(inp.wl.heads):
            np.testing.assert_allclose(out[b, h], wv[h] @ cg, rtol=1e-13, atol=1e-15)


def test_zero_query_gives_uniform_average():
    inp = W.generate(tiny(seq_len=7))
    inp.q[:] = 0
    out = run(orc.decode, inp)
    cf = orc.widen(inp.latent_cache, "fp32")
    g = orc.widen(inp.gate_table, "fp32")
    wv = orc.widen(inp.w_uv, "fp32")
    for b in range(inp.wl.batch):
        rows = inp.slots_of(b)
        mean = (cf[rows, :4] * g[inp.token_ids[rows]]).mean(0)
        for h in range(inp.wl.heads):
            np.testing.assert_allclose(out[b, h], wv[h] @ mean, rtol=1e-12, atol=1e-15)


def test_empty_sequence_gives_zeros():
    inp = W.generate(tiny(batch=3, seq_len=5), seq_lens=np.array([5, 0, 2]))
    out = run(orc.decode, inp)
    assert np.all(out[1] == 0) and np.all(np.isfinite(out))
    assert np.abs(out[0]).sum() > 0 and np.abs(out[2]).sum() > 0


# ---- P6: reduction to a library routine (torch SDPA, fp64 CPU) ---------------
def test_identity_weights_single_head_is_sdpa():
    wl = tiny(batch=2, heads=1, head_dim=6, v_head_dim=6, latent_dim=6, gate_dim=6, rope_dim=0, seq_len=11)
    inp = W.generate(wl)
    eye = np.eye(6, dtype=np.float32)[None]
    inp.w_uk[:] = eye
    inp.w_uv[:] = eye
    out = run(orc.decode, inp)
    cf = orc.widen(inp.latent_cache, "fp32")
    g = orc.widen(inp.gate_table, "fp32")
    q = orc.widen(inp.q, "fp32")
    for b in range(2):
        rows = inp.slots_of(b)
        kv = torch.from_numpy(cf[rows, :6] * g[inp.token_ids[rows]])[None, None]
        qq = torch.from_numpy(q[b, :, :6])[None, :, None, :]
        ref = torch.nn.functional.scaled_dot_product_attention(qq, kv, kv)[0, 0, 0].numpy()
        np.testing.assert_allclose(out[b, 0], ref, rtol=1e-12, atol=1e-15)


def test_random_weights_with_rope_is_sdpa_per_head():
    """Keys/values built per Eq. (C.2),(C.6),(C.12); SDPA's default 1/sqrt(E) scale with
    E = d_h + d_r fixes the softmax temperature of Eq. (C.13) independently of d_c."""
    wl = tiny(batch=2, heads=3, head_dim=5, v_head_dim=4, latent_dim=7, gate_dim=7, rope_dim=4, seq_len=13,
              vocab=11, paged=True)
    inp = W.generate(wl)
    out = run(orc.decode, inp)
    cf = orc.widen(inp.latent_cache, "fp32")
    g = orc.widen(inp.gate_table, "fp32")
    q = orc.widen(inp.q, "fp32")
    wk = orc.widen(inp.w_uk, "fp32")
    wv = orc.widen(inp.w_uv, "fp32")
    for b in range(2):
        rows = inp.slots_of(b)
        cg = torch.from_numpy(cf[rows, :7] * g[inp.token_ids[rows]])
        kr = torch.from_numpy(cf[rows, 7:])
        for h in range(3):
            k = torch.cat([cg @ torch.from_numpy(wk[h]).T, kr], 1)[None, None]
            v = (cg @ torch.from_numpy(wv[h]).T)[None, None]
            qq = torch.from_numpy(q[b, h])[None, None, None]
            ref = torch.nn.functional.scaled_dot_product_attention(qq, k, v)[0, 0, 0].numpy()
            np.testing.assert_allclose(out[b, h], ref, rtol=1e-11, atol=1e-14)


# ---- P7: layout and permutation invariance -----------------------------------
def test_paged_equals_contiguous_bitwise():
    inp = W.generate(tiny(batch=3, seq_len=10, page_size=4))
    # Build a paged copy: random physical page per logical page.
    rng = np.random.default_rng(5)
    P, mp = 4, inp.max_pages
    perm = rng.permutation(3 * mp)
    pt = perm.reshape(3, mp).astype(np.int32)
    cache2 = np.zeros_like(inp.latent_cache)
    ids2 = np.zeros_like(inp.token_ids)
    for b in range(3):
        for j in range(10):
            src = inp.slot(b, j)
            dst = pt[b, j // P] * P + j % P
            cache2[dst] = inp.latent_cache[src]
            ids2[dst] = inp.token_ids[src]
    a = run(orc.decode, inp)
    args = kw(inp)
    args["page_table"] = pt
    b_ = orc.decode(inp.q, cache2, ids2, inp.gate_table, inp.w_uk, inp.w_uv, inp.seq_lens, **args)
    assert np.array_equal(a, b_)


def test_token_permutation_invariance():
    inp = W.generate(tiny(batch=2, seq_len=12))
    a = run(orc.decode, inp)
    rng = np.random.default_rng(9)
    for b in range(2):
        rows = inp.slots_of(b)
        p = rng.permutation(rows.size)
        inp.latent_cache[rows] = inp.latent_cache[rows[p]]
        inp.token_ids[rows] = inp.token_ids[rows[p]]
    assert rel_err(run(orc.decode, inp), a) < 1e-13
    # ids that do not travel with their tokens do change the result (the gather is by id)
    inp.token_ids[inp.slots_of(0)] = np.roll(inp.token_ids[inp.slots_of(0)], 1)
    assert rel_err(run(orc.decode, inp)[0], a[0]) > 1e-4


# ---- P8: softmax shift invariance via the RoPE part -----------------------------
def test_constant_rope_key_cancels():
    inp = W.generate(tiny(batch=2, seq_len=9, rope_dim=2))
    wl = inp.wl
    inp.latent_cache[:, wl.latent_dim:] = inp.latent_cache[0, wl.latent_dim:]
    full = run(orc.decode, inp)
    tau = orc.softmax_scale(wl.head_dim, wl.rope_dim)
    args = kw(inp)
    args.update(rope_dim=0, scale=tau)
    no_rope = orc.decode(np.ascontiguousarray(inp.q[:, :, :wl.head_dim]), np.ascontiguousarray(
        inp.latent_cache[:, :wl.latent_dim]), inp.token_ids, inp.gate_table, inp.w_uk, inp.w_uv, inp.seq_lens, **args)
    assert rel_err(full, no_rope) < 1e-13


def test_peaked_logits_are_finite_and_match_brute():
    inp = W.generate(tiny(batch=1, seq_len=8))
    inp.q *= 400.0
    out = run(orc.decode, inp)
    assert np.all(np.isfinite(out))
    L = to_lists(inp)
    wl = inp.wl
    got = brute.decode(L["q"], L["cache"], L["token_ids"], L["gate"], L["w_uk"], L["w_uv"], L["seq_lens"],
                       lambda b: [inp.slot(b, j) for j in range(int(inp.seq_lens[b]))],
                       latent_dim=wl.latent_dim, head_dim=wl.head_dim, rope_dim=wl.rope_dim)
    assert rel_err(out, np.array(got)) < 1e-12


# ---- prefill -------------------------------------------------------------------
def test_prefill_rows_equal_decode_of_prefix():
    wl = tiny(heads=3, seq_len=1)
    pin = W.generate_prefill(wl, 10)
    pre = orc.prefill(pin.q, pin.latent, pin.token_ids, pin.gate_table, pin.w_uk, pin.w_uv,
                      latent_dim=wl.latent_dim, head_dim=wl.head_dim, rope_dim=wl.rope_dim, storage=wl.dtype)
    for t in range(10):
        d = orc.decode(pin.q[t][None], pin.latent, pin.token_ids, pin.gate_table, pin.w_uk, pin.w_uv,
                       np.array([t + 1]), latent_dim=wl.latent_dim, head_dim=wl.head_dim, rope_dim=wl.rope_dim,
                       storage=wl.dtype, page_table=None, page_size=64, max_pages=0)
        assert rel_err(pre[t], d[0]) < 1e-12


def test_prefill_is_causal_sdpa():
    wl = tiny(heads=2, head_dim=4, v_head_dim=3, latent_dim=5, gate_dim=5, rope_dim=2, vocab=9)
    pin = W.generate_prefill(wl, 12)
    pre = orc.prefill(pin.q, pin.latent, pin.token_ids, pin.gate_table, pin.w_uk, pin.w_uv,
                      latent_dim=5, head_dim=4, rope_dim=2, storage="fp32")
    lf = orc.widen(pin.latent, "fp32")
    cg = torch.from_numpy(lf[:, :5] * orc.widen(pin.gate_table, "fp32")[pin.token_ids])
    kr = torch.from_numpy(lf[:, 5:])
    for h in range(2):
        k = torch.cat([cg @ torch.from_numpy(orc.widen(pin.w_uk, "fp32")[h]).T, kr], 1)[None, None]
        v = (cg @ torch.from_numpy(orc.widen(pin.w_uv, "fp32")[h]).T)[None, None]
        qq = torch.from_numpy(orc.widen(pin.q, "fp32")[:, h])[None, None]
        ref = torch.nn.functional.scaled_dot_product_attention(qq, k, v, is_causal=True)[0, 0].numpy()
        np.testing.assert_allclose(pre[:, h], ref, rtol=1e-11, atol=1e-14)


# ---- append ------------------------------------------------------------------------
def test_rope_closed_forms():
    rng = np.random.default_rng(0)
    r = rng.standard_normal((5, 8))
    # position 0 is the identity
    np.testing.assert_array_equal(orc.rope_rotate(r, np.zeros(5)), r)
    # rotation preserves the norm of every (2i, 2i+1) pair
    rot = orc.rope_rotate(r, np.array([1, 7, 100, 4095, 32767]))
    np.testing.assert_allclose(np.hypot(rot[:, 0::2], rot[:, 1::2]), np.hypot(r[:, 0::2], r[:, 1::2]), rtol=1e-13)
    # dot products depend only on the relative position
    a, b = r[0:1], r[1:2]
    d1 = (orc.rope_rotate(a, np.array([10])) * orc.rope_rotate(b, np.array([3]))).sum()
    d2 = (orc.rope_rotate(a, np.array([107])) * orc.rope_rotate(b, np.array([100]))).sum()
    assert abs(d1 - d2) < 1e-12
    # pair 0 turns by exactly `pos` radians (theta_0 = 1)
    e = np.zeros((1, 8))
    e[0, 0] = 1
    out = orc.rope_rotate(e, np.array([2.0]))
    np.testing.assert_allclose(out[0, :2], [math.cos(2.0), math.sin(2.0)], rtol=1e-14)


def test_append_projection_and_norm():
    wl = tiny(hidden=6, latent_dim=4, rope_dim=2)
    ap = W.generate_append(wl, 5, 20)
    rows = orc.append(ap.x, ap.w_dkv, None, np.zeros(5, dtype=np.int32), latent_dim=4, rope_dim=2, storage="fp32")
    x = orc.widen(ap.x, "fp32")
    w = orc.widen(ap.w_dkv, "fp32")
    for i in range(5):
        for o in range(6):
            assert abs(rows[i, o] - sum(w[o, k] * x[i, k] for k in range(6))) < 1e-12
    normed = orc.append(ap.x, ap.w_dkv, np.ones(4, np.float32), np.zeros(5, dtype=np.int32), latent_dim=4,
                        rope_dim=2, storage="fp32")
    rms = np.sqrt((normed[:, :4] ** 2).mean(1))
    ms = (rows[:, :4] ** 2).mean(1)
    np.testing.assert_allclose(rms, np.sqrt(ms / (ms + orc.RMS_EPS)), rtol=1e-12)
    np.testing.assert_array_equal(normed[:, 4:], rows[:, 4:])


# ---- storage widening ------------------------------------------------------------
def test_bf16_widening_is_exact():
    vals = np.array([1.0, -2.5, 3.140625, 1e-3, 65504.0, -0.0], dtype=np.float32)
    bits = W.f32_to_bf16_bits(vals)
    back = orc.widen(bits, "bf16")
    ref = torch.from_numpy(vals).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(back, ref)


# ---- the paper-literal gate (Sec. 3.1 Eq. (2)-(5) as printed) --------------
def literal(inp, lg, **over):
    wl = inp.wl
    args = kw(inp)
    args.update(over)
    return orc.decode_literal(inp.q, inp.latent_cache, inp.token_ids, lg.gate_full, inp.w_uk, inp.w_uv, lg.ln_w,
                              lg.ln_b, inp.seq_lens, **args)


@pytest.mark.parametrize("mode,use_ln", [("mul", True), ("mul", False), ("add", True), ("add", False)])
@pytest.mark.parametrize("over", [dict(), dict(paged=True, heads=3, v_head_dim=2)])
def test_literal_gate_brute_force(mode, use_ln, over):
    wl = tiny(**over)
    inp = W.generate(wl)
    lg = W.generate_literal_gate(wl)
    L = to_lists(inp)
    f = lambda a: orc.widen(a, wl.dtype).tolist()
    got = brute.decode_literal(L["q"], L["cache"], L["token_ids"], f(lg.gate_full), L["w_uk"], L["w_uv"],
                               f(lg.ln_w), f(lg.ln_b), L["seq_lens"],
                               lambda b: [inp.slot(b, j) for j in range(int(inp.seq_lens[b]))],
                               latent_dim=wl.latent_dim, head_dim=wl.head_dim, rope_dim=wl.rope_dim, mode=mode,
                               use_ln=use_ln)
    ref = literal(inp, lg, mode=mode, use_ln=use_ln)
    assert rel_err(ref, np.array(got)) < 1e-12


def test_literal_without_ln_and_unit_gate_is_plain_mla():
    # no LayerNorm and an all-ones product gate (or a zero additive gate) leave
    # plain MLA, which the absorbed decode computes by another route
    wl = tiny(seq_len=9, batch=3)
    inp = W.generate(wl)
    lg = W.generate_literal_gate(wl)
    plain = run(orc.decode, inp, use_gate=False)
    ones = dataclass_replace(lg, gate_full=np.ones_like(lg.gate_full))
    zeros = dataclass_replace(lg, gate_full=np.zeros_like(lg.gate_full))
    assert rel_err(literal(inp, ones, use_ln=False), plain) < 1e-12
    assert rel_err(literal(inp, zeros, mode="add", use_ln=False), plain) < 1e-12


def dataclass_replace(obj, **kw_):
    import dataclasses
    return dataclasses.replace(obj, **kw_)


def test_literal_kv_rows_are_layer_normalised():
    # with unit weight and zero bias every gated row has mean 0 and variance
    # var / (var + eps) over all heads' dims
    wl = tiny(heads=4, head_dim=5, v_head_dim=3)
    inp = W.generate(wl)
    lg = W.generate_literal_gate(wl)
    c = orc.widen(inp.latent_cache, wl.dtype)[:, :wl.latent_dim]
    width = wl.heads * (wl.head_dim + wl.v_head_dim)
    x = orc.literal_kv(c, inp.token_ids, orc.widen(lg.gate_full, wl.dtype), orc.widen(inp.w_uk, wl.dtype),
                       orc.widen(inp.w_uv, wl.dtype), np.ones(width), np.zeros(width))
    raw = orc.literal_kv(c, inp.token_ids, orc.widen(lg.gate_full, wl.dtype), orc.widen(inp.w_uk, wl.dtype),
                         orc.widen(inp.w_uv, wl.dtype), None, None, use_ln=False)
    var = raw.var(axis=1)
    np.testing.assert_allclose(x.mean(axis=1), 0.0, atol=1e-12)
    np.testing.assert_allclose(x.var(axis=1), var / (var + orc.LN_EPS), rtol=1e-12)
    # head-major split: head h's key rows are W_UK[h] c, its value rows W_UV[h] c (before the gate)
    kv = orc.literal_kv(c, inp.token_ids, np.ones_like(orc.widen(lg.gate_full, wl.dtype)),
                        orc.widen(inp.w_uk, wl.dtype), orc.widen(inp.w_uv, wl.dtype), None, None, use_ln=False)
    h = 2
    d = wl.head_dim + wl.v_head_dim
    np.testing.assert_allclose(kv[:, h * d:h * d + wl.head_dim], c @ orc.widen(inp.w_uk, wl.dtype)[h].T, rtol=1e-13)
    np.testing.assert_allclose(kv[:, h * d + wl.head_dim:(h + 1) * d], c @ orc.widen(inp.w_uv, wl.dtype)[h].T,
                               rtol=1e-13)


def test_literal_zero_ln_weight_returns_bias_values():
    # LN weight 0: every key and value is the bias, so each head's output is its
    # value part of the bias (the softmax weights sum to one)
    wl = tiny(seq_len=8)
    inp = W.generate(wl)
    lg = W.generate_literal_gate(wl)
    lg0 = dataclass_replace(lg, ln_w=np.zeros_like(lg.ln_w))
    out = literal(inp, lg0)
    b = orc.widen(lg.ln_b, wl.dtype)
    d = wl.head_dim + wl.v_head_dim
    for h in range(wl.heads):
        np.testing.assert_allclose(out[:, h], np.broadcast_to(b[h * d + wl.head_dim:(h + 1) * d], out[:, h].shape),
                                   rtol=1e-12, atol=1e-14)


def test_literal_ln_removes_latent_scale():
    # scaling one token's cached latent by 3 scales its gated row by 3, which the
    # LayerNorm removes up to its epsilon (LN(3x) normalises with eps / 9: a
    # change of order eps / var); without the norm the output changes
    wl = tiny(seq_len=7)
    inp = W.generate(wl)
    lg = W.generate_literal_gate(wl)
    base = literal(inp, lg)
    inp2 = W.generate(wl)
    r = inp2.slot(0, 3)
    inp2.latent_cache[r, :wl.latent_dim] *= 3
    assert rel_err(literal(inp2, lg), base) < 1e-5
    assert rel_err(literal(inp2, lg, use_ln=False), literal(inp, lg, use_ln=False)) > 1e-3


# ---- App. H: layer grouping ----------------------------------------------------
def test_layer_group_layers_read_the_shared_rows():
    """Each layer of a group attends over the one shared set of cached rows with its
    own query, weights and gate table: its output is SDPA (fp64, CPU) over keys and
    values built from the shared rows with that layer's W_UK, W_UV and gate, and
    layers with different weights give different outputs."""
    wl = tiny(batch=2, heads=2, head_dim=5, v_head_dim=4, latent_dim=7, gate_dim=7, rope_dim=4, seq_len=9,
              vocab=11, paged=True)
    layers = W.generate_layer_group(wl, 3)
    base = layers[0]
    outs = orc.decode_layer_group(base.latent_cache, base.token_ids, base.seq_lens,
                                  [(l.q, l.gate_table, l.w_uk, l.w_uv) for l in layers], **kw(base))
    cf = orc.widen(base.latent_cache, "fp32")
    for lay, out in zip(layers, outs):
        assert lay.latent_cache is base.latent_cache and lay.token_ids is base.token_ids
        g = orc.widen(lay.gate_table, "fp32")
        q = orc.widen(lay.q, "fp32")
        wk, wv = orc.widen(lay.w_uk, "fp32"), orc.widen(lay.w_uv, "fp32")
        for b in range(2):
            rows = base.slots_of(b)
            cg = torch.from_numpy(cf[rows, :7] * g[base.token_ids[rows]])
            kr = torch.from_numpy(cf[rows, 7:])
            for h in range(2):
                k = torch.cat([cg @ torch.from_numpy(wk[h]).T, kr], 1)[None, None]
                v = (cg @ torch.from_numpy(wv[h]).T)[None, None]
                ref = torch.nn.functional.scaled_dot_product_attention(torch.from_numpy(q[b, h])[None, None, None],
                                                                       k, v)[0, 0, 0].numpy()
                np.testing.assert_allclose(out[b, h], ref, rtol=1e-11, atol=1e-14)
    assert rel_err(outs[0], outs[1]) > 1e-3 and rel_err(outs[1], outs[2]) > 1e-3
