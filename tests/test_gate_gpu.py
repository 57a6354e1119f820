"""GPU parity of eg_mla_gate_rows (Sec. 3.1 Eq. (3)-(4)) and of the decode fed
with gates computed from the embedding, against the fp64 oracle through the C
ABI.

Two uses: folding the whole vocabulary into the gate table the decode takes
(the table-lookup variant of Sec. 5.2), and the unfolded model's per-step
gates (one row per cached token, handed to the decode with the row indices as
token ids).  The references take the oracle's own fp64 gate rows; the GPU
path stores its rows in the storage type, which the bf16 tolerances absorb.
"""
import numpy as np
import pytest

from oracle import eg_mla_oracle as orc
from paper_2509_16686_amd import binding as B
from paper_2509_16686_amd import workloads as W
from parity import assert_close, say

pytestmark = pytest.mark.gpu


def gpu_gate_rows(wl, ge, ids):
    """Device tensor [n, d_c] of W^UE Emb[ids] from the library."""
    import torch
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    out = torch.empty((len(ids), wl.latent_dim), dtype=dt, device="cuda")
    ids_d = B.to_device_tensor(np.ascontiguousarray(ids, dtype=np.int32), "int")
    B.gate_rows(B.dims_for(wl), ids_d, B.to_device_tensor(ge.emb, wl.dtype), B.to_device_tensor(ge.w_ue, wl.dtype),
                out)
    torch.cuda.synchronize()
    return out


def check_rows(got, ge, ids, storage):
    """Element-wise bound: one rounding to the storage type of the fp32 sum,
    plus fp32 accumulation error against the sum of |products|."""
    ref = orc.gate_rows(ge.emb, ge.w_ue, ids, storage=storage)
    ef = orc.widen(ge.emb, storage)[np.clip(ids, 0, ge.emb.shape[0] - 1)]
    mag = np.abs(ef) @ np.abs(orc.widen(ge.w_ue, storage)).T
    rnd = 2.0 ** -8 if storage == "bf16" else 2.0 ** -23
    bound = rnd * np.abs(ref) + 2.0 ** -22 * np.sqrt(ef.shape[1]) * mag + 1e-30
    assert got.shape == ref.shape
    assert np.all(np.isfinite(got))
    err = np.abs(got - ref)
    worst = float((err / bound).max()) if err.size else 0.0
    say(f"  gate rows: max |err| {float(err.max()) if err.size else 0.0:.3e}, worst err/bound {worst:.3f}")
    assert worst <= 1.0


@pytest.mark.parametrize("latent_dim,emb_dim,dtype,n", [
    (128, 512, "bf16", 1000),     # MFMA, one pass, one 128-column slice, ragged last block
    (128, 512, "bf16", 200003),   # several blocks per wave through the two-half pipeline
    (512, 512, "bf16", 777),      # four column slices
    (128, 384, "bf16", 65),       # one pass of 24 chunks
    (96, 256, "bf16", 70),        # slice padded past d_c (96 of 128 columns)
    (64, 128, "bf16", 33),        # two 32-column blocks
    (32, 128, "bf16", 50),        # d_c 32: a padded 64-column slice
    (32, 768, "bf16", 90),        # one 32-column block, passes of 256 components
    (128, 1024, "bf16", 40),      # passes of 256 components
    (64, 640, "bf16", 100),       # passes of 128 components
    (128, 96, "bf16", 65),        # VALU: embedding width not a multiple of 128
    (144, 40, "bf16", 33),        # VALU: d_c not a multiple of 32
    (32, 32, "fp32", 300),        # VALU, fp32 storage
    (128, 512, "bf16", 1),        # a single row
])
def test_gate_rows_match_oracle(gpu, latent_dim, emb_dim, dtype, n):
    wl = W.WORKLOADS[1].replace(latent_dim=latent_dim, gate_dim=latent_dim, dtype=dtype, vocab=3000, seed=51)
    ge = W.generate_gate_embedding(wl, emb_dim)
    ids = np.random.default_rng(7).integers(-5, wl.vocab + 5, size=n).astype(np.int32)  # out of range: clamped
    say(f"gate rows d_c={latent_dim} e={emb_dim} {dtype} n={n}")
    check_rows(B.out_to_f64(gpu_gate_rows(wl, ge, ids)), ge, ids, dtype)


def test_gate_rows_empty(gpu):
    import torch
    wl = W.WORKLOADS[1]
    ge = W.generate_gate_embedding(wl.replace(vocab=16), 64)
    out = torch.empty((0, wl.latent_dim), dtype=torch.bfloat16, device="cuda")
    ids = torch.empty((0,), dtype=torch.int32, device="cuda")
    say("gate rows n=0")
    B.gate_rows(B.dims_for(wl), ids, B.to_device_tensor(ge.emb, "bf16"), B.to_device_tensor(ge.w_ue, "bf16"), out)
    torch.cuda.synchronize()


def test_fold_vocabulary_then_decode(gpu):
    # G = Emb W^UE^T over the whole vocabulary on the GPU, then the decode
    # reads it as its gate table
    import torch
    wl = W.WORKLOADS[1].replace(batch=3, seq_len=700, seed=52)
    inp = W.generate(wl)
    ge = W.generate_gate_embedding(wl, 512)
    ids = np.arange(wl.vocab, dtype=np.int32)
    say(f"fold {wl.vocab} gate rows (e=512), then decode {wl.name} batch 3 L700")
    G = gpu_gate_rows(wl, ge, ids)
    check_rows(B.out_to_f64(G), ge, ids, "bf16")
    dd = B.stage_decode(inp)
    dd.gate = G
    B.run_decode(dd)
    torch.cuda.synchronize()
    Gref = orc.gate_rows(ge.emb, ge.w_ue, ids, storage="bf16")
    ref = orc.decode(orc.widen(inp.q, "bf16"), orc.widen(inp.latent_cache, "bf16"), inp.token_ids, Gref,
                     orc.widen(inp.w_uk, "bf16"), orc.widen(inp.w_uv, "bf16"), inp.seq_lens,
                     latent_dim=wl.latent_dim, head_dim=wl.head_dim, rope_dim=wl.rope_dim, storage="f64",
                     page_table=inp.page_table, page_size=wl.page_size, max_pages=inp.max_pages)
    assert_close(B.out_to_f64(dd.out), ref, "bf16", "folded decode")


@pytest.mark.parametrize("wl", [
    W.WORKLOADS[1].replace(batch=2, seq_len=500, vocab=8192, seed=53),
    W.WORKLOADS[4].replace(batch=3, seq_len_range=(100, 700), vocab=8192, seed=54),
], ids=["dc128", "dc512_paged"])
def test_unfolded_step_decode(gpu, wl):
    # the unfolded model's step: one gate row per cache row (from that row's
    # token embedding), then the decode with row indices as its ids
    import torch
    inp = W.generate(wl)
    ge = W.generate_gate_embedding(wl, 512)
    say(f"unfolded step {wl.name}: {inp.num_rows} gate rows (e=512), then decode")
    rows = gpu_gate_rows(wl, ge, inp.token_ids)
    dd = B.stage_decode(inp)
    dd.dims = B.dims_for(wl.replace(vocab=inp.num_rows))
    dd.gate = rows
    dd.ids = torch.arange(inp.num_rows, dtype=torch.int32, device="cuda")
    B.run_decode(dd)
    torch.cuda.synchronize()
    # reference: the gate of Eq. (3)-(4) per cached token, exact in fp64
    Grow = orc.gate_rows(ge.emb, ge.w_ue, inp.token_ids, storage="bf16")
    ref = orc.decode(orc.widen(inp.q, "bf16"), orc.widen(inp.latent_cache, "bf16"),
                     np.arange(inp.num_rows, dtype=np.int32), Grow, orc.widen(inp.w_uk, "bf16"),
                     orc.widen(inp.w_uv, "bf16"), inp.seq_lens, latent_dim=wl.latent_dim, head_dim=wl.head_dim,
                     rope_dim=wl.rope_dim, storage="f64", page_table=inp.page_table, page_size=wl.page_size,
                     max_pages=inp.max_pages)
    assert_close(B.out_to_f64(dd.out), ref, "bf16", f"unfolded {wl.name}")


def gpu_gate_table(wl, ge, ids, table, marks, stamp):
    """eg_mla_gate_table into `table` (device [emb_vocab, d_c]) with the given marks and stamp."""
    import torch
    ids_d = B.to_device_tensor(np.ascontiguousarray(ids, dtype=np.int32), "int")
    B.gate_table(B.dims_for(wl), ids_d, B.to_device_tensor(ge.emb, wl.dtype), B.to_device_tensor(ge.w_ue, wl.dtype),
                 table, marks, stamp)
    torch.cuda.synchronize()


@pytest.mark.parametrize("latent_dim,emb_dim,n,vocab", [
    (128, 512, 5000, 700),     # MFMA claims: about 7 rows per id
    (512, 512, 3001, 900),     # four column slices, each claiming its ids
    (128, 256, 65, 64),        # a ragged last block
    (32, 128, 300, 40),        # d_c 32: a padded 64-column slice
    (128, 1024, 300, 200),     # passes of 256 components: every row stores
    (144, 40, 90, 50),         # VALU: every row stores
])
def test_gate_table_rows(gpu, latent_dim, emb_dim, n, vocab):
    # table[id] = W^UE Emb[id] for the distinct ids of a list: the same bits
    # as eg_mla_gate_rows, within the oracle's bound, other rows untouched;
    # then a second call with another stamp and another list
    import torch
    wl = W.WORKLOADS[1].replace(latent_dim=latent_dim, gate_dim=latent_dim, vocab=vocab, seed=55)
    ge = W.generate_gate_embedding(wl, emb_dim)
    dims = B.dims_for(wl)
    rng = np.random.default_rng(8)
    ids1 = rng.integers(-3, vocab // 2 + 3, size=n).astype(np.int32)   # out of range: clamped
    ids2 = rng.integers(vocab // 3, vocab, size=n).astype(np.int32)
    sentinel = 0x7bcd
    table = torch.full((vocab, latent_dim), sentinel, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    mbytes = B.gate_table_marks_size(dims, emb_dim, vocab)
    assert mbytes > 0
    marks = torch.zeros((mbytes + 3) // 4, dtype=torch.int32, device="cuda")
    written = np.zeros(vocab, dtype=bool)
    for stamp, ids in ((1, ids1), (2, ids2)):
        say(f"gate table d_c={latent_dim} e={emb_dim} n={n} vocab={vocab} stamp={stamp}")
        gpu_gate_table(wl, ge, ids, table, marks, stamp)
        rows = gpu_gate_rows(wl, ge, ids)
        got = table.view(torch.int16).cpu().numpy()
        cid = np.clip(ids, 0, vocab - 1)
        assert np.array_equal(got[cid], rows.view(torch.int16).cpu().numpy()), "table rows differ from gate rows"
        written[cid] = True
        assert np.all(got[~written] == sentinel), "a row outside the lists was written"
    distinct = np.flatnonzero(written).astype(np.int32)
    check_rows(B.out_to_f64(table[torch.from_numpy(distinct).long().cuda()]), ge, distinct, "bf16")


def test_unfolded_step_through_table(gpu):
    # the unfolded step with each distinct id computed once: the decode takes
    # the table with the step's own token ids
    import torch
    wl = W.WORKLOADS[1].replace(batch=3, seq_len=900, vocab=2000, seed=56)
    inp = W.generate(wl)
    ge = W.generate_gate_embedding(wl, 512)
    dims = B.dims_for(wl)
    table = torch.zeros((wl.vocab, wl.latent_dim), dtype=torch.bfloat16, device="cuda")
    marks = torch.zeros((B.gate_table_marks_size(dims, 512, wl.vocab) + 3) // 4, dtype=torch.int32, device="cuda")
    say(f"unfolded step through the table {wl.name}: {inp.num_rows} rows, then decode")
    gpu_gate_table(wl, ge, inp.token_ids, table, marks, 1)
    dd = B.stage_decode(inp)
    dd.gate = table
    B.run_decode(dd)
    torch.cuda.synchronize()
    Gref = orc.gate_rows(ge.emb, ge.w_ue, np.arange(wl.vocab, dtype=np.int32), storage="bf16")
    ref = orc.decode(orc.widen(inp.q, "bf16"), orc.widen(inp.latent_cache, "bf16"), inp.token_ids, Gref,
                     orc.widen(inp.w_uk, "bf16"), orc.widen(inp.w_uv, "bf16"), inp.seq_lens,
                     latent_dim=wl.latent_dim, head_dim=wl.head_dim, rope_dim=wl.rope_dim, storage="f64",
                     page_table=inp.page_table, page_size=wl.page_size, max_pages=inp.max_pages)
    assert_close(B.out_to_f64(dd.out), ref, "bf16", "unfolded step through the table")
