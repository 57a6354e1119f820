"""GPU parity of eg_mla_prefill_varlen (App. C Eq. (C.13), with the latent-space
gate of Sec. 3.1 Eq. (5)) against the fp64 oracle's single-sequence prefill, run
sequence by sequence over the same packed inputs: the absorbed form (d_c 128,
16 heads) and the explicit form (the 128-head d_c 512 layer and other shapes)."""
import numpy as np
import pytest
import torch

from oracle import eg_mla_oracle as orc
from paper_2509_16686_amd import binding as B
from paper_2509_16686_amd import workloads as W
from parity import assert_close, say

pytestmark = pytest.mark.gpu

LAYER = W.WORKLOADS[1]  # 16 heads, d_c 128, d_r 64, bf16
WIDE = W.WORKLOADS[4].replace(vocab=8192)  # 128 heads, d_c 512, d_r 64, bf16 (a smaller gate table)


def run_varlen(pb):
    wl = pb.wl
    T = int(pb.cu_seqlens[-1])
    dims = B.dims_for(wl)
    ws = B.alloc_workspace(B.prefill_varlen_workspace_size(dims, T))
    out = torch.empty((T, wl.heads, wl.v_head_dim), dtype=torch.bfloat16, device="cuda")
    st = wl.dtype
    B.prefill_varlen(dims, B.to_device_tensor(pb.cu_seqlens, "int"), B.to_device_tensor(pb.q, st),
                     B.to_device_tensor(pb.latent, st), B.to_device_tensor(pb.token_ids, "int"),
                     B.to_device_tensor(pb.gate_table, st), B.to_device_tensor(pb.w_uk, st),
                     B.to_device_tensor(pb.w_uv, st), ws, out)
    torch.cuda.synchronize()
    return B.out_to_f64(out)


def oracle_varlen(pb):
    wl = pb.wl
    parts = []
    for b in range(len(pb.cu_seqlens) - 1):
        s = pb.sequence(b)
        if s.q.shape[0] == 0:
            continue
        parts.append(orc.prefill(s.q, s.latent, s.token_ids, s.gate_table, s.w_uk, s.w_uv, latent_dim=wl.latent_dim,
                                 head_dim=wl.head_dim, rope_dim=wl.rope_dim, storage=wl.dtype))
    return np.concatenate(parts, 0)


@pytest.mark.parametrize("lens", [
    [1],                          # one token: the tile holds a single key
    [16],                         # one full block
    [17, 15],                     # a block straddling two sequences
    [300],                        # several tiles, ragged last tile
    [5, 0, 64, 1, 130, 0, 33],    # empty sequences, exact tiles, short ones
    [1000, 3, 700],               # long sequences around a short one
])
def test_prefill_varlen_matches_oracle(gpu, lens):
    pb = W.generate_prefill_batch(LAYER, lens, seed=61)
    say(f"prefill_varlen lens={lens}")
    got = run_varlen(pb)
    ref = oracle_varlen(pb)
    # short sequences give outputs of a few units: the bf16 bound scales with max|ref|
    assert_close(got, ref, "bf16", f"prefill varlen {lens}")


def test_prefill_varlen_peaked(gpu):
    # queries x 8 (exact in bf16): rows dominated by a few keys, where a bf16 gated latent
    # or query alone would exceed the element-wise bound
    pb = W.generate_prefill_batch(LAYER, [300, 77], seed=68)
    pb.q = W.f32_to_bf16_bits((orc.widen(pb.q, "bf16") * 8.0).astype(np.float32))
    say("prefill_varlen peaked q x8")
    assert_close(run_varlen(pb), oracle_varlen(pb), "bf16", "prefill varlen q x8")


def test_prefill_varlen_equals_prefill_ref(gpu):
    # the same sequence through the MFMA path and the plain explicit-form kernels
    wl = LAYER
    pb = W.generate_prefill_batch(wl, [257], seed=62)
    say("prefill_varlen vs prefill_ref T=257")
    got = run_varlen(pb)
    T = 257
    dims = B.dims_for(wl)
    ws = B.alloc_workspace(B.prefill_workspace_size(dims, T))
    out = torch.empty((T, wl.heads, wl.v_head_dim), dtype=torch.bfloat16, device="cuda")
    B.prefill_ref(dims, B.to_device_tensor(pb.q, "bf16"), B.to_device_tensor(pb.latent, "bf16"),
                  B.to_device_tensor(pb.token_ids, "int"), B.to_device_tensor(pb.gate_table, "bf16"),
                  B.to_device_tensor(pb.w_uk, "bf16"), B.to_device_tensor(pb.w_uv, "bf16"), ws, out)
    torch.cuda.synchronize()
    assert_close(got, B.out_to_f64(out), "bf16", "varlen vs ref")


def test_prefill_varlen_long_sequence_sampled(gpu):
    # 4096 tokens (the decode workload's context): every 97th row against the oracle's causal row
    wl = LAYER
    T = 4096
    pb = W.generate_prefill_batch(wl, [T], seed=63)
    say("prefill_varlen T=4096 sampled rows")
    got = run_varlen(pb)
    rows = np.arange(0, T, 97)
    rows = np.append(rows, T - 1)
    # row t of a causal prefill is the decode of the prefix 0..t with query q_t
    ref = orc.decode(pb.q[rows], pb.latent, pb.token_ids, pb.gate_table, pb.w_uk, pb.w_uv,
                     (rows + 1).astype(np.int32), latent_dim=wl.latent_dim, head_dim=wl.head_dim,
                     rope_dim=wl.rope_dim, storage="bf16", page_table=np.zeros((len(rows), T // 64), np.int32)
                     + np.arange(T // 64, dtype=np.int32)[None, :], page_size=64, max_pages=T // 64)
    assert_close(got[rows], ref, "bf16", "prefill varlen T=4096 sampled")


@pytest.mark.parametrize("lens", [
    [1],                          # one token: the tile holds a single key
    [17, 15],                     # a block straddling two sequences
    [300],                        # several tiles, ragged last tile and block
    [129, 127],                   # sequences straddling a 128-token block by one
    [5, 0, 64, 1, 130, 0, 33],    # empty sequences, exact tiles, short ones
    [700, 3, 300],                # long sequences around a short one
])
def test_prefill_varlen_explicit_matches_oracle(gpu, lens):
    # the 128-head d_c 512 layer: projection to fp16 K^C, V, then attention per head
    pb = W.generate_prefill_batch(WIDE, lens, seed=64)
    say(f"prefill_varlen explicit lens={lens}")
    assert_close(run_varlen(pb), oracle_varlen(pb), "bf16", f"prefill varlen explicit {lens}")


def test_prefill_varlen_explicit_peaked(gpu):
    # queries x 8 (exact in bf16): rows dominated by a few keys, where a key or value
    # rounded to bf16 alone would exceed the element-wise bound
    pb = W.generate_prefill_batch(WIDE, [300, 77], seed=65)
    pb.q = W.f32_to_bf16_bits((orc.widen(pb.q, "bf16") * 8.0).astype(np.float32))
    say("prefill_varlen explicit peaked q x8")
    assert_close(run_varlen(pb), oracle_varlen(pb), "bf16", "prefill varlen explicit q x8")


@pytest.mark.parametrize("form", ["absorbed", "explicit"])
def test_prefill_varlen_out_of_range_ids_clamped(gpu, form):
    # ids below 0 or at least V select the first or last gate row (the gate
    # passes clamp them); the oracle is fed the clamped ids
    wl = LAYER if form == "absorbed" else WIDE
    pb = W.generate_prefill_batch(wl, [130, 61], seed=67)
    bad = np.random.default_rng(67).choice(len(pb.token_ids), 24, replace=False)
    pb.token_ids[bad[:12]] = -3
    pb.token_ids[bad[12:]] = wl.vocab + 7
    say(f"prefill_varlen {form}: out-of-range ids")
    got = run_varlen(pb)
    pb.token_ids = np.clip(pb.token_ids, 0, wl.vocab - 1).astype(np.int32)
    assert_close(got, oracle_varlen(pb), "bf16", f"prefill varlen {form} clamped ids")


@pytest.mark.parametrize("heads,dc,lens", [(8, 256, [200, 57]), (16, 512, [150]), (32, 128, [97, 64])])
def test_prefill_varlen_explicit_other_shapes(gpu, heads, dc, lens):
    wl = WIDE.replace(heads=heads, latent_dim=dc, gate_dim=dc)
    pb = W.generate_prefill_batch(wl, lens, seed=66)
    say(f"prefill_varlen explicit H={heads} d_c={dc} lens={lens}")
    assert_close(run_varlen(pb), oracle_varlen(pb), "bf16", f"prefill varlen explicit H{heads} dc{dc}")


def test_prefill_varlen_explicit_long_sequence_sampled(gpu):
    # 4096 tokens of the 128-head layer: every 97th row against the oracle's causal row
    wl = WIDE
    T = 4096
    pb = W.generate_prefill_batch(wl, [T], seed=67)
    say("prefill_varlen explicit T=4096 sampled rows")
    got = run_varlen(pb)
    rows = np.append(np.arange(0, T, 97), T - 1)
    ref = orc.decode(pb.q[rows], pb.latent, pb.token_ids, pb.gate_table, pb.w_uk, pb.w_uv,
                     (rows + 1).astype(np.int32), latent_dim=wl.latent_dim, head_dim=wl.head_dim,
                     rope_dim=wl.rope_dim, storage="bf16", page_table=np.zeros((len(rows), T // 64), np.int32)
                     + np.arange(T // 64, dtype=np.int32)[None, :], page_size=64, max_pages=T // 64)
    assert_close(got[rows], ref, "bf16", "prefill varlen explicit T=4096 sampled")
