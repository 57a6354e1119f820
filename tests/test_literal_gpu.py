"""GPU parity of eg_mla_decode_literal (the paper-literal gate of Sec. 3.1
Eq. (2)-(5): gate on the up-projected keys and values, LayerNorm over all
heads' dims, and the two ablations) against the fp64 oracle."""
import numpy as np
import pytest
import torch

from oracle import eg_mla_oracle as orc
from paper_2509_16686_amd import binding as B
from paper_2509_16686_amd import workloads as W
from parity import assert_close, say

pytestmark = pytest.mark.gpu

MODES = [(0, "mul", True), (B.LITERAL_NO_LN, "mul", False), (B.LITERAL_ADD, "add", True),
         (B.LITERAL_NO_LN | B.LITERAL_ADD, "add", False)]


def run_literal(inp, lg, flags):
    dd = B.stage_decode(inp)
    ws = B.alloc_workspace(B.decode_literal_workspace_size(dd.dims, int(dd.q.shape[0]), dd.max_pages))
    gate = B.to_device_tensor(lg.gate_full, "bf16")
    lw, lb = B.to_device_tensor(lg.ln_w, "bf16"), B.to_device_tensor(lg.ln_b, "bf16")
    B.decode_literal(dd, gate, lw, lb, flags, ws)
    torch.cuda.synchronize()
    return B.out_to_f64(dd.out)


def run_literal_storage(inp, lg, flags):
    """As run_literal, with the gate and LayerNorm arrays in the workload's storage type."""
    st = inp.wl.dtype
    dd = B.stage_decode(inp)
    ws = B.alloc_workspace(B.decode_literal_workspace_size(dd.dims, int(dd.q.shape[0]), dd.max_pages))
    gate = B.to_device_tensor(lg.gate_full, st)
    lw, lb = B.to_device_tensor(lg.ln_w, st), B.to_device_tensor(lg.ln_b, st)
    B.decode_literal(dd, gate, lw, lb, flags, ws)
    torch.cuda.synchronize()
    return B.out_to_f64(dd.out)


def oracle_literal(inp, lg, mode, use_ln):
    wl = inp.wl
    return orc.decode_literal(inp.q, inp.latent_cache, inp.token_ids, lg.gate_full, inp.w_uk, inp.w_uv, lg.ln_w,
                              lg.ln_b, inp.seq_lens, latent_dim=wl.latent_dim, head_dim=wl.head_dim,
                              rope_dim=wl.rope_dim, storage=wl.dtype, page_table=inp.page_table,
                              page_size=wl.page_size, max_pages=inp.max_pages, mode=mode, use_ln=use_ln)


@pytest.mark.parametrize("flags,mode,use_ln", MODES, ids=["mul_ln", "mul", "add_ln", "add"])
def test_literal_contiguous(gpu, flags, mode, use_ln):
    wl = W.WORKLOADS[1].replace(batch=3, seq_len=300, vocab=2000, seed=81)
    inp = W.generate(wl)
    lg = W.generate_literal_gate(wl)
    say(f"literal decode contiguous mode={mode} ln={use_ln}")
    assert_close(run_literal(inp, lg, flags), oracle_literal(inp, lg, mode, use_ln), "bf16",
                 f"literal {mode} ln={use_ln}")


def test_literal_paged_ragged_with_empty(gpu):
    wl = W.WORKLOADS[1].replace(batch=5, seq_len=None, seq_len_range=(1, 700), paged=True, vocab=3000, seed=82)
    inp = W.generate(wl, seq_lens=np.array([1, 128, 0, 129, 700]))
    lg = W.generate_literal_gate(wl)
    say("literal decode paged ragged lens 1,128,0,129,700")
    got = run_literal(inp, lg, 0)
    ref = oracle_literal(inp, lg, "mul", True)
    assert np.all(got[2] == 0)
    assert_close(got, ref, "bf16", "literal paged ragged")


@pytest.mark.parametrize("heads,lens,flags,mode,use_ln", [
    (4, [33000, 257], 0, "mul", True),                     # past 32768 tokens: 258 tiles merged
    (20, [300, 1], B.LITERAL_ADD, "add", True),            # 20 heads: tile state beyond 80 KB of LDS
    (1, [129, 64], B.LITERAL_NO_LN, "mul", False),          # a single head
    (3, [260, 5], 0, "mul", True),                          # odd head count: a pair of heads, then the last alone
], ids=["h4_l33000", "h20", "h1", "h3"])
def test_literal_head_counts_and_long_context(gpu, heads, lens, flags, mode, use_ln):
    wl = W.WORKLOADS[1].replace(batch=len(lens), heads=heads, seq_len=None, seq_len_range=(1, max(lens)),
                                vocab=1500, seed=83)
    inp = W.generate(wl, seq_lens=np.array(lens))
    lg = W.generate_literal_gate(wl)
    say(f"literal decode H={heads} lens {lens} mode={mode} ln={use_ln}")
    assert_close(run_literal(inp, lg, flags), oracle_literal(inp, lg, mode, use_ln), "bf16",
                 f"literal H={heads}")


def test_literal_layernorm_offset_rows(gpu):
    # additive gate rows centred at 100: every gated row has a mean about 100
    # times its spread, where moments taken as m2 - m1^2 in fp32 lose the
    # variance; the LayerNorm must still match the oracle's two-pass moments
    wl = W.WORKLOADS[1].replace(batch=3, seq_len=None, seq_len_range=(1, 600), vocab=1000, seed=84)
    inp = W.generate(wl, seq_lens=np.array([600, 129, 1]))
    lg = W.generate_literal_gate(wl, center=100.0)
    say("literal decode additive gate centred at 100, LayerNorm")
    assert_close(run_literal(inp, lg, B.LITERAL_ADD), oracle_literal(inp, lg, "add", True), "bf16",
                 "literal add, offset rows")


def test_literal_full_size_sampled(gpu):
    # the bench's workload and launch (B32 H16 L4096, 50304 gate rows, LayerNorm);
    # the oracle recomputes two sampled sequences on their own, from their cache
    # rows and the gate rows their ids select
    wl = W.WORKLOADS[1]
    inp = W.generate(wl)
    lg = W.generate_literal_gate(wl)
    say(f"literal decode full size {wl.name}, sampled sequences")
    got = run_literal(inp, lg, 0)
    P = wl.page_size
    for b in (0, wl.batch - 1):
        L = int(inp.seq_lens[b])
        j = np.arange(L)
        if inp.page_table is None:
            rows = b * inp.max_pages * P + j
        else:
            rows = inp.page_table[b, j // P].astype(np.int64) * P + j % P
        uniq, inv = np.unique(inp.token_ids[rows], return_inverse=True)
        ref = orc.decode_literal(inp.q[b:b + 1], inp.latent_cache[rows], inv.astype(np.int32), lg.gate_full[uniq],
                                 inp.w_uk, inp.w_uv, lg.ln_w, lg.ln_b, np.array([L], dtype=np.int32),
                                 latent_dim=wl.latent_dim, head_dim=wl.head_dim, rope_dim=wl.rope_dim,
                                 storage=wl.dtype, page_table=None, page_size=P, max_pages=-(-L // P), mode="mul",
                                 use_ln=True)
        assert_close(got[b:b + 1], ref, "bf16", f"literal full size, sequence {b}")


@pytest.mark.parametrize("flags,mode,use_ln", MODES, ids=["mul_ln", "mul", "add_ln", "add"])
def test_literal_generic_dc512_h128(gpu, flags, mode, use_ln):
    # the 128-head d_c 512 layer (paged, ragged): the generic kernel
    wl = W.WORKLOADS[4].replace(batch=3, seq_len_range=(1, 300), vocab=500, seed=85)
    inp = W.generate(wl, seq_lens=np.array([300, 129, 1]))
    lg = W.generate_literal_gate(wl)
    say(f"literal decode generic H128 d_c512 mode={mode} ln={use_ln}")
    assert_close(run_literal_storage(inp, lg, flags), oracle_literal(inp, lg, mode, use_ln), "bf16",
                 f"literal generic d_c512 {mode} ln={use_ln}")


@pytest.mark.parametrize("case", ["fp32_tiny", "bf16_odd", "bf16_offset_rows"])
def test_literal_generic_shapes(gpu, case):
    # other layers: the tiny fp32 one (no RoPE part), a bf16 one with d_h != d_v and
    # a short latent, and additive gate rows centred at 100 (|mu| ~ 100 sigma)
    if case == "fp32_tiny":
        wl = W.WORKLOADS[0].replace(batch=3, seq_len=None, seq_len_range=(1, 300), seed=86)
        lens, flags, mode, use_ln, center = [300, 0, 77], 0, "mul", True, 1.0
    else:
        wl = W.WORKLOADS[1].replace(heads=5, head_dim=64, v_head_dim=48, latent_dim=96, gate_dim=96, rope_dim=32,
                                    batch=2, seq_len=None, seq_len_range=(1, 260), paged=True, vocab=700, seed=87)
        lens = [260, 31]
        flags, mode, use_ln, center = ((0, "mul", True, 1.0) if case == "bf16_odd"
                                       else (B.LITERAL_ADD, "add", True, 100.0))
    inp = W.generate(wl, seq_lens=np.array(lens))
    lg = W.generate_literal_gate(wl, center=center)
    say(f"literal decode generic {case}")
    assert_close(run_literal_storage(inp, lg, flags), oracle_literal(inp, lg, mode, use_ln), wl.dtype,
                 f"literal generic {case}")
