"""GPU parity of eg_mla_prefill_ref and eg_mla_append against the fp64 oracle."""
import numpy as np
import pytest
import torch

from oracle import eg_mla_oracle as orc
from paper_2509_16686_amd import binding as B
from paper_2509_16686_amd import workloads as W
from parity import assert_close, oracle_decode, say

pytestmark = pytest.mark.gpu


def stage(a, storage):
    return B.to_device_tensor(a, storage)


def run_append(entry, dims, x, token_ids, positions, slots, w_dkv, kv_norm_w, cache, idc):
    """eg_mla_append, or eg_mla_append_ws with a workspace of the size it asks for."""
    if entry == "append":
        B.append(dims, x, token_ids, positions, slots, w_dkv, kv_norm_w, cache, idc)
    else:
        ws = B.alloc_workspace(B.append_workspace_size(dims, int(x.shape[0]), int(x.shape[1])))
        B.append_ws(dims, x, token_ids, positions, slots, w_dkv, kv_norm_w, cache, idc, ws)


@pytest.mark.parametrize("wl,T", [(W.WORKLOADS[0], 128), (W.WORKLOADS[1], 300),
                                  (W.WORKLOADS[4].replace(heads=16), 130)])
def test_prefill_ref_matches_oracle(gpu, wl, T):
    pin = W.generate_prefill(wl, T)
    st = wl.dtype
    say(f"prefill_ref {wl.name} T={T}")
    dims = B.dims_for(wl)
    ws = B.alloc_workspace(B.prefill_workspace_size(dims, T))
    out = torch.empty((T, wl.heads, wl.v_head_dim), dtype=torch.bfloat16 if st == "bf16" else torch.float32,
                      device="cuda")
    B.prefill_ref(dims, stage(pin.q, st), stage(pin.latent, st), stage(pin.token_ids, "int"),
                  stage(pin.gate_table, st), stage(pin.w_uk, st), stage(pin.w_uv, st), ws, out)
    torch.cuda.synchronize()
    ref = orc.prefill(pin.q, pin.latent, pin.token_ids, pin.gate_table, pin.w_uk, pin.w_uv, latent_dim=wl.latent_dim,
                      head_dim=wl.head_dim, rope_dim=wl.rope_dim, storage=st)
    assert_close(B.out_to_f64(out), ref, st, f"prefill {wl.name}")


def test_decode_row_equals_prefill_row(gpu):
    """Decode of the prefix 0..t with query q_t equals prefill row t (two device paths)."""
    wl = W.WORKLOADS[1].replace(batch=1, seq_len=200)
    pin = W.generate_prefill(wl, 200)
    dims = B.dims_for(wl)
    ws = B.alloc_workspace(B.prefill_workspace_size(dims, 200))
    pre = torch.empty((200, wl.heads, wl.v_head_dim), dtype=torch.bfloat16, device="cuda")
    q = stage(pin.q, "bf16")
    lat = stage(pin.latent, "bf16")
    ids = stage(pin.token_ids, "int")
    gate, wk, wv = stage(pin.gate_table, "bf16"), stage(pin.w_uk, "bf16"), stage(pin.w_uv, "bf16")
    say("prefill vs decode rows")
    B.prefill_ref(dims, q, lat, ids, gate, wk, wv, ws, pre)
    # decode: each row t is one "sequence" of length t+1 over the same contiguous rows
    rows = [0, 1, 31, 32, 63, 64, 199]
    qd = q[rows].contiguous()
    lens = torch.tensor([t + 1 for t in rows], dtype=torch.int32, device="cuda")
    # contiguous layout: sequence b starts at row b * capacity, so give every sequence its own copy
    P = wl.page_size
    cap = 256
    cache = torch.zeros((len(rows) * cap, lat.shape[1]), dtype=torch.bfloat16, device="cuda")
    idc = torch.zeros((len(rows) * cap,), dtype=torch.int32, device="cuda")
    for i in range(len(rows)):
        cache[i * cap:i * cap + 200] = lat
        idc[i * cap:i * cap + 200] = ids
    out = torch.empty((len(rows), wl.heads, wl.v_head_dim), dtype=torch.bfloat16, device="cuda")
    wsd = B.alloc_workspace(B.decode_workspace_size(dims, len(rows), cap // P))
    B.decode(dims, qd, cache, idc, gate, wk, wv, lens, None, cap // P, wsd, out)
    torch.cuda.synchronize()
    a = B.out_to_f64(out)
    b = B.out_to_f64(pre)[rows]
    assert_close(a, b, "bf16", "decode vs prefill")


@pytest.mark.parametrize("entry", ["append", "append_ws"])
@pytest.mark.parametrize("wl,norm", [(W.WORKLOADS[1], True), (W.WORKLOADS[1], False), (W.WORKLOADS[4], True),
                                     (W.WORKLOADS[4], False), (W.WORKLOADS[0], True)])
def test_append_matches_oracle(gpu, wl, norm, entry):
    n, rows = 37, 256
    ap = W.generate_append(wl, n, rows, with_norm=norm)
    st = wl.dtype
    dims = B.dims_for(wl)
    dt = torch.bfloat16 if st == "bf16" else torch.float32
    cache = torch.zeros((rows, wl.row_dim), dtype=dt, device="cuda")
    idc = torch.full((rows,), -7, dtype=torch.int32, device="cuda")
    slots = ap.slots.copy()
    slots[5] = rows + 3          # out of range: skipped
    say(f"{entry} {wl.name} n={n} norm={norm}")
    run_append(entry, dims, stage(ap.x, st), stage(ap.token_ids, "int"), stage(ap.positions, "int"),
               stage(slots, "int"), stage(ap.w_dkv, st), None if ap.kv_norm_w is None else stage(ap.kv_norm_w, st),
               cache, idc)
    torch.cuda.synchronize()
    ref = orc.append(ap.x, ap.w_dkv, ap.kv_norm_w, ap.positions, latent_dim=wl.latent_dim, rope_dim=wl.rope_dim,
                     storage=st)
    got = B.out_to_f64(cache)
    ids = idc.cpu().numpy()
    keep = [i for i in range(n) if i != 5]
    g = got[slots[keep]]
    r = ref[keep]
    # one rounding of an fp32 result to the storage type: within one unit in the last place
    ulp = 2.0 ** -7 if st == "bf16" else 2.0 ** -22
    assert np.all(np.abs(g - r) <= ulp * np.abs(r) + 1e-5), float(np.max(np.abs(g - r) - ulp * np.abs(r)))
    np.testing.assert_array_equal(ids[slots[keep]], ap.token_ids[keep])
    untouched = np.setdiff1d(np.arange(rows), slots[keep])
    assert np.all(got[untouched] == 0) and np.all(ids[untouched] == -7)


def test_append_then_decode(gpu):
    """Rows written by append decode like rows the oracle writes itself."""
    wl = W.WORKLOADS[1].replace(batch=2, seq_len=70)
    inp = W.generate(wl)
    dims = B.dims_for(wl)
    dd = B.stage_decode(inp)
    ap = W.generate_append(wl, 2, inp.num_rows)
    # overwrite the last token of each sequence through append
    slots = np.array([inp.slot(0, 69), inp.slot(1, 69)], dtype=np.int32)
    say("append then decode")
    B.append(dims, stage(ap.x, "bf16"), stage(ap.token_ids, "int"), stage(ap.positions, "int"), stage(slots, "int"),
             stage(ap.w_dkv, "bf16"), stage(ap.kv_norm_w, "bf16"), dd.cache, dd.ids)
    B.run_decode(dd)
    torch.cuda.synchronize()
    got = B.out_to_f64(dd.out)
    # the reference rows come from the oracle's own append, rounded to the storage type
    rows = orc.append(ap.x, ap.w_dkv, ap.kv_norm_w, ap.positions, latent_dim=wl.latent_dim, rope_dim=wl.rope_dim,
                      storage="bf16")
    inp.latent_cache[slots] = W.f32_to_bf16_bits(rows.astype(np.float32))
    inp.token_ids[slots] = ap.token_ids
    assert_close(got, oracle_decode(inp), "bf16", "append then decode")


@pytest.mark.parametrize("wi,entry,n", [(1, "append", 1), (1, "append", 31), (1, "append", 33), (1, "append", 8192),
                                        (1, "append", 8193), (1, "append", 9000), (1, "append_ws", 1),
                                        (1, "append_ws", 32), (1, "append_ws", 33), (1, "append_ws", 2048),
                                        (1, "append_ws", 2049), (1, "append_ws", 300), (4, "append_ws", 1),
                                        (4, "append_ws", 64), (4, "append_ws", 97), (4, "append_ws", 255),
                                        (4, "append_ws", 256), (4, "append_ws", 512), (4, "append_ws", 3001),
                                        (4, "append_ws", 9000)])
def test_append_token_counts(gpu, wi, entry, n):
    # the d_c 128 / d_r 64 layer's one-pass MFMA append: hidden split over the
    # waves up to 8192 tokens, 128 tokens per work-group above; the two-pass
    # append of both bf16 layers (d_c 128 at hidden 2048, d_c 512 at hidden
    # 7168), its first pass from global memory below 256 tokens and LDS-tiled
    # from 256, from 28 slices down to one; ragged last tiles
    wl = W.WORKLOADS[wi]
    rows = n + 300
    ap = W.generate_append(wl, n, rows, with_norm=True, seed=71 + n)
    dims = B.dims_for(wl)
    cache = torch.zeros((rows, wl.row_dim), dtype=torch.bfloat16, device="cuda")
    idc = torch.full((rows,), -7, dtype=torch.int32, device="cuda")
    say(f"{entry} {wl.name} n={n}")
    run_append(entry, dims, stage(ap.x, "bf16"), stage(ap.token_ids, "int"), stage(ap.positions, "int"),
               stage(ap.slots, "int"), stage(ap.w_dkv, "bf16"), stage(ap.kv_norm_w, "bf16"), cache, idc)
    torch.cuda.synchronize()
    ref = orc.append(ap.x, ap.w_dkv, ap.kv_norm_w, ap.positions, latent_dim=wl.latent_dim, rope_dim=wl.rope_dim,
                     storage="bf16")
    got = B.out_to_f64(cache)[ap.slots]
    assert np.all(np.abs(got - ref) <= 2.0 ** -7 * np.abs(ref) + 1e-5), float(np.max(np.abs(got - ref)))
    np.testing.assert_array_equal(idc.cpu().numpy()[ap.slots], ap.token_ids)
