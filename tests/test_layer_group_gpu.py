"""Layer grouping (App. H): the layers of a group share one cached [c | k^R]
row and token id per token.  The group's first layer appends the new tokens;
every layer decodes the shared rows with its own query, W_UK, W_UV and gate
table through eg_mla_decode.  Each layer is compared with the fp64 oracle, and
the shared cache must come out of the decodes unchanged."""
import numpy as np
import pytest
import torch

from oracle import eg_mla_oracle as orc
from paper_2509_16686_amd import binding as B
from paper_2509_16686_amd import workloads as W
from parity import assert_close, say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("wl,group", [
    (W.WORKLOADS[1].replace(name="group3_dc128", batch=3, seq_len=None, seq_len_range=(1, 700), paged=True, seed=95), 3),
    (W.WORKLOADS[4].replace(name="group2_dc512", batch=2, seq_len_range=(100, 600), seed=96), 2),
])
def test_layer_group_appends_once_and_every_layer_decodes(gpu, wl, group):
    layers = W.generate_layer_group(wl, group)
    base = layers[0]
    dims = B.dims_for(wl)
    shared = B.stage_decode(base)                 # the group's cache, ids, lengths and pages on the device
    # the first layer appends the current token of every sequence (position L - 1) into the shared rows
    lens = base.seq_lens.astype(np.int64)
    slots = np.array([base.slot(b, int(lens[b]) - 1) for b in range(wl.batch)], dtype=np.int32)
    ap = W.generate_append(wl, wl.batch, base.num_rows, seed=97)
    ap.positions[:] = (lens - 1).astype(np.int32)
    say(f"layer group {wl.name}: append by the first layer, then {group} layers decode")
    B.append(dims, B.to_device_tensor(ap.x, "bf16"), B.to_device_tensor(ap.token_ids, "int"),
             B.to_device_tensor(ap.positions, "int"), B.to_device_tensor(slots, "int"),
             B.to_device_tensor(ap.w_dkv, "bf16"), B.to_device_tensor(ap.kv_norm_w, "bf16"), shared.cache, shared.ids)
    torch.cuda.synchronize()
    cache_before = shared.cache.clone()
    got = []
    for lay in layers:
        dd = B.stage_decode(lay)
        dd.cache, dd.ids = shared.cache, shared.ids    # every layer reads the one shared cache
        B.run_decode(dd)
        torch.cuda.synchronize()
        got.append(B.out_to_f64(dd.out))
    assert torch.equal(shared.cache, cache_before), "a decode wrote to the shared cache"
    # the oracle's own append of the same tokens, rounded to the storage type, then every layer
    rows = orc.append(ap.x, ap.w_dkv, ap.kv_norm_w, ap.positions, latent_dim=wl.latent_dim, rope_dim=wl.rope_dim,
                      storage="bf16")
    base.latent_cache[slots] = W.f32_to_bf16_bits(rows.astype(np.float32))
    base.token_ids[slots] = ap.token_ids
    refs = orc.decode_layer_group(base.latent_cache, base.token_ids, base.seq_lens,
                                  [(l.q, l.gate_table, l.w_uk, l.w_uv) for l in layers], latent_dim=wl.latent_dim,
                                  head_dim=wl.head_dim, rope_dim=wl.rope_dim, storage="bf16",
                                  page_table=base.page_table, page_size=wl.page_size, max_pages=base.max_pages)
    for k, (g, r) in enumerate(zip(got, refs)):
        assert_close(g, r, "bf16", f"{wl.name} layer {k}")
