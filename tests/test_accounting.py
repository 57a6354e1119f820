"""The KV-cache calculator against the per-token counts the paper prints (App. F, Table 5)."""
import json
import os

import numpy as np

from paper_2509_16686_amd import accounting as A
from paper_2509_16686_amd import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden", "kv_cache_per_token.json")


def _printed_k(s):
    return float(s.rstrip("K")) * 1000


def test_app_f_elements_per_token():
    g = json.load(open(GOLD))
    got = {}
    for row in g["rows"]:
        n = A.kv_cache_elements_per_token(row["mechanism"], layers=g["layers"], heads=row.get("heads", 0),
                                          head_dim=row.get("head_dim", 0), latent_dim=row.get("latent_dim", 0),
                                          rope_dim=0 if row["mechanism"] == "mha" else g["rope_dim"])
        # the paper prints thousands rounded to two decimals
        assert round(n / 1000, 2) == _printed_k(row["printed"]) / 1000, row
        got[row["model"]] = n
    red = g["reductions"]
    kv64, mla, mha, kv16 = got["EG-MLA-Base-kv64"], got["MLA-Base"], got["MHA-Base"], got["EG-MLA-Base-kv16"]
    # 59.9 % is what the *rounded* printed counts give; the exact counts give 60.0 %
    assert round(100 * (1 - 1.54 / 3.84), 1) == red["kv64_vs_mla_percent_printed"]
    assert round(100 * (1 - kv64 / mla), 1) == 60.0
    assert int(100 * (1 - kv64 / mha) * 10) / 10 == red["kv64_vs_mha_percent_printed"]
    assert round(100 * (1 - kv16 / mha), 1) == red["kv16_vs_mha_percent_printed"]


def test_table5_other_mechanisms():
    assert A.kv_cache_elements_per_token("gqa", layers=2, groups=4, head_dim=8) == 2 * 4 * 8 * 2
    assert A.kv_cache_elements_per_token("mqa", layers=3, head_dim=8) == 2 * 8 * 3
    assert A.kv_cache_elements_per_token("eg-mla", layers=1, latent_dim=256, rope_dim=64, compression=4) == 128


def test_layer1b_decode_bytes():
    wl = W.WORKLOADS[1]
    N = wl.batch * wl.seq_len
    t = A.decode_bytes(batch=wl.batch, heads=wl.heads, head_dim=wl.head_dim, v_head_dim=wl.v_head_dim,
                       latent_dim=wl.latent_dim, rope_dim=wl.rope_dim, elem_bytes=2, total_tokens=N,
                       distinct_ids=46_600)
    assert t.cache_rows == N * 384 == 50_331_648
    assert t.token_ids == N * 4
    # expected distinct rows of V uniform draws over N tokens: V (1 - exp(-N/V))
    exp_unique = wl.vocab * (1 - np.exp(-N / wl.vocab))
    assert abs(exp_unique - 46_600) / 46_600 < 0.01
    assert 63e6 < t.total < 65e6


def test_flops_count():
    f = A.decode_flops(batch=1, heads=1, head_dim=2, v_head_dim=2, latent_dim=2, rope_dim=0, total_tokens=1)
    # score 2 + value 2 MACs, absorb 4, up 4, gate 1 -> 13 MACs
    assert f == 2 * (1 * (2 + 2) + 4 + 4 + 1)


def test_layer_group_cache_rows():
    # App. H: lgz consecutive layers share one cached row; lgz = 1 is the App. F count
    g = json.load(open(GOLD))
    kv64 = A.kv_cache_elements_per_token("eg-mla", layers=12, latent_dim=64, rope_dim=64)
    assert round(kv64 / 1000, 2) == 1.54                                   # App. F, EG-MLA-Base-kv64
    assert A.kv_cache_elements_per_token("eg-mla", layers=12, latent_dim=64, rope_dim=64, layer_group=1) == kv64
    assert A.kv_cache_elements_per_token("eg-mla", layers=12, latent_dim=64, rope_dim=64, layer_group=2) == kv64 // 2
    assert A.kv_cache_elements_per_token("eg-mla", layers=12, latent_dim=64, rope_dim=64, layer_group=3) == kv64 // 3
    # a last group shorter than lgz still keeps its row: 24 layers, lgz 5 -> 5 rows
    assert A.kv_cache_elements_per_token("mla", layers=24, latent_dim=128, rope_dim=64, layer_group=5) == 5 * 192
    assert g["layers"] == 12
    # bytes of this library's cache (bf16 rows + int32 id) for the 24-layer 1.2B-class model
    assert A.cache_bytes_per_token(layers=24, latent_dim=128, rope_dim=64, elem_bytes=2) == 24 * 388
    assert A.cache_bytes_per_token(layers=24, latent_dim=128, rope_dim=64, elem_bytes=2, layer_group=2) == 12 * 388
    assert A.cache_bytes_per_token(layers=24, latent_dim=128, rope_dim=64, elem_bytes=2, layer_group=3) == 8 * 388
