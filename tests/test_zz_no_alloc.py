"""eg_mla_decode_noalloc (no workspace argument: the library's static scratch
array) against eg_mla_decode on the same inputs, through the C ABI: the same
kernels and plan, so the outputs must agree bit for bit.  Calls in a row with
shrinking inputs check that the scratch array's stale contents from a larger
call do not leak into a smaller one."""
import numpy as np
import pytest
import torch

from paper_2509_16686_amd import binding as B
from paper_2509_16686_amd import workloads as W
from parity import assert_close, oracle_decode, say

pytestmark = pytest.mark.gpu


def decode_both(inp):
    dd = B.stage_decode(inp)
    B.run_decode(dd)                      # eg_mla_decode with a workspace of its own
    torch.cuda.synchronize()
    with_ws = B.out_to_f64(dd.out).copy()
    out = torch.full_like(dd.out, float("nan"))
    B.decode_noalloc(dd.dims, dd.q, dd.cache, dd.ids, dd.gate, dd.w_uk, dd.w_uv, dd.seq_lens, dd.page_table,
                     dd.max_pages, out)
    torch.cuda.synchronize()
    return with_ws, B.out_to_f64(out)


def test_noalloc_matches_decode_calls_in_a_row(gpu):
    cases = [
        W.WORKLOADS[1],                                                        # B32 L4096: 2.5 MB of scratch
        W.WORKLOADS[1].replace(name="noalloc_small", batch=5, seq_len=None, seq_len_range=(1, 700), paged=True,
                               seed=91),                                       # smaller, ragged, paged
        W.WORKLOADS[0],                                                        # fp32, VALU path
    ]
    for wl in cases:
        inp = W.generate(wl)
        need = B.decode_workspace_size(B.dims_for(wl), wl.batch, inp.max_pages)
        assert 0 < need <= B.NOALLOC_SCRATCH_BYTES
        say(f"decode_noalloc {wl.name} B={wl.batch} (plan workspace {need} bytes)")
        with_ws, noalloc = decode_both(inp)
        assert np.all(np.isfinite(noalloc))
        assert np.array_equal(with_ws, noalloc), f"{wl.name}: outputs differ"
        if wl.batch <= 8:
            assert_close(noalloc, oracle_decode(inp), wl.dtype, f"noalloc {wl.name}")


def test_noalloc_rejects_a_plan_beyond_the_scratch(gpu):
    # the 128-head d_c 512 layer at batch 64 needs far more than 32 MiB of partials
    wl = W.WORKLOADS[4].replace(batch=64, seq_len_range=(512, 1024))
    dims = B.dims_for(wl)
    assert B.decode_workspace_size(dims, 64, 256) > B.NOALLOC_SCRATCH_BYTES
    q = torch.zeros((64, wl.heads, wl.qk_dim), dtype=torch.bfloat16, device="cuda")
    cache = torch.zeros((256, wl.row_dim), dtype=torch.bfloat16, device="cuda")  # never read: rejected first
    ids = torch.zeros(cache.shape[0], dtype=torch.int32, device="cuda")
    out = torch.zeros((64, wl.heads, wl.v_head_dim), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(B.EgMlaError) as e:
        B.decode_noalloc(dims, q, cache, ids, cache, q, q, ids[:64], None, 256, out)
    assert e.value.status == B.ERR_WORKSPACE
