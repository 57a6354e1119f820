"""The C-ABI library on the host: it loads, exports every symbol the header
declares, and rejects malformed calls before touching a device."""
import ctypes
import os
import re

import pytest

from paper_2509_16686_amd import binding as B

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "eg_mla.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(eg_mla_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    return B.lib()


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert len(names) >= 8
    for n in names:
        assert hasattr(L, n), n
    assert sorted(B.EXPORTS) == names


def dims(**kw):
    base = dict(num_heads=16, head_dim=128, v_head_dim=128, latent_dim=128, rope_dim=64, vocab_size=50304,
                page_size=64, dtype=B.BF16)
    base.update(kw)
    return B.make_dims(**base)


def test_status_strings(L):
    for s in range(5):
        assert B.status_string(s).startswith("EG_MLA_")
    assert "UNKNOWN" in B.status_string(77)


@pytest.mark.parametrize("kw,expect", [
    (dict(), B.OK),
    (dict(dtype=B.FP32, latent_dim=32, rope_dim=0, head_dim=32, v_head_dim=32, num_heads=4), B.OK),
    (dict(num_heads=0), B.ERR_INVALID_ARG),
    (dict(page_size=0), B.ERR_INVALID_ARG),
    (dict(dtype=7), B.ERR_INVALID_ARG),
    (dict(gate_dim=64), B.ERR_UNSUPPORTED),
    (dict(latent_dim=132), B.ERR_UNSUPPORTED),        # bf16 rows need 8-element multiples
    (dict(latent_dim=1024), B.ERR_UNSUPPORTED),       # beyond the LDS tile
    (dict(softmax_scale=float("nan")), B.ERR_INVALID_ARG),
])
def test_check_dims(L, kw, expect):
    assert B.check_dims(dims(**kw)) == expect


def test_workspace_size_queries(L):
    d = dims()
    auto = B.decode_workspace_size(d, 32, 64)
    assert auto > 32 * 16 * 192 * 4
    # explicit split of 512 tokens without id slices: 8 splits per 4096-token sequence
    # (the split kernel absorbs the query itself: one 8-byte stamp per split)
    ws512 = B.decode_workspace_size(d, 32, 64, B.make_plan(B.PATH_MFMA, 512, id_slices=1))
    stamps = 32 * 8 * 8
    expect = 32 * 16 * 192 * 4 + 32 * 8 * 16 * 2 * 4 + 32 * 8 * 16 * 128 * 4 + stamps
    assert expect <= ws512 <= expect + 4 * 256
    # ... and with 8 id slices: 8 partials per split
    ws512s = B.decode_workspace_size(d, 32, 64, B.make_plan(B.PATH_MFMA, 512, id_slices=8))
    expect = 32 * 16 * 192 * 4 + 32 * 64 * 16 * 2 * 4 + 32 * 64 * 16 * 128 * 4
    assert expect <= ws512s <= expect + 3 * 256
    # automatic: no id slices, 512-token splits (256 work items)
    assert auto == ws512
    # 8 id slices, automatic split: one 4096-token split per sequence, as many partials as above
    # (and a separate absorption kernel: no stamps)
    assert B.decode_workspace_size(d, 32, 64, B.make_plan(B.PATH_MFMA, 0, id_slices=8)) == ws512 - stamps
    assert B.decode_workspace_size(d, 32, 64, B.make_plan(B.PATH_MFMA, 4096)) > 0       # sliced kernel: up to 4096
    assert B.decode_workspace_size(d, 32, 64, B.make_plan(B.PATH_MFMA, 4128)) == 0
    assert B.decode_workspace_size(d, 32, 64, B.make_plan(B.PATH_MFMA, 0, id_slices=3)) == 0  # 0, 1 or 8 only
    assert B.decode_workspace_size(d, 32, 64, B.make_plan(B.PATH_MFMA, 100)) == 0   # not a multiple of 32
    assert B.decode_workspace_size(dims(num_heads=8), 1, 1, B.make_plan(B.PATH_MFMA, 0)) == 0  # no MFMA kernel
    assert B.decode_workspace_size(dims(gate_dim=1), 1, 1, None) == 0
    assert B.prefill_workspace_size(d, 100) >= 16 * 100 * (192 + 128) * 4


def _decode_call(L, d, ws_bytes=1 << 20, ptr=256, batch=2, max_pages=4, num_slots=512, page_table=None, plan=None):
    p = ctypes.c_void_p(ptr)
    args = (ctypes.byref(d), batch, p, p, p, p, p, p, p, page_table, max_pages, num_slots,
            ctypes.c_void_p(ptr) if ws_bytes else None, ws_bytes, p, None)
    if plan is None:
        return L.eg_mla_decode(*args)
    return L.eg_mla_decode_planned(*args, ctypes.byref(plan))


def test_decode_rejects_before_launch(L):
    d = dims()
    # null operands
    z = ctypes.c_void_p(0)
    st = L.eg_mla_decode(ctypes.byref(d), 2, None, z, z, z, z, z, z, None, 4, 512, None, 0, None, None)
    assert st == B.ERR_INVALID_ARG
    # workspace too small / missing
    assert _decode_call(L, d, ws_bytes=16) == B.ERR_WORKSPACE
    assert _decode_call(L, d, ws_bytes=0) == B.ERR_WORKSPACE
    # contiguous cache smaller than batch * capacity
    assert _decode_call(L, d, num_slots=100) == B.ERR_INVALID_ARG
    # misaligned operand pointers
    assert _decode_call(L, d, ptr=258) == B.ERR_INVALID_ARG
    # forced MFMA on a shape without an MFMA kernel
    assert _decode_call(L, dims(num_heads=8), plan=B.make_plan(B.PATH_MFMA, 0)) == B.ERR_UNSUPPORTED
    # bad plan values
    assert _decode_call(L, d, plan=B.make_plan(9, 0)) == B.ERR_INVALID_ARG
    assert _decode_call(L, d, plan=B.make_plan(B.PATH_AUTO, 33)) == B.ERR_INVALID_ARG
    # negative sizes
    assert _decode_call(L, d, batch=-1) == B.ERR_INVALID_ARG
    assert _decode_call(L, d, max_pages=-1) == B.ERR_INVALID_ARG
    # batch 0 is a valid no-op that touches nothing
    assert _decode_call(L, d, batch=0) == B.OK


def test_decode_noalloc_rejects_before_launch(L):
    z = ctypes.c_void_p(16 * 4096)
    def call(d, batch=2, max_pages=4, num_slots=1 << 20):
        return L.eg_mla_decode_noalloc(ctypes.byref(d), batch, z, z, z, z, z, z, z, None, max_pages, num_slots, z,
                                       None)
    # a plan beyond the scratch array: the 128-head d_c 512 layer at batch 64, 16384 tokens each
    big = dims(num_heads=128, latent_dim=512, gate_dim=512, vocab_size=129280)
    assert B.decode_workspace_size(big, 64, 256) > B.NOALLOC_SCRATCH_BYTES
    assert call(big, batch=64, max_pages=256) == B.ERR_WORKSPACE
    # the 16-head d_c 128 layer at batch 32, context 4096 fits
    assert B.decode_workspace_size(dims(), 32, 64) <= B.NOALLOC_SCRATCH_BYTES
    assert call(dims(num_heads=0)) == B.ERR_INVALID_ARG
    assert call(dims(), batch=-1) == B.ERR_INVALID_ARG
    assert call(dims(), max_pages=-1) == B.ERR_INVALID_ARG
    assert call(dims(), batch=0) == B.OK      # a valid no-op that touches nothing


def test_append_ws_sizes_and_rejections(L):
    d = dims()
    # fp32 partial sums of the d_c + d_r outputs per token and slice.  The slice count is
    # the fewest dividing hidden / 256 that give the first pass its target of work-groups
    # (else hidden / 256): 512 of 32 outputs x 32 tokens (64 above 32 tokens), or from
    # 256 x 576 outputs on, 128 of 192 outputs x 128 tokens (the LDS-tiled product)
    assert B.append_workspace_size(d, 32, 2048) == 8 * 32 * 192 * 4        # 8 x 1 x 6 groups
    assert B.append_workspace_size(d, 700, 2048) == 8 * 700 * 192 * 4      # 8 x 11 x 6 >= 512
    assert B.append_workspace_size(d, 2048, 2048) == 8 * 2048 * 192 * 4    # tiled: 8 x 16 x 1
    d512 = dims(latent_dim=512, gate_dim=512, num_heads=128)
    assert B.append_workspace_size(d512, 64, 7168) == 28 * 64 * 576 * 4    # 28 x 1 x 18
    assert B.append_workspace_size(d512, 255, 7168) == 14 * 255 * 576 * 4  # 14 x 4 x 18 >= 512
    assert B.append_workspace_size(d512, 512, 7168) == 14 * 512 * 576 * 4  # tiled: 14 x 4 x 3 >= 128
    assert B.append_workspace_size(d512, 4096, 7168) == 2 * 4096 * 576 * 4  # tiled: 2 x 32 x 3
    assert B.append_workspace_size(d512, 16384, 7168) == 16384 * 576 * 4   # tiled: 1 x 128 x 3
    assert B.append_workspace_size(d512, 1, 2048) == 8 * 576 * 4
    # calls the split passes do not take (d_c 128 above 2048 tokens, hidden not a
    # multiple of 256, another layer shape) run the one-pass append and need no workspace
    assert B.append_workspace_size(d, 2049, 2048) == 256
    assert B.append_workspace_size(d, 32, 2000) == 256
    assert B.append_workspace_size(dims(latent_dim=256, gate_dim=256), 32, 2048) == 256
    assert B.append_workspace_size(dims(latent_dim=512, gate_dim=512, rope_dim=32), 32, 2048) == 256
    assert B.append_workspace_size(dims(num_heads=0), 32, 2048) == 0
    assert B.append_workspace_size(d, -1, 2048) == 0
    vp = ctypes.c_void_p(256)
    def call(n, hidden, ws, ws_bytes):
        return L.eg_mla_append_ws(ctypes.byref(d), n, hidden, vp, vp, vp, vp, vp, None, 0.0, vp, vp, 1 << 20, ws,
                                  ws_bytes, None)
    assert call(0, 2048, None, 0) == B.OK                                   # no-op
    assert call(32, 2048, None, 0) == B.ERR_WORKSPACE                       # split path needs one
    assert call(32, 2048, ctypes.c_void_p(4096), 8 * 32 * 192 * 4 - 1) == B.ERR_WORKSPACE   # too small
    assert call(32, 2048, ctypes.c_void_p(4096 + 16), 8 * 32 * 192 * 4) == B.ERR_WORKSPACE  # misaligned
    assert call(32, 40000, ctypes.c_void_p(4096), 1 << 30) == B.ERR_UNSUPPORTED


def test_append_and_prefill_reject_before_launch(L):
    d = dims()
    vp = ctypes.c_void_p(256)
    assert L.eg_mla_append(ctypes.byref(d), 0, 64, None, None, None, None, None, None, 0.0, None, None, 0,
                           None) == B.OK
    assert L.eg_mla_append(ctypes.byref(d), 4, 64, None, vp, vp, vp, vp, None, 0.0, vp, vp, 8, None) == \
        B.ERR_INVALID_ARG
    assert L.eg_mla_append(ctypes.byref(d), 4, 0, vp, vp, vp, vp, vp, None, 0.0, vp, vp, 8, None) == \
        B.ERR_INVALID_ARG
    assert L.eg_mla_append(ctypes.byref(d), 4, 40000, vp, vp, vp, vp, vp, None, 0.0, vp, vp, 8, None) == \
        B.ERR_UNSUPPORTED
    assert L.eg_mla_prefill_ref(ctypes.byref(d), 0, None, None, None, None, None, None, None, 0, None,
                                None) == B.OK
    assert L.eg_mla_prefill_ref(ctypes.byref(d), 10, vp, vp, vp, vp, vp, vp, vp, 16, vp, None) == B.ERR_WORKSPACE
    assert L.eg_mla_prefill_ref(ctypes.byref(d), 40000, vp, vp, vp, vp, vp, vp, vp, 1 << 40, vp, None) == \
        B.ERR_UNSUPPORTED
    assert L.eg_mla_prefill_ref(ctypes.byref(d), -1, vp, vp, vp, vp, vp, vp, vp, 1 << 20, vp, None) == \
        B.ERR_INVALID_ARG


def test_gate_rows_rejects_before_launch(L):
    d = dims()
    vp = ctypes.c_void_p(256)
    # n == 0 is a no-op whatever the pointers
    assert L.eg_mla_gate_rows(ctypes.byref(d), 512, 1000, 0, None, None, None, None, None) == B.OK
    assert L.eg_mla_gate_rows(ctypes.byref(d), 512, 1000, 5, None, vp, vp, vp, None) == B.ERR_INVALID_ARG
    assert L.eg_mla_gate_rows(ctypes.byref(d), 512, 1000, 5, vp, vp, vp, None, None) == B.ERR_INVALID_ARG
    assert L.eg_mla_gate_rows(ctypes.byref(d), 0, 1000, 5, vp, vp, vp, vp, None) == B.ERR_INVALID_ARG
    assert L.eg_mla_gate_rows(ctypes.byref(d), 512, 0, 5, vp, vp, vp, vp, None) == B.ERR_INVALID_ARG
    assert L.eg_mla_gate_rows(ctypes.byref(d), 512, 1000, -1, vp, vp, vp, vp, None) == B.ERR_INVALID_ARG
    assert L.eg_mla_gate_rows(ctypes.byref(d), 20000, 1000, 5, vp, vp, vp, vp, None) == B.ERR_UNSUPPORTED
    bad = dims(gate_dim=64)
    assert L.eg_mla_gate_rows(ctypes.byref(bad), 512, 1000, 5, vp, vp, vp, vp, None) == B.ERR_UNSUPPORTED


def test_gate_table_sizes_and_rejections(L):
    # marks: a stamp line (128 bytes) per id, two list counters, a list of up to V ids
    d = dims()
    assert L.eg_mla_gate_table_marks_size(ctypes.byref(d), 512, 1000) == (33 * 1000 + 2) * 4  # stamp lines, counts, list
    d512 = dims(latent_dim=512, gate_dim=512)
    assert L.eg_mla_gate_table_marks_size(ctypes.byref(d512), 512, 1000) == (33 * 1000 + 2) * 4
    assert L.eg_mla_gate_table_marks_size(ctypes.byref(d), 0, 1000) == 0
    assert L.eg_mla_gate_table_marks_size(ctypes.byref(d), 512, 0) == 0
    vp = ctypes.c_void_p(256)
    mk = ctypes.c_void_p(4096)
    need = (33 * 1000 + 2) * 4
    call = L.eg_mla_gate_table
    assert call(ctypes.byref(d), 512, 1000, 0, None, None, None, None, None, 0, 1, None) == B.OK  # no-op
    assert call(ctypes.byref(d), 512, 1000, 5, vp, vp, vp, vp, mk, need, 0, None) == B.ERR_INVALID_ARG  # stamp 0
    assert call(ctypes.byref(d), 512, 1000, 5, None, vp, vp, vp, mk, need, 1, None) == B.ERR_INVALID_ARG
    assert call(ctypes.byref(d), 512, 1000, 5, vp, vp, vp, None, mk, need, 1, None) == B.ERR_INVALID_ARG
    assert call(ctypes.byref(d), 512, 1000, 5, vp, vp, vp, vp, None, need, 1, None) == B.ERR_WORKSPACE
    assert call(ctypes.byref(d), 512, 1000, 5, vp, vp, vp, vp, mk, need - 4, 1, None) == B.ERR_WORKSPACE
    assert call(ctypes.byref(d), 512, 1000, 5, vp, vp, vp, vp, ctypes.c_void_p(4098), need, 1, None) == \
        B.ERR_WORKSPACE
    assert call(ctypes.byref(d), 20000, 1000, 5, vp, vp, vp, vp, mk, need, 1, None) == B.ERR_UNSUPPORTED


def test_prefill_varlen_rejects_before_launch(L):
    d = dims()
    vp = ctypes.c_void_p(256)
    ws = ctypes.c_void_p(4096)
    n = 100
    need = L.eg_mla_prefill_varlen_workspace_size(ctypes.byref(d), n)
    assert need >= n * 16 * (192 + 128) * 2
    args = lambda **kw: [kw.get(k, v) for k, v in [("cu", vp), ("q", vp), ("lat", vp), ("ids", vp), ("gate", vp),
                                                     ("wk", vp), ("wv", vp), ("ws", ws), ("wsb", need),
                                                     ("out", vp)]]
    call = lambda dd, batch, T, **kw: L.eg_mla_prefill_varlen(ctypes.byref(dd), batch, T, *args(**kw), None)
    # zero tokens is a no-op whatever the pointers
    assert L.eg_mla_prefill_varlen(ctypes.byref(d), 1, 0, *[None] * 7, None, 0, None, None) == B.OK
    assert call(d, 0, n) == B.ERR_INVALID_ARG
    assert call(d, 2, -1) == B.ERR_INVALID_ARG
    assert call(d, 2, n, cu=None) == B.ERR_INVALID_ARG
    assert call(d, 2, n, out=None) == B.ERR_INVALID_ARG
    assert call(d, 2, n, q=ctypes.c_void_p(258)) == B.ERR_INVALID_ARG  # misaligned
    assert call(d, 2, n, wsb=need - 1) == B.ERR_WORKSPACE
    assert call(d, 2, n, ws=ctypes.c_void_p(4100)) == B.ERR_WORKSPACE
    # the MFMA prefill covers bf16 layers with d_h = d_v = 128 and d_r = 64: the absorbed
    # form for d_c 128 with 16 heads, the explicit form for any other head count and
    # d_c a multiple of 64 (workspace: sequence starts, then K^C and V in fp16 per head)
    for bad in (dims(latent_dim=96, gate_dim=96), dims(rope_dim=32), dims(dtype=B.FP32), dims(v_head_dim=64),
                dims(head_dim=64)):
        assert call(bad, 2, n) == B.ERR_UNSUPPORTED
        assert L.eg_mla_prefill_varlen_workspace_size(ctypes.byref(bad), n) == 0
    al = lambda x: (x + 255) // 256 * 256
    for good, H in ((dims(num_heads=32), 32), (dims(latent_dim=512, gate_dim=512, num_heads=128), 128),
                    (dims(latent_dim=256, gate_dim=256, num_heads=16), 16)):
        need_x = L.eg_mla_prefill_varlen_workspace_size(ctypes.byref(good), n)
        # sequence starts, K^C and V (fp16), the gated latent as bf16 hi and lo rows
        assert need_x == al(n * 4) + 2 * al(n * H * 128 * 2) + 2 * al(n * good.latent_dim * 2)
        assert call(good, 2, n, wsb=need_x - 1) == B.ERR_WORKSPACE


def test_decode_literal_rejects_before_launch(L):
    d = dims()
    vp = ctypes.c_void_p(256)
    ws = ctypes.c_void_p(4096)
    slots = 64 * 64
    need = L.eg_mla_decode_literal_workspace_size(ctypes.byref(d), 2, 4)
    assert need >= 2 * (4 * 64 // 128) * 16 * (128 + 4) * 4   # fp32 partials per (sequence, 128-token tile, head)
    assert L.eg_mla_decode_literal_workspace_size(ctypes.byref(d), 2, 5) > need  # a ragged last tile counts

    def call(dd=d, batch=2, flags=0, lnw=vp, lnb=vp, pt=None, maxp=4, nslots=slots, wsp=ws, wsb=need, q=vp):
        return L.eg_mla_decode_literal(ctypes.byref(dd), batch, q, vp, vp, vp, vp, vp, lnw, lnb, flags, vp, pt, maxp,
                                       nslots, wsp, wsb, vp, None)
    assert call(batch=0) == B.OK
    assert call(flags=4) == B.ERR_INVALID_ARG
    assert call(lnw=None) == B.ERR_INVALID_ARG            # the LayerNorm needs its weight ...
    assert call(lnb=None) == B.ERR_INVALID_ARG            # ... and bias
    assert call(q=ctypes.c_void_p(258)) == B.ERR_INVALID_ARG
    assert call(nslots=2 * 4 * 64 - 1) == B.ERR_INVALID_ARG  # contiguous rows must hold every sequence
    assert call(wsb=need - 1) == B.ERR_WORKSPACE
    assert call(wsp=ctypes.c_void_p(4100)) == B.ERR_WORKSPACE
    big = L.eg_mla_decode_literal_workspace_size(ctypes.byref(d), 2, 1024)
    assert big >= 2 * (1024 * 64 // 128) * 16 * (128 + 4) * 4  # 65536-token capacity: no limit on the context
    assert call(maxp=1024, nslots=2 * 1024 * 64, wsb=big - 1) == B.ERR_WORKSPACE
    # the tile kernel takes bf16, d_c = d_h = d_v = 128, d_r = 64, at most 160 heads and a gate
    # table below 4 GB; other layers take the generic kernel while its tile state fits the LDS
    # (value sums of all heads, [H][d_v] fp32, and 8 latents)
    assert call(dd=dims(vocab_size=600000)) == B.ERR_UNSUPPORTED   # a gate table of 4 GB or more
    for dd in (dims(latent_dim=512, gate_dim=512, num_heads=128), dims(rope_dim=32), dims(dtype=B.FP32),
               dims(v_head_dim=64), dims(num_heads=161)):
        n = L.eg_mla_decode_literal_workspace_size(ctypes.byref(dd), 2, 4)
        assert call(dd=dd, wsb=n - 1) == B.ERR_WORKSPACE            # accepted shapes, checked up to the workspace
    for bad in (dims(num_heads=320),                              # 320 x 128 value sums: 160 KB of LDS
                dims(latent_dim=4096, gate_dim=4096, num_heads=250)):
        assert call(dd=bad) == B.ERR_UNSUPPORTED
