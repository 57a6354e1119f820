"""Thin ctypes binding of libegmla.so.

Argument marshalling only: every step of append / decode / prefill runs in
the library's HIP kernels.  Tensors are torch tensors on the GPU (torch is
used for device memory and streams); bf16 storage is ``torch.bfloat16``.
The functions carry the C entry points' names without the ``eg_mla_``
prefix.  If the library is missing this module raises; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libegmla.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = range(5)
FP32, BF16 = 0, 1
PATH_AUTO, PATH_VALU, PATH_MFMA = 0, 1, 2

# Every symbol include/eg_mla.h declares.
EXPORTS = ["eg_mla_status_string", "eg_mla_check_dims", "eg_mla_append", "eg_mla_decode_workspace_size",
           "eg_mla_decode", "eg_mla_decode_planned", "eg_mla_gate_rows", "eg_mla_prefill_workspace_size",
           "eg_mla_prefill_ref", "eg_mla_prefill_varlen_workspace_size", "eg_mla_prefill_varlen",
           "eg_mla_decode_literal_workspace_size", "eg_mla_decode_literal", "eg_mla_decode_noalloc",
           "eg_mla_append_workspace_size", "eg_mla_append_ws", "eg_mla_gate_table_marks_size",
           "eg_mla_gate_table"]
NOALLOC_SCRATCH_BYTES = 32 << 20  # EG_MLA_NOALLOC_SCRATCH_BYTES
LITERAL_NO_LN, LITERAL_ADD = 1, 2


class Dims(ctypes.Structure):
    _fields_ = [("num_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("v_head_dim", ctypes.c_int32),
                ("latent_dim", ctypes.c_int32), ("rope_dim", ctypes.c_int32), ("gate_dim", ctypes.c_int32),
                ("vocab_size", ctypes.c_int32), ("page_size", ctypes.c_int32), ("softmax_scale", ctypes.c_float),
                ("dtype", ctypes.c_int32)]


class Plan(ctypes.Structure):
    _fields_ = [("path", ctypes.c_int32), ("split_tokens", ctypes.c_int32),
                ("split_start_event", ctypes.c_void_p), ("split_stop_event", ctypes.c_void_p),
                ("id_slices", ctypes.c_int32)]


class EgMlaError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)}")


_lib = None


def lib() -> ctypes.CDLL:
    """Loads libegmla.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2509_16686_amd.build`")
    # torch first: its HIP runtime carries the same SONAME, so the library binds to that one instance
    import torch  # noqa: F401
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    pd, pp = ctypes.POINTER(Dims), ctypes.POINTER(Plan)
    L.eg_mla_status_string.restype = ctypes.c_char_p
    L.eg_mla_status_string.argtypes = [ctypes.c_int]
    L.eg_mla_check_dims.restype = ctypes.c_int
    L.eg_mla_check_dims.argtypes = [pd]
    L.eg_mla_append.restype = ctypes.c_int
    L.eg_mla_append.argtypes = [pd, i32, i32, vp, vp, vp, vp, vp, vp, ctypes.c_float, vp, vp, i64, vp]
    L.eg_mla_append_workspace_size.restype = sz
    L.eg_mla_append_workspace_size.argtypes = [pd, i32, i32]
    L.eg_mla_append_ws.restype = ctypes.c_int
    L.eg_mla_append_ws.argtypes = [pd, i32, i32, vp, vp, vp, vp, vp, vp, ctypes.c_float, vp, vp, i64, vp, sz, vp]
    L.eg_mla_decode_workspace_size.restype = sz
    L.eg_mla_decode_workspace_size.argtypes = [pd, i32, i32, pp]
    L.eg_mla_decode.restype = ctypes.c_int
    L.eg_mla_decode.argtypes = [pd, i32, vp, vp, vp, vp, vp, vp, vp, vp, i32, i64, vp, sz, vp, vp]
    L.eg_mla_decode_planned.restype = ctypes.c_int
    L.eg_mla_decode_planned.argtypes = [pd, i32, vp, vp, vp, vp, vp, vp, vp, vp, i32, i64, vp, sz, vp, vp, pp]
    L.eg_mla_decode_noalloc.restype = ctypes.c_int
    L.eg_mla_decode_noalloc.argtypes = [pd, i32, vp, vp, vp, vp, vp, vp, vp, vp, i32, i64, vp, vp]
    L.eg_mla_gate_rows.restype = ctypes.c_int
    L.eg_mla_gate_rows.argtypes = [pd, i32, i32, i64, vp, vp, vp, vp, vp]
    L.eg_mla_gate_table_marks_size.restype = sz
    L.eg_mla_gate_table_marks_size.argtypes = [pd, i32, i32]
    L.eg_mla_gate_table.restype = ctypes.c_int
    L.eg_mla_gate_table.argtypes = [pd, i32, i32, i64, vp, vp, vp, vp, vp, sz, ctypes.c_uint32, vp]
    L.eg_mla_prefill_workspace_size.restype = sz
    L.eg_mla_prefill_workspace_size.argtypes = [pd, i32]
    L.eg_mla_prefill_ref.restype = ctypes.c_int
    L.eg_mla_prefill_ref.argtypes = [pd, i32, vp, vp, vp, vp, vp, vp, vp, sz, vp, vp]
    L.eg_mla_prefill_varlen_workspace_size.restype = sz
    L.eg_mla_prefill_varlen_workspace_size.argtypes = [pd, i32]
    L.eg_mla_prefill_varlen.restype = ctypes.c_int
    L.eg_mla_prefill_varlen.argtypes = [pd, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp, vp]
    L.eg_mla_decode_literal_workspace_size.restype = sz
    L.eg_mla_decode_literal_workspace_size.argtypes = [pd, i32, i32]
    L.eg_mla_decode_literal.restype = ctypes.c_int
    L.eg_mla_decode_literal.argtypes = [pd, i32, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_uint32, vp, vp, i32, i64,
                                        vp, sz, vp, vp]
    _lib = L
    return L


def status_string(status: int) -> str:
    return lib().eg_mla_status_string(status).decode()


def make_dims(*, num_heads, head_dim, v_head_dim, latent_dim, rope_dim, vocab_size, page_size=64,
              gate_dim=None, softmax_scale=0.0, dtype=BF16) -> Dims:
    return Dims(num_heads, head_dim, v_head_dim, latent_dim, rope_dim,
                latent_dim if gate_dim is None else gate_dim, vocab_size, page_size, softmax_scale, dtype)


def make_plan(path: int = PATH_AUTO, split_tokens: int = 0, start_event=None, stop_event=None,
              id_slices: int = 0) -> Plan:
    return Plan(path, split_tokens, start_event, stop_event, id_slices)


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


def _check(st: int, where: str):
    if st != OK:
        raise EgMlaError(st, where)


def check_dims(dims: Dims) -> int:
    return lib().eg_mla_check_dims(ctypes.byref(dims))


def decode_workspace_size(dims: Dims, batch: int, max_pages_per_seq: int, plan: Optional[Plan] = None) -> int:
    return lib().eg_mla_decode_workspace_size(ctypes.byref(dims), batch, max_pages_per_seq,
                                               None if plan is None else ctypes.byref(plan))


def prefill_workspace_size(dims: Dims, seq_len: int) -> int:
    return lib().eg_mla_prefill_workspace_size(ctypes.byref(dims), seq_len)


def decode(dims: Dims, q, latent_cache, token_id_cache, gate_table, w_uk, w_uv, seq_lens, page_table,
           max_pages_per_seq: int, workspace, out, plan: Optional[Plan] = None, stream=None) -> None:
    """eg_mla_decode / eg_mla_decode_planned over device tensors."""
    L = lib()
    batch = int(q.shape[0])
    num_slots = int(latent_cache.shape[0])
    ws_bytes = workspace.numel() * workspace.element_size()
    args = (ctypes.byref(dims), batch, _ptr(q), _ptr(latent_cache), _ptr(token_id_cache), _ptr(gate_table),
            _ptr(w_uk), _ptr(w_uv), _ptr(seq_lens), _ptr(page_table), max_pages_per_seq, num_slots,
            _ptr(workspace), ws_bytes, _ptr(out), _stream(stream))
    if plan is None:
        _check(L.eg_mla_decode(*args), "eg_mla_decode")
    else:
        _check(L.eg_mla_decode_planned(*args, ctypes.byref(plan)), "eg_mla_decode_planned")


def decode_noalloc(dims: Dims, q, latent_cache, token_id_cache, gate_table, w_uk, w_uv, seq_lens, page_table,
                   max_pages_per_seq: int, out, stream=None) -> None:
    """eg_mla_decode_noalloc over device tensors (no workspace: the library's scratch array)."""
    _check(lib().eg_mla_decode_noalloc(ctypes.byref(dims), int(q.shape[0]), _ptr(q), _ptr(latent_cache),
                                       _ptr(token_id_cache), _ptr(gate_table), _ptr(w_uk), _ptr(w_uv), _ptr(seq_lens),
                                       _ptr(page_table), max_pages_per_seq, int(latent_cache.shape[0]), _ptr(out),
                                       _stream(stream)), "eg_mla_decode_noalloc")


def append(dims: Dims, x, token_ids, positions, slots, w_dkv, kv_norm_w, latent_cache, token_id_cache,
           rope_theta: float = 10000.0, stream=None) -> None:
    """eg_mla_append over device tensors."""
    n, hidden = int(x.shape[0]), int(x.shape[1])
    _check(lib().eg_mla_append(ctypes.byref(dims), n, hidden, _ptr(x), _ptr(token_ids), _ptr(positions),
                               _ptr(slots), _ptr(w_dkv), _ptr(kv_norm_w), rope_theta, _ptr(latent_cache),
                               _ptr(token_id_cache), int(latent_cache.shape[0]), _stream(stream)), "eg_mla_append")


def append_workspace_size(dims: Dims, n_tokens: int, hidden: int) -> int:
    return lib().eg_mla_append_workspace_size(ctypes.byref(dims), n_tokens, hidden)


def append_ws(dims: Dims, x, token_ids, positions, slots, w_dkv, kv_norm_w, latent_cache, token_id_cache, workspace,
              rope_theta: float = 10000.0, stream=None) -> None:
    """eg_mla_append_ws over device tensors (workspace: a uint8 device tensor)."""
    n, hidden = int(x.shape[0]), int(x.shape[1])
    _check(lib().eg_mla_append_ws(ctypes.byref(dims), n, hidden, _ptr(x), _ptr(token_ids), _ptr(positions),
                                  _ptr(slots), _ptr(w_dkv), _ptr(kv_norm_w), rope_theta, _ptr(latent_cache),
                                  _ptr(token_id_cache), int(latent_cache.shape[0]), _ptr(workspace),
                                  int(workspace.numel()) if workspace is not None else 0, _stream(stream)),
           "eg_mla_append_ws")


def gate_rows(dims: Dims, ids, emb, w_ue, out, stream=None) -> None:
    """eg_mla_gate_rows over device tensors: out[i] = W_UE Emb[ids[i]]."""
    n = int(ids.shape[0])
    emb_vocab, emb_dim = int(emb.shape[0]), int(emb.shape[1])
    _check(lib().eg_mla_gate_rows(ctypes.byref(dims), emb_dim, emb_vocab, n, _ptr(ids), _ptr(emb), _ptr(w_ue),
                                  _ptr(out), _stream(stream)), "eg_mla_gate_rows")


def gate_table_marks_size(dims: Dims, emb_dim: int, emb_vocab: int) -> int:
    return int(lib().eg_mla_gate_table_marks_size(ctypes.byref(dims), emb_dim, emb_vocab))


def gate_table(dims: Dims, ids, emb, w_ue, table, marks, stamp: int, stream=None) -> None:
    """eg_mla_gate_table over device tensors: table[id] = W_UE Emb[id] for the distinct ids."""
    n = int(ids.shape[0])
    emb_vocab, emb_dim = int(emb.shape[0]), int(emb.shape[1])
    _check(lib().eg_mla_gate_table(ctypes.byref(dims), emb_dim, emb_vocab, n, _ptr(ids), _ptr(emb), _ptr(w_ue),
                                   _ptr(table), _ptr(marks), int(marks.numel() * marks.element_size()), stamp,
                                   _stream(stream)), "eg_mla_gate_table")


def decode_literal_workspace_size(dims: Dims, batch: int, max_pages: int) -> int:
    return lib().eg_mla_decode_literal_workspace_size(ctypes.byref(dims), batch, max_pages)


def decode_literal(dd, gate_full, ln_w, ln_b, flags: int, workspace, stream=None) -> None:
    """eg_mla_decode_literal over a staged DeviceDecode (its gate table is not used)."""
    _check(lib().eg_mla_decode_literal(ctypes.byref(dd.dims), int(dd.q.shape[0]), _ptr(dd.q), _ptr(dd.cache),
                                       _ptr(dd.ids), _ptr(gate_full), _ptr(dd.w_uk), _ptr(dd.w_uv), _ptr(ln_w),
                                       _ptr(ln_b), flags, _ptr(dd.seq_lens), _ptr(dd.page_table), dd.max_pages,
                                       int(dd.cache.shape[0]), _ptr(workspace),
                                       workspace.numel() * workspace.element_size(), _ptr(dd.out), _stream(stream)),
           "eg_mla_decode_literal")


def prefill_varlen_workspace_size(dims: Dims, total_tokens: int) -> int:
    return lib().eg_mla_prefill_varlen_workspace_size(ctypes.byref(dims), total_tokens)


def prefill_varlen(dims: Dims, cu_seqlens, q, latent, token_ids, gate_table, w_uk, w_uv, workspace, out,
                   stream=None) -> None:
    """eg_mla_prefill_varlen over device tensors (sequences packed back to back)."""
    batch = int(cu_seqlens.shape[0]) - 1
    T = int(q.shape[0])
    _check(lib().eg_mla_prefill_varlen(ctypes.byref(dims), batch, T, _ptr(cu_seqlens), _ptr(q), _ptr(latent),
                                       _ptr(token_ids), _ptr(gate_table), _ptr(w_uk), _ptr(w_uv), _ptr(workspace),
                                       workspace.numel() * workspace.element_size(), _ptr(out), _stream(stream)),
           "eg_mla_prefill_varlen")


def prefill_ref(dims: Dims, q, latent, token_ids, gate_table, w_uk, w_uv, workspace, out, stream=None) -> None:
    """eg_mla_prefill_ref over device tensors."""
    T = int(q.shape[0])
    _check(lib().eg_mla_prefill_ref(ctypes.byref(dims), T, _ptr(q), _ptr(latent), _ptr(token_ids),
                                    _ptr(gate_table), _ptr(w_uk), _ptr(w_uv), _ptr(workspace),
                                    workspace.numel() * workspace.element_size(), _ptr(out), _stream(stream)),
           "eg_mla_prefill_ref")


# ---------------------------------------------------------------------------
# device-side staging of generated workloads (plain copies, no arithmetic)
# ---------------------------------------------------------------------------
@dataclass
class DeviceDecode:
    dims: Dims
    q: object
    cache: object
    ids: object
    gate: object
    w_uk: object
    w_uv: object
    seq_lens: object
    page_table: object
    max_pages: int
    out: object


def dims_for(wl) -> Dims:
    return make_dims(num_heads=wl.heads, head_dim=wl.head_dim, v_head_dim=wl.v_head_dim, latent_dim=wl.latent_dim,
                     rope_dim=wl.rope_dim, vocab_size=wl.vocab, page_size=wl.page_size,
                     gate_dim=wl.gate_dim, dtype=BF16 if wl.dtype == "bf16" else FP32)


def to_device_tensor(a, storage: str, device="cuda"):
    """Host array (bf16 as uint16 bits) -> device tensor of the storage type."""
    import numpy as np
    import torch
    if storage == "bf16" and a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def stage_decode(inp, device="cuda") -> DeviceDecode:
    """Copies a generated DecodeInputs to the device and allocates `out`."""
    import torch
    wl = inp.wl
    st = wl.dtype
    dt = torch.bfloat16 if st == "bf16" else torch.float32
    return DeviceDecode(
        dims=dims_for(wl), q=to_device_tensor(inp.q, st, device), cache=to_device_tensor(inp.latent_cache, st, device),
        ids=to_device_tensor(inp.token_ids, "int", device), gate=to_device_tensor(inp.gate_table, st, device),
        w_uk=to_device_tensor(inp.w_uk, st, device), w_uv=to_device_tensor(inp.w_uv, st, device),
        seq_lens=to_device_tensor(inp.seq_lens, "int", device),
        page_table=None if inp.page_table is None else to_device_tensor(inp.page_table, "int", device),
        max_pages=inp.max_pages, out=torch.empty((wl.batch, wl.heads, wl.v_head_dim), dtype=dt, device=device))


def alloc_workspace(nbytes: int, device="cuda"):
    import torch
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


def run_decode(dd: DeviceDecode, plan: Optional[Plan] = None, workspace=None, stream=None):
    """Sizes a workspace (unless given) and runs one decode; returns dd.out."""
    if workspace is None:
        workspace = alloc_workspace(decode_workspace_size(dd.dims, int(dd.q.shape[0]), dd.max_pages, plan))
    decode(dd.dims, dd.q, dd.cache, dd.ids, dd.gate, dd.w_uk, dd.w_uv, dd.seq_lens, dd.page_table, dd.max_pages,
           workspace, dd.out, plan=plan, stream=stream)
    return dd.out


def out_to_f64(t):
    """Device output -> float64 numpy (exact widening)."""
    import torch
    return t.detach().to(torch.float64).cpu().numpy()
