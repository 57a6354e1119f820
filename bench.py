#!/usr/bin/env python3
"""EG-MLA decode throughput on one MI355X.

One step = one eg_mla_decode call over one batch of synthetic, seeded input:
absorption, the token-streaming split kernel (gate gather, gating, scores,
online softmax, latent value sum) and the split merge with W_UV.  Default
workload: ~1B-model layer, batch 32, 16 heads, d_c 128, d_r 64, context 4096,
bf16 storage.

Timing: inputs are resident in HBM; R distinct copies of every input (>= 1 GB
in total) are rotated so the 256 MB last-level cache cannot serve a call from
the previous one.  The host enqueues the K timed calls behind a GPU spin
kernel, so launch overhead is hidden and the events measure back-to-back GPU
execution.  HIP events around every split-kernel launch (on the call's
stream) give that kernel's average duration for the roofline figure.

Prints ONE JSON line on stdout; progress goes to stderr.
"""
import argparse
import ctypes
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode tokens/s + achieved HBM GB/s (% of peak) for eg_mla_decode, 1 GPU"
HBM_PEAK_GBPS = 8000.0
REPO = os.path.dirname(os.path.abspath(__file__))
# Calibrated FETCH_SIZE + WRITE_SIZE counters of the split kernel on the default workload,
# valid only while the kernel's sources hash to the recorded value.
TRAFFIC_PROFILE = os.path.join(REPO, "profiles", "split_slice_b32_h16_dc128_dr64_l4096_traffic.md")
# Streaming-read reference (csrc/stream_probe.hip): context for the roofline, not a target.
STREAM_PROFILE = os.path.join(REPO, "profiles", "stream_read_ceiling.md")
# Layers of the paper's largest model (App. A), for an indicative whole-model rate.
MODEL_LAYERS = 24




def split_kernel_name(wl, path):
    """The split kernel the library launches for this workload and path (see host_plan.cpp)."""
    if wl.dtype != "bf16" or path == "valu":
        return "split_valu_kernel"
    if wl.latent_dim == 128 and wl.rope_dim == 64:
        return "split_slice_kernel"
    if wl.latent_dim == 512 and wl.rope_dim == 64 and wl.heads % 128 == 0:
        return "split_wide_kernel"
    if wl.heads % 16 == 0 and wl.rope_dim == 64 and wl.latent_dim in (320, 512):
        return "split_mfma_kernel"
    return "split_valu_kernel"

def recorded_traffic():
    """Bytes per split-kernel launch from the committed counter summary, or None when the
    summary is missing or the kernel sources changed since the counters were taken."""
    import hashlib
    try:
        fields = {}
        for line in open(TRAFFIC_PROFILE):
            if ":" in line and line.split(":", 1)[0] in ("traffic_bytes_per_launch", "kernel_sources",
                                                        "kernel_sources_sha256"):
                k, v = line.split(":", 1)
                fields[k] = v.strip()
        h = hashlib.sha256()
        for rel in fields["kernel_sources"].split():
            with open(os.path.join(REPO, rel), "rb") as f:
                h.update(f.read())
        if h.hexdigest() != fields["kernel_sources_sha256"]:
            return None
        return int(fields["traffic_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None

def log(*a):
    print(*a, file=sys.stderr, flush=True)


class Hip:
    """hipEvent calls through the HIP runtime torch already loaded."""

    def __init__(self):
        self.L = ctypes.CDLL("libamdhip64.so.7")
        self.L.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.L.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.L.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.L.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.L.hipEventSynchronize.argtypes = [ctypes.c_void_p]

    def event(self):
        e = ctypes.c_void_p()
        assert self.L.hipEventCreate(ctypes.byref(e)) == 0
        return e

    def record(self, e, stream):
        assert self.L.hipEventRecord(e, ctypes.c_void_p(stream)) == 0

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        assert self.L.hipEventElapsedTime(ctypes.byref(ms), a, b) == 0
        return ms.value

    def destroy(self, e):
        self.L.hipEventDestroy(e)


def cpu_model():
    """The host CPU's model name, as the kernel reports it."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def recorded_stream_ceiling(mib=60):
    """GB/s of the streaming-read reference program for a launch of `mib` MiB (best work-group
    count), from its committed summary; None when missing."""
    try:
        for line in open(STREAM_PROFILE):
            cells = [c.strip() for c in line.strip().strip("|").split("|")]
            if len(cells) >= 4 and cells[0] == str(mib):
                return float(cells[3])
    except (OSError, ValueError):
        pass
    return None


def cpu_baseline(inp, seconds):
    """The fp64 oracle as it stands, timed on the host over whole batches: with every
    BLAS thread the process has (the reported value), then limited to one thread."""
    from oracle import eg_mla_oracle as orc
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threads = max([i["num_threads"] for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:
        threadpool_limits = None
        threads = 1
    wl = inp.wl

    def rate(budget):
        reps = 0
        t0 = time.perf_counter()
        while True:
            orc.decode(inp.q, inp.latent_cache, inp.token_ids, inp.gate_table, inp.w_uk, inp.w_uv, inp.seq_lens,
                       latent_dim=wl.latent_dim, head_dim=wl.head_dim, rope_dim=wl.rope_dim, storage=wl.dtype,
                       page_table=inp.page_table, page_size=wl.page_size, max_pages=inp.max_pages)
            reps += 1
            el = time.perf_counter() - t0
            if el >= budget or reps >= 100:
                return reps, el

    reps, el = rate(seconds)
    out = {"value": wl.batch * reps / el, "unit": "tokens/s", "cores": threads, "kind": "oracle",
           "sample": f"{reps} full decode steps of the same workload ({wl.batch} sequences each), "
                     f"{el:.1f} s, numpy fp64 with {threads} BLAS threads",
           "cpu_model": cpu_model(), "host_cpus": len(os.sched_getaffinity(0))}
    if threadpool_limits is not None:
        with threadpool_limits(limits=1, user_api="blas"):
            reps1, el1 = rate(seconds / 2)
        out["single_thread"] = {"value": wl.batch * reps1 / el1, "unit": "tokens/s", "cores": 1,
                                "sample": f"{reps1} full decode steps, {el1:.1f} s, one BLAS thread"}
    return out


PREFILL_METRIC = "prefill tokens/s + achieved bf16 TFLOP/s (% of MFMA peak) for eg_mla_prefill_varlen, 1 GPU"
MFMA_BF16_PEAK_TFLOPS = 2500.0


def prefill_flops(lens, heads=16, dc=128, dr=64, dh=128, dv=128):
    """Algorithmic flops of one causal prefill call.  Absorbed form (d_c 128, 16 heads): scores and
    values over every (row, key <= row) pair of each sequence in the latent space, plus the absorption
    and the up-projection of every row.  Explicit form (other layers): the projection of every token's
    gated latent to each head's key and value, then scores and values per pair in the head space."""
    pairs = sum(t * (t + 1) // 2 for t in lens)
    rows = sum(lens) * heads
    if dc == 128 and heads == 16:
        return pairs * heads * 2 * (dc + dr + dc) + rows * 2 * dh * dc + rows * 2 * dc * dv
    return pairs * heads * 2 * (dh + dr + dv) + rows * 2 * dc * (dh + dv)


def prefill_cpu_baseline(wl, seconds):
    """The fp64 oracle's prefill of one 512-token sequence, repeated for about `seconds`."""
    from oracle import eg_mla_oracle as orc
    from paper_2509_16686_amd import workloads as W
    try:
        from threadpoolctl import threadpool_info
        threads = max([i["num_threads"] for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:
        threads = 1
    pin = W.generate_prefill(wl, 512, seed=wl.seed + 3001)
    reps = 0
    t0 = time.perf_counter()
    while True:
        orc.prefill(pin.q, pin.latent, pin.token_ids, pin.gate_table, pin.w_uk, pin.w_uv, latent_dim=wl.latent_dim,
                    head_dim=wl.head_dim, rope_dim=wl.rope_dim, storage=wl.dtype)
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds or reps >= 100:
            break
    return {"value": 512 * reps / el, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{reps} causal prefills of one 512-token sequence of the same layer, {el:.1f} s, "
                      f"numpy fp64 with {threads} BLAS threads",
            "cpu_model": cpu_model(), "host_cpus": len(os.sched_getaffinity(0))}


def prefill_main(args):
    """Times eg_mla_prefill_varlen on `--prefill BxT` (B sequences of T tokens, packed)."""
    import numpy as np
    import torch

    from paper_2509_16686_amd import binding as B
    from paper_2509_16686_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    L = B.lib()
    hip = Hip()
    nb, T = (int(x) for x in args.prefill.lower().split("x"))
    lens = [T] * nb
    wl = W.WORKLOADS[args.workload] if args.workload in (1, 4) else W.WORKLOADS[1]
    log(f"bench: generating a prefill of {nb} x {T} tokens ({wl.name} layer)")
    pb = W.generate_prefill_batch(wl, lens, seed=wl.seed + 3000)
    total = int(pb.cu_seqlens[-1])
    dims = B.dims_for(wl)
    copy_bytes = pb.q.nbytes + pb.latent.nbytes + pb.token_ids.nbytes + total * wl.heads * wl.v_head_dim * 2
    R = max(1, math.ceil(args.rotate_bytes / copy_bytes))
    st = wl.dtype
    shared = [B.to_device_tensor(pb.cu_seqlens, "int"), B.to_device_tensor(pb.gate_table, st),
              B.to_device_tensor(pb.w_uk, st), B.to_device_tensor(pb.w_uv, st)]
    copies = []
    for _ in range(R):
        copies.append([B.to_device_tensor(pb.q, st), B.to_device_tensor(pb.latent, st),
                       B.to_device_tensor(pb.token_ids, "int"),
                       torch.empty((total, wl.heads, wl.v_head_dim), dtype=torch.bfloat16, device="cuda")])
    ws_bytes = B.prefill_varlen_workspace_size(dims, total)
    ws = B.alloc_workspace(ws_bytes)
    stream = torch.cuda.current_stream().cuda_stream
    call = L.eg_mla_prefill_varlen

    def argset(c):
        cu, gate, wk, wv = shared
        q, lat, ids, out = c
        return (ctypes.byref(dims), nb, total, cu.data_ptr(), q.data_ptr(), lat.data_ptr(), ids.data_ptr(),
                gate.data_ptr(), wk.data_ptr(), wv.data_ptr(), ws.data_ptr(), ws_bytes, out.data_ptr(), stream)

    K, Wm = args.steps, args.warmup
    arglist = [argset(copies[k % R]) for k in range(K)]
    for k in range(max(Wm, 1)):
        assert call(*argset(copies[k % R])) == 0
    torch.cuda.synchronize()
    e0, e1 = hip.event(), hip.event()
    torch.cuda._sleep(20_000_000)  # the host enqueues the K calls behind a spin
    hip.record(e0, stream)
    for a in arglist:
        call(*a)
    hip.record(e1, stream)
    torch.cuda.synchronize()
    ms = hip.elapsed_ms(e0, e1) / K
    fl = prefill_flops(lens, heads=wl.heads, dc=wl.latent_dim, dr=wl.rope_dim, dh=wl.head_dim, dv=wl.v_head_dim)
    tflops = fl / (ms * 1e-3) / 1e12
    log(f"bench: prefill {nb} x {T}: {ms * 1e3:.1f} us/call, {total / ms * 1e3 / 1e6:.2f} M tokens/s, "
        f"{tflops:.0f} TFLOP/s ({100 * tflops / MFMA_BF16_PEAK_TFLOPS:.1f} % of the bf16 MFMA peak)")
    out = {
        "metric": PREFILL_METRIC, "value": total / (ms * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": K,
        "warmup": Wm, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"prefill_{nb}x{T}_{wl.name}", "sequences": nb, "tokens_per_sequence": T,
                   "heads": wl.heads, "latent_dim": wl.latent_dim, "rope_dim": wl.rope_dim, "storage": wl.dtype,
                   "rotating_copies": R},
        "roofline": {"bound": "mfma", "kernel": ("eg_mla_prefill_varlen (whole call: absorption, attention, "
                                                 "up-projection)") if wl.heads == 16 and wl.latent_dim == 128 else
                                                ("eg_mla_prefill_varlen (whole call: projection to per-head keys "
                                                 "and values, attention)"),
                     "achieved": tflops, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": tflops / MFMA_BF16_PEAK_TFLOPS, "traffic": None, "algorithmic_flops_per_call": fl,
                     "call_us": ms * 1e3},
    }
    if not args.no_cpu_baseline:
        log(f"bench: timing the fp64 oracle's prefill on the host for ~{args.cpu_seconds:.0f} s")
        out["cpu_baseline"] = prefill_cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def append_main(args):
    """Times eg_mla_append_ws (and the one-pass eg_mla_append) of `--append N` tokens (one call per step)."""
    import torch

    from paper_2509_16686_amd import binding as B
    from paper_2509_16686_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    L = B.lib()
    hip = Hip()
    wl = W.WORKLOADS[args.workload] if args.workload < len(W.WORKLOADS) else W.MLA_DC320_BIGBATCH
    n = args.append
    rows = max(2 * n, 4096)
    log(f"bench: generating an append of {n} tokens ({wl.name} layer, hidden {wl.hidden})")
    ai = W.generate_append(wl, n, rows, with_norm=True)
    dims = B.dims_for(wl)
    st = wl.dtype
    t = lambda a, kind: B.to_device_tensor(a, kind)
    x, ids, pos, slots = t(ai.x, st), t(ai.token_ids, "int"), t(ai.positions, "int"), t(ai.slots, "int")
    w, nw = t(ai.w_dkv, st), t(ai.kv_norm_w, st)
    cache = torch.zeros((rows, wl.row_dim), dtype=torch.bfloat16 if st == "bf16" else torch.float32, device="cuda")
    idc = torch.zeros((rows,), dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    a = (ctypes.byref(dims), n, wl.hidden, x.data_ptr(), ids.data_ptr(), pos.data_ptr(), slots.data_ptr(), w.data_ptr(),
         nw.data_ptr(), ai.rope_theta, cache.data_ptr(), idc.data_ptr(), rows)
    ws = B.alloc_workspace(B.append_workspace_size(dims, n, wl.hidden))
    K, Wm = args.steps, args.warmup

    def time_calls(call, extra):
        for _ in range(max(Wm, 1)):
            assert call(*a, *extra) == 0
        torch.cuda.synchronize()
        e0, e1 = hip.event(), hip.event()
        torch.cuda._sleep(20_000_000)  # the K calls queue behind a spin: GPU time, not host enqueue time
        hip.record(e0, stream)
        for _ in range(K):
            call(*a, *extra)
        hip.record(e1, stream)
        torch.cuda.synchronize()
        return hip.elapsed_ms(e0, e1) / K

    ms_one = time_calls(L.eg_mla_append, (stream,))
    ms = time_calls(L.eg_mla_append_ws, (ws.data_ptr(), ws.numel(), stream))
    flops = 2.0 * n * wl.hidden * wl.row_dim
    log(f"bench: append of {n} tokens: {ms * 1e3:.1f} us/call with the workspace ({ms_one * 1e3:.1f} us one-pass), "
        f"{n / ms * 1e3 / 1e6:.2f} M tokens/s, {flops / (ms * 1e-3) / 1e12:.1f} TFLOP/s")
    out = {"metric": "append tokens/s for eg_mla_append_ws, 1 GPU", "value": n / (ms * 1e-3), "unit": "tokens/s",
           "one_pass_us_per_call": ms_one * 1e3,
           "n_gpus": 1, "steps": K, "warmup": Wm, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16" if st == "bf16" else "fp32", "data": "synthetic",
           "config": {"workload": f"append_{n}_{wl.name}", "tokens": n, "hidden": wl.hidden,
                      "row_dim": wl.row_dim, "latent_norm": True}}
    # whole call against HBM: hidden states and W_DKV read once, rows and ids written,
    # slots / ids / positions read (4 bytes each), the norm weight
    esz = 2 if st == "bf16" else 4
    nbytes = n * wl.hidden * esz + wl.row_dim * wl.hidden * esz + n * (wl.row_dim * esz + 4) + 12 * n + \
        wl.latent_dim * esz
    gbs = nbytes / (ms * 1e-3) / 1e9
    tflops = flops / (ms * 1e-3) / 1e12
    if st == "bf16" and flops / (MFMA_BF16_PEAK_TFLOPS * 1e12) > nbytes / (HBM_PEAK_GBPS * 1e9):
        # many tokens: the product W_DKV x is the longer of the two floors
        out["roofline"] = {"bound": "mfma", "kernel": "eg_mla_append_ws (whole call)", "achieved": tflops,
                           "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": tflops / MFMA_BF16_PEAK_TFLOPS,
                           "traffic": None, "algorithmic_flops_per_call": flops, "hbm_gbs": gbs}
    else:
        out["roofline"] = {"bound": "hbm", "kernel": "eg_mla_append_ws (whole call)", "achieved": gbs,
                           "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": gbs / HBM_PEAK_GBPS, "traffic": None,
                           "algorithmic_bytes_per_call": nbytes, "mfma_tflops": tflops}
    print(json.dumps(out), flush=True)


def literal_main(args):
    """Times eg_mla_decode_literal on the decode workload (one step = one call)."""
    import torch

    from paper_2509_16686_amd import binding as B
    from paper_2509_16686_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    L = B.lib()
    hip = Hip()
    wl = W.WORKLOADS[args.workload] if args.workload < len(W.WORKLOADS) else W.MLA_DC320_BIGBATCH
    log(f"bench: generating {wl.name} with the literal gate ({args.literal})")
    inp = W.generate(wl)
    lg = W.generate_literal_gate(wl)
    flags = {"mul_ln": 0, "mul": B.LITERAL_NO_LN, "add_ln": B.LITERAL_ADD,
             "add": B.LITERAL_NO_LN | B.LITERAL_ADD}[args.literal]
    dd = B.stage_decode(inp)
    gate = B.to_device_tensor(lg.gate_full, wl.dtype)
    lw, lb = B.to_device_tensor(lg.ln_w, wl.dtype), B.to_device_tensor(lg.ln_b, wl.dtype)
    nslots = int(dd.cache.shape[0])
    ws_bytes = B.decode_literal_workspace_size(dd.dims, wl.batch, dd.max_pages)
    ws = B.alloc_workspace(ws_bytes)
    stream = torch.cuda.current_stream().cuda_stream
    a = (ctypes.byref(dd.dims), wl.batch, dd.q.data_ptr(), dd.cache.data_ptr(), dd.ids.data_ptr(), gate.data_ptr(),
         dd.w_uk.data_ptr(), dd.w_uv.data_ptr(), lw.data_ptr(), lb.data_ptr(), flags, dd.seq_lens.data_ptr(),
         None if dd.page_table is None else dd.page_table.data_ptr(), dd.max_pages, nslots, ws.data_ptr(), ws_bytes,
         dd.out.data_ptr(), stream)
    call = L.eg_mla_decode_literal
    K, Wm = args.steps, args.warmup
    for _ in range(max(Wm, 1)):
        assert call(*a) == 0
    torch.cuda.synchronize()
    e0, e1 = hip.event(), hip.event()
    torch.cuda._sleep(20_000_000)
    hip.record(e0, stream)
    for _ in range(K):
        call(*a)
    hip.record(e1, stream)
    torch.cuda.synchronize()
    ms = hip.elapsed_ms(e0, e1) / K
    tokens = inp.total_tokens()
    width = wl.heads * (wl.head_dim + wl.v_head_dim)
    flops = tokens * 2 * width * wl.latent_dim
    log(f"bench: literal ({args.literal}) {ms * 1e3:.1f} us/step, {wl.batch / ms * 1e3:.0f} tokens/s; up-projection "
        f"{flops / 1e9:.1f} GFLOP per step")
    out = {"metric": METRIC.replace("eg_mla_decode", "eg_mla_decode_literal"), "value": wl.batch / (ms * 1e-3),
           "unit": "tokens/s", "n_gpus": 1, "steps": K, "warmup": Wm, "ms_per_step": ms, "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
           "config": {"workload": wl.name, "gate": f"literal ({args.literal}): after the up-projection, width {width}",
                      "batch": wl.batch, "heads": wl.heads, "latent_dim": wl.latent_dim,
                      "context": wl.seq_len if wl.seq_len else list(wl.seq_len_range)},
           "up_projection_gflop_per_step": flops / 1e9,
           "gate_bytes_per_step": tokens * width * 2}
    # whole step against HBM: each cached token's gate row once, its cache row and id,
    # the weights, queries and outputs (the value halves re-read by the kernel's
    # second pass are its own overhead, not counted)
    nbytes = tokens * (width * 2 + (wl.latent_dim + wl.rope_dim) * 2 + 4) + \
        wl.heads * (wl.head_dim + wl.v_head_dim) * wl.latent_dim * 2 + \
        wl.batch * wl.heads * (wl.head_dim + wl.rope_dim + wl.v_head_dim) * 2 + width * 4
    gbs = nbytes / (ms * 1e-3) / 1e9
    out["roofline"] = {"bound": "hbm", "kernel": "eg_mla_decode_literal (whole call: tile and merge kernels)",
                       "achieved": gbs, "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": gbs / HBM_PEAK_GBPS,
                       "traffic": None, "algorithmic_bytes_per_call": nbytes}
    print(json.dumps(out), flush=True)


def layer_group_main(args):
    """Times a layer group (App. H): G layers decode one shared cache back to back,
    each with its own query, W_UK, W_UV and gate table, against G layers each
    decoding a cache of its own (no sharing).  One step = the G decode calls."""
    import numpy as np
    import torch

    from paper_2509_16686_amd import accounting as A
    from paper_2509_16686_amd import binding as B
    from paper_2509_16686_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    L = B.lib()
    hip = Hip()
    G = args.layer_group
    wl = W.WORKLOADS[args.workload] if args.workload < len(W.WORKLOADS) else W.MLA_DC320_BIGBATCH
    log(f"bench: generating a group of {G} layers of {wl.name}")
    layers = W.generate_layer_group(wl, G)
    staged = [B.stage_decode(l) for l in layers]
    cache_bytes = staged[0].cache.numel() * staged[0].cache.element_size() + staged[0].ids.numel() * 4
    per_layer = sum(t.numel() * t.element_size() for t in (staged[0].gate, staged[0].w_uk, staged[0].w_uv,
                                                            staged[0].q))
    # rotating copies of the whole group (its own caches in the unshared case), so that
    # nothing is served from the MALL from one step to the next
    R = max(1, math.ceil(args.rotate_bytes / (G * (cache_bytes + per_layer))))
    ws_bytes = B.decode_workspace_size(staged[0].dims, wl.batch, staged[0].max_pages)
    ws = B.alloc_workspace(ws_bytes)
    stream = torch.cuda.current_stream().cuda_stream

    def copy_layer(dd, cache, ids):
        return B.DeviceDecode(dims=dd.dims, q=dd.q.clone(), cache=cache, ids=ids, gate=dd.gate.clone(),
                              w_uk=dd.w_uk.clone(), w_uv=dd.w_uv.clone(), seq_lens=dd.seq_lens,
                              page_table=dd.page_table, max_pages=dd.max_pages, out=torch.empty_like(dd.out))

    shared, separate = [], []
    for _ in range(R):
        c, i = staged[0].cache.clone(), staged[0].ids.clone()
        shared.append([copy_layer(dd, c, i) for dd in staged])
        separate.append([copy_layer(dd, staged[0].cache.clone(), staged[0].ids.clone()) for dd in staged])
    call = L.eg_mla_decode

    def args_of(dd):
        return (ctypes.byref(dd.dims), wl.batch, dd.q.data_ptr(), dd.cache.data_ptr(), dd.ids.data_ptr(),
                dd.gate.data_ptr(), dd.w_uk.data_ptr(), dd.w_uv.data_ptr(), dd.seq_lens.data_ptr(),
                None if dd.page_table is None else dd.page_table.data_ptr(), dd.max_pages, int(dd.cache.shape[0]),
                ws.data_ptr(), ws_bytes, dd.out.data_ptr(), stream)

    K, Wm = args.steps, args.warmup

    def time_group(groups):
        steps = [[args_of(dd) for dd in groups[k % R]] for k in range(K)]
        for k in range(max(Wm, 1)):
            for a in steps[k % K]:
                assert call(*a) == 0
        torch.cuda.synchronize()
        e0, e1 = hip.event(), hip.event()
        torch.cuda._sleep(40_000_000)
        hip.record(e0, stream)
        for st in steps:
            for a in st:
                call(*a)
        hip.record(e1, stream)
        torch.cuda.synchronize()
        return hip.elapsed_ms(e0, e1) / K

    ms_shared = time_group(shared)
    ms_sep = time_group(separate)
    layers_model = MODEL_LAYERS
    cache_tok = A.cache_bytes_per_token(layers=layers_model, latent_dim=wl.latent_dim, rope_dim=wl.rope_dim,
                                        elem_bytes=wl.elem_bytes, layer_group=G)
    cache_tok1 = A.cache_bytes_per_token(layers=layers_model, latent_dim=wl.latent_dim, rope_dim=wl.rope_dim,
                                         elem_bytes=wl.elem_bytes)
    log(f"bench: layer group of {G}: {ms_shared * 1e3 / G:.2f} us per layer on the shared cache, "
        f"{ms_sep * 1e3 / G:.2f} us per layer on separate caches; cache {cache_tok} B/token over "
        f"{layers_model} layers ({cache_tok1} B without grouping)")
    out = {"metric": METRIC, "value": wl.batch / (ms_shared * 1e-3 / G), "unit": "tokens/s", "n_gpus": 1,
           "steps": K, "warmup": Wm, "ms_per_step": ms_shared, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16" if wl.dtype == "bf16" else "fp32", "data": "synthetic",
           "config": {"workload": f"layer_group{G}_{wl.name}", "layers_per_step": G, "rotating_copies": R},
           "layer_group": {"size": G, "us_per_layer_shared": ms_shared * 1e3 / G,
                           "us_per_layer_separate": ms_sep * 1e3 / G,
                           "cache_bytes_per_token_model": cache_tok, "cache_bytes_per_token_model_ungrouped": cache_tok1,
                           "model_layers": layers_model}}
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", type=int, default=1,
                    help="index into workloads.WORKLOADS; 5 = the plain-MLA comparison (d_c 320, all-ones gate) "
                         "of the large-batch case")
    ap.add_argument("--path", choices=["auto", "valu", "mfma"], default="auto")
    ap.add_argument("--split", type=int, default=0, help="tokens per split (0 = automatic)")
    ap.add_argument("--id-slices", type=int, default=0, choices=[0, 1, 8],
                    help="token-id slices per split of the d_c=128 kernel (0 = automatic)")
    ap.add_argument("--rotate-bytes", type=float, default=1.0e9)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibration-copy-mib", type=int, default=0,
                    help="also run one device copy of this many MiB (a known byte count for profiler counters)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--prefill", default="", metavar="BxT",
                    help="time the causal prefill (eg_mla_prefill_varlen) of B packed sequences of T tokens "
                         "instead of the decode, e.g. 8x4096")
    ap.add_argument("--append", type=int, default=0, metavar="N",
                    help="time eg_mla_append of N new tokens (the default workload's layer, with the latent norm) "
                         "instead of the decode")
    ap.add_argument("--literal", default="", choices=["", "mul_ln", "mul", "add_ln", "add"],
                    help="time eg_mla_decode_literal (the paper-literal gate after the up-projection, with or "
                         "without the LayerNorm, product or sum) on the same workload instead of the decode")
    ap.add_argument("--unfolded-gate", type=int, default=0, metavar="E",
                    help="unfolded gate with embedding width E (the paper recommends 512): every step first "
                         "computes one gate row per cache row from its token embedding (eg_mla_gate_rows), then "
                         "decodes with the row indices as ids; 0 = the folded gate table")
    ap.add_argument("--unfolded-distinct", action="store_true",
                    help="with --unfolded-gate: each step computes the gate row of each distinct token id once "
                         "into a [V, d_c] table (eg_mla_gate_table), which the decode takes with the step's own ids")
    ap.add_argument("--layer-group", type=int, default=0, metavar="G",
                    help="time G layers of a layer group (App. H) decoding one shared cache, against G layers "
                         "with caches of their own")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py: this build measures one GPU; --gpus {args.gpus} (WORLD_SIZE {world}) is not supported. "
              "The decode path shards by sequence with no communication; see the design notes.", file=sys.stderr)
        sys.exit(2)

    if args.prefill:
        return prefill_main(args)
    if args.literal:
        return literal_main(args)
    if args.append:
        return append_main(args)
    if args.layer_group:
        return layer_group_main(args)

    import numpy as np
    import torch

    from paper_2509_16686_amd import accounting as A
    from paper_2509_16686_amd import binding as B
    from paper_2509_16686_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    L = B.lib()
    hip = Hip()
    wl = W.WORKLOADS[args.workload] if args.workload < len(W.WORKLOADS) else W.MLA_DC320_BIGBATCH
    log(f"bench: generating {wl.name}")
    inp = W.generate(wl)
    traffic = A.decode_bytes(batch=wl.batch, heads=wl.heads, head_dim=wl.head_dim, v_head_dim=wl.v_head_dim,
                             latent_dim=wl.latent_dim, rope_dim=wl.rope_dim, elem_bytes=wl.elem_bytes,
                             total_tokens=inp.total_tokens(), distinct_ids=inp.unique_ids())
    copies_bytes = (inp.latent_cache.nbytes + inp.token_ids.nbytes + inp.gate_table.nbytes + inp.q.nbytes +
                    inp.w_uk.nbytes + inp.w_uv.nbytes)
    R = max(1, math.ceil(args.rotate_bytes / copies_bytes))
    dd0 = B.stage_decode(inp)
    copies = [dd0]
    for _ in range(R - 1):
        copies.append(B.DeviceDecode(dims=dd0.dims, q=dd0.q.clone(), cache=dd0.cache.clone(), ids=dd0.ids.clone(),
                                     gate=dd0.gate.clone(), w_uk=dd0.w_uk.clone(), w_uv=dd0.w_uv.clone(),
                                     seq_lens=dd0.seq_lens.clone(),
                                     page_table=None if dd0.page_table is None else dd0.page_table.clone(),
                                     max_pages=dd0.max_pages, out=torch.empty_like(dd0.out)))
    E = args.unfolded_gate
    if E > 0:
        # per-step gate rows: one per cache row, written to one buffer the decode then reads
        ge = W.generate_gate_embedding(wl, E)
        emb_d, wue_d = B.to_device_tensor(ge.emb, wl.dtype), B.to_device_tensor(ge.w_ue, wl.dtype)
        n_rows = inp.num_rows
        n_distinct = int(np.unique(np.clip(inp.token_ids, 0, wl.vocab - 1)).size)
        if args.unfolded_distinct:
            # a [V, d_c] table refilled each step for the step's distinct ids;
            # the decode keeps its own ids and dims
            row_gate = torch.empty((wl.vocab, wl.latent_dim), dtype=dd0.gate.dtype, device="cuda")
            dims_g = B.dims_for(wl)
            marks_bytes = B.gate_table_marks_size(dims_g, E, wl.vocab)
            marks = torch.zeros((marks_bytes + 3) // 4, dtype=torch.int32, device="cuda")
            for k, c in enumerate(copies):
                c.gate_src_ids, c.gate = c.ids, row_gate
                c.emb = emb_d if k == 0 else emb_d.clone()
            gate_call = L.eg_mla_gate_table
        else:
            row_gate = torch.empty((n_rows, wl.latent_dim), dtype=dd0.gate.dtype, device="cuda")
            row_ids = torch.arange(n_rows, dtype=torch.int32, device="cuda")
            dims_u = B.dims_for(wl.replace(vocab=n_rows))
            # one embedding table per rotating copy, so that the table (tens of MB)
            # is not served from the 256 MB MALL from one step to the next
            for k, c in enumerate(copies):
                c.gate_src_ids, c.dims, c.gate, c.ids = c.ids, dims_u, row_gate, row_ids
                c.emb = emb_d if k == 0 else emb_d.clone()
            gate_call = L.eg_mla_gate_rows
            # the decode now gathers one distinct gate row per cache row
            traffic = A.decode_bytes(batch=wl.batch, heads=wl.heads, head_dim=wl.head_dim,
                                     v_head_dim=wl.v_head_dim, latent_dim=wl.latent_dim, rope_dim=wl.rope_dim,
                                     elem_bytes=wl.elem_bytes, total_tokens=inp.total_tokens(),
                                     distinct_ids=inp.total_tokens())
    path = {"auto": B.PATH_AUTO, "valu": B.PATH_VALU, "mfma": B.PATH_MFMA}[args.path]
    plan0 = B.make_plan(path, args.split, id_slices=args.id_slices)
    ws_bytes = B.decode_workspace_size(dd0.dims, wl.batch, dd0.max_pages, plan0)
    assert ws_bytes > 0, "no plan for this workload"
    ws = B.alloc_workspace(ws_bytes)
    stream = torch.cuda.current_stream().cuda_stream
    K, Wm = args.steps, args.warmup
    log(f"bench: {R} rotating input copies of {copies_bytes / 1e6:.1f} MB, workspace {ws_bytes / 1e6:.1f} MB")

    ev0 = [hip.event() for _ in range(K)]
    ev1 = [hip.event() for _ in range(K)]
    plans = [B.make_plan(path, args.split, ev0[k], ev1[k], id_slices=args.id_slices) for k in range(K)]

    def argset(dd, plan):
        return (ctypes.byref(dd.dims), wl.batch, dd.q.data_ptr(), dd.cache.data_ptr(), dd.ids.data_ptr(),
                dd.gate.data_ptr(), dd.w_uk.data_ptr(), dd.w_uv.data_ptr(), dd.seq_lens.data_ptr(),
                None if dd.page_table is None else dd.page_table.data_ptr(), dd.max_pages,
                int(dd.cache.shape[0]), ws.data_ptr(), ws_bytes, dd.out.data_ptr(), stream, ctypes.byref(plan))

    call = L.eg_mla_decode_planned

    stamp = [0]

    def gate_args(dd):
        if args.unfolded_distinct:
            # a fresh stamp for every call: each call computes every distinct id of its step
            stamp[0] += 1
            return (ctypes.byref(dims_g), E, int(dd.emb.shape[0]), n_rows, dd.gate_src_ids.data_ptr(),
                    dd.emb.data_ptr(), wue_d.data_ptr(), row_gate.data_ptr(), marks.data_ptr(), marks_bytes,
                    stamp[0], stream)
        return (ctypes.byref(dd.dims), E, int(dd.emb.shape[0]), n_rows, dd.gate_src_ids.data_ptr(),
                dd.emb.data_ptr(), wue_d.data_ptr(), row_gate.data_ptr(), stream)

    def step(dd, plan):
        """One step: a list of (function, arguments) calls."""
        calls = [(call, argset(dd, plan))]
        if E > 0:
            calls.insert(0, (gate_call, gate_args(dd)))
        return calls

    warm_args = [step(copies[k % R], plan0) for k in range(max(Wm, 1))]
    step_args = [step(copies[k % R], plan0) for k in range(K)]
    timed_args = [step(copies[k % R], plans[k]) for k in range(K)]

    for s in warm_args:
        for f, a in s:
            st = f(*a)
            assert st == 0, B.status_string(st)
    torch.cuda.synchronize()
    # host enqueue rate, to size the spin that hides launch overhead
    h0 = time.perf_counter()
    for s in warm_args:
        for f, a in s:
            f(*a)
    host_per_call = (time.perf_counter() - h0) / len(warm_args)
    torch.cuda.synchronize()

    # calibrate the spin kernel
    s0, s1 = hip.event(), hip.event()
    hip.record(s0, stream)
    torch.cuda._sleep(1_000_000)
    hip.record(s1, stream)
    torch.cuda.synchronize()
    cycles_per_ms = 1_000_000 / max(hip.elapsed_ms(s0, s1), 1e-3)
    spin_ms = 2.0 * host_per_call * K * 1e3 + 5.0

    def timed_loop(arglist):
        """K calls queued behind a spin kernel; returns (GPU ms between the outer events, wall s)."""
        t_start, t_stop = hip.event(), hip.event()
        torch.cuda.synchronize()
        wall0 = time.perf_counter()
        torch.cuda._sleep(int(spin_ms * cycles_per_ms))
        hip.record(t_start, stream)
        for s in arglist:
            for f, a in s:
                f(*a)
        hip.record(t_stop, stream)
        enq = time.perf_counter() - wall0
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
        if enq * 1e3 > spin_ms:
            log(f"bench: warning: enqueue took {enq * 1e3:.1f} ms > spin {spin_ms:.1f} ms; GPU may have idled")
        return hip.elapsed_ms(t_start, t_stop), wall

    if args.calibration_copy_mib > 0:
        src = torch.empty(args.calibration_copy_mib << 20, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # (1) whole-call throughput: plain back-to-back calls, nothing between them
    total_ms, wall = timed_loop(step_args)
    # (2) the split kernel alone: the same calls with a start/stop event pair per split-kernel
    #     launch, stamped by the dispatch itself (hipExtLaunchKernelGGL), on the kernel's stream
    timed_loop(timed_args)
    kernel_ms = [hip.elapsed_ms(ev0[k], ev1[k]) for k in range(K)]
    if E > 0:
        # (3) the gate-row kernel alone: an event pair around each launch (one kernel per call)
        g0 = [hip.event() for _ in range(K)]
        g1 = [hip.event() for _ in range(K)]
        torch.cuda.synchronize()
        torch.cuda._sleep(int(spin_ms * cycles_per_ms))
        for k in range(K):
            hip.record(g0[k], stream)
            gate_call(*gate_args(copies[k % R]))
            hip.record(g1[k], stream)
        torch.cuda.synchronize()
        gate_ms = float(np.mean([hip.elapsed_ms(g0[k], g1[k]) for k in range(K)]))

    ms_per_step = total_ms / K
    k_avg_ms = float(np.mean(kernel_ms))
    # the d_c 128 split kernel absorbs the query itself (automatic plan, no id slices, d_h 128)
    absorbing = (wl.dtype == "bf16" and wl.latent_dim == 128 and wl.rope_dim == 64 and wl.head_dim == 128
                 and args.path != "valu" and args.id_slices != 8)
    k_bytes = traffic.main_kernel_absorbing if absorbing else traffic.main_kernel
    achieved = k_bytes / (k_avg_ms * 1e-3) / 1e9
    # counters were taken on the default workload with the automatic plan only
    t_bytes = recorded_traffic() if (args.workload == 1 and args.path == "auto" and args.split == 0
                                     and args.id_slices == 0 and E == 0) else None
    traffic_gbps = None if t_bytes is None else t_bytes / (k_avg_ms * 1e-3) / 1e9
    tokens_per_s = wl.batch / (ms_per_step * 1e-3)
    log(f"bench: {ms_per_step * 1e3:.2f} us/step, split kernel {k_avg_ms * 1e3:.2f} us "
        f"({achieved:.0f} GB/s, {100 * achieved / HBM_PEAK_GBPS:.1f}% of peak), host {host_per_call * 1e6:.1f} us/call, "
        f"wall {wall:.3f} s")

    out = {
        "metric": METRIC,
        "value": tokens_per_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": Wm,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "fp32",
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": wl.batch, "heads": wl.heads, "head_dim": wl.head_dim,
                   "latent_dim": wl.latent_dim, "rope_dim": wl.rope_dim, "vocab": wl.vocab,
                   "context": wl.seq_len if wl.seq_len else list(wl.seq_len_range), "paged": wl.paged,
                   "storage": wl.dtype, "path": args.path, "split_tokens": args.split, "id_slices": args.id_slices,
                   "rotating_copies": R,
                   "gate": (f"unfolded, embedding width {E}" + (", per distinct id" if args.unfolded_distinct else ""))
                   if E > 0 else "folded table"},
        "hbm_gbps_call": traffic.total / (ms_per_step * 1e-3) / 1e9,
        "hbm_frac_call": traffic.total / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        # estimate, not a measurement: every layer of a 24-layer model taking one such call
        "model_tokens_per_s_estimate": tokens_per_s / MODEL_LAYERS,
        # context: a plain streaming read of ~60 MiB in one launch (committed reference profile)
        "stream_read_ceiling_gbps": recorded_stream_ceiling(),
        "roofline": {"bound": "hbm", "kernel": split_kernel_name(wl, args.path),
                     "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": traffic_gbps,
                     "algorithmic_bytes_per_launch": k_bytes, "traffic_bytes_per_launch": t_bytes, "kernel_us": k_avg_ms * 1e3},
    }
    if E > 0:
        # algorithmic: the gathered embedding rows, the gate rows written, the ids, W^UE once (distinct
        # ids: one embedding row and one table row per distinct id, the ids and one claim per row)
        n_g = n_distinct if args.unfolded_distinct else n_rows
        g_bytes = (n_g * (E * wl.elem_bytes + wl.latent_dim * wl.elem_bytes) + n_rows * 4 * (2 if args.unfolded_distinct else 1)
                   + wl.latent_dim * E * wl.elem_bytes)
        out["unfolded_gate"] = {"emb_dim": E, "rows": n_rows, "distinct_ids": n_distinct,
                                "per_distinct_id": bool(args.unfolded_distinct), "gate_rows_us": gate_ms * 1e3,
                                "gate_rows_gbps": g_bytes / (gate_ms * 1e-3) / 1e9,
                                "gate_rows_tflops": 2.0 * n_g * E * wl.latent_dim / (gate_ms * 1e-3) / 1e12,
                                "algorithmic_bytes": g_bytes}
        log(f"bench: gate rows {gate_ms * 1e3:.2f} us ({out['unfolded_gate']['gate_rows_gbps']:.0f} GB/s)")
    if not args.no_cpu_baseline:
        log(f"bench: timing the fp64 oracle on the host for ~{args.cpu_seconds:.0f} s")
        out["cpu_baseline"] = cpu_baseline(inp, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
