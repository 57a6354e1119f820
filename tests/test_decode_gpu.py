"""GPU parity of eg_mla_decode against the fp64 oracle, through the C ABI.

Covers the five workloads at full size in the automatic plan (the launch
configuration the benchmark times), both kernel paths, several split sizes,
ragged and paged layouts, and the degenerate cases (empty, single-token,
full-capacity and shorter-than-a-split sequences, peaked logits).
"""
import functools

import numpy as np
import pytest

from paper_2509_16686_amd import binding as B
from paper_2509_16686_amd import workloads as W
from parity import assert_close, oracle_decode, say

pytestmark = pytest.mark.gpu


@functools.lru_cache(maxsize=None)
def full_inputs(idx):
    return W.generate(W.WORKLOADS[idx])


@functools.lru_cache(maxsize=None)
def full_ref(idx):
    return oracle_decode(full_inputs(idx))


def gpu_decode(inp, plan=None):
    dd = B.stage_decode(inp)
    B.run_decode(dd, plan=plan)
    import torch
    torch.cuda.synchronize()
    return B.out_to_f64(dd.out)


@pytest.mark.parametrize("idx", [0, 1, 2, 3, 4])
def test_workload_full_size_auto_plan(gpu, idx):
    inp = full_inputs(idx)
    wl = inp.wl
    say(f"decode {wl.name} seed={wl.seed} auto plan")
    got = gpu_decode(inp)
    max_abs, rel = assert_close(got, full_ref(idx), wl.dtype, wl.name)
    say(f"  max_abs={max_abs:.3e} rel_l2={rel:.3e}")


def test_plain_mla_dc320_all_ones_gate(gpu):
    wl = W.MLA_DC320_BIGBATCH.replace(batch=32)
    inp = W.generate(wl)
    say(f"decode {wl.name} (batch 32) auto plan")
    got = gpu_decode(inp)
    assert_close(got, oracle_decode(inp), "bf16", wl.name)
    # an all-ones gate is plain MLA: the oracle without the gate gives the same reference
    np.testing.assert_array_equal(oracle_decode(inp), oracle_decode(inp, use_gate=False))


SMALL = W.WORKLOADS[1].replace(name="small_h16", batch=4, seq_len=None, seq_len_range=(1, 900), paged=True,
                               page_size=64, seed=21)


# (path, token-id slices of the d_c = 128 MFMA kernel)
PATHS = [(B.PATH_VALU, 0), (B.PATH_MFMA, 1), (B.PATH_MFMA, 8)]


@pytest.mark.parametrize("path,slices", PATHS)
@pytest.mark.parametrize("split", [32, 64, 256, 2048, 4096])
def test_small_ragged_paged_all_splits(gpu, path, slices, split):
    inp = W.generate(SMALL, seq_lens=np.array([1, 33, 777, 900]))
    say(f"decode small ragged paged path={path} slices={slices} split={split}")
    got = gpu_decode(inp, B.make_plan(path, split, id_slices=slices))
    assert_close(got, oracle_decode(inp), "bf16", f"path {path} slices {slices} split {split}")


@pytest.mark.parametrize("slices", [1, 8])
def test_id_slices_skewed_and_empty(gpu, slices):
    # every id in one slice (7 of 8 slices without tokens), and sequences of 1..7 tokens whose
    # slices are mostly empty: the merge must skip partials without tokens
    inp = W.generate(SMALL.replace(seed=25, batch=6), seq_lens=np.array([1, 2, 7, 300, 0, 901]))
    ids_one = inp.token_ids.copy()
    ids_one[:] = (ids_one // 8) * 8 + 5
    ids_one[ids_one >= inp.wl.vocab] -= 8
    for what, ids in (("random ids", inp.token_ids.copy()), ("one slice", ids_one)):
        inp.token_ids[:] = ids
        say(f"decode id slices={slices} {what}")
        got = gpu_decode(inp, B.make_plan(B.PATH_MFMA, 256, id_slices=slices))
        assert np.all(got[4] == 0)
        assert_close(got, oracle_decode(inp), "bf16", f"slices {slices} {what}")


@pytest.mark.parametrize("paged", [False, True])
def test_pages_not_multiple_of_four(gpu, paged):
    # 6-token pages: slots of 4 consecutive positions are not 16-byte aligned, so the
    # sliced kernel loads ids one by one; contiguous capacity 18 is not a multiple of 4 either
    wl = SMALL.replace(seed=26, batch=4, page_size=6, paged=paged)
    inp = W.generate(wl, seq_lens=np.array([13, 5, 1, 12]))
    for slices in (1, 8):
        say(f"decode 6-token pages paged={paged} slices={slices}")
        got = gpu_decode(inp, B.make_plan(B.PATH_MFMA, 32, id_slices=slices))
        assert_close(got, oracle_decode(inp), "bf16", f"P=6 paged={paged} slices {slices}")


@pytest.mark.parametrize("path,slices", PATHS)
def test_edge_lengths(gpu, path, slices):
    wl = SMALL.replace(batch=6, paged=False, seq_len_range=(1, 320))
    # empty, single token, full capacity, exactly one tile, one past a tile, shorter than the split
    lens = np.array([0, 1, 320, 32, 33, 100])
    inp = W.generate(wl, seq_lens=lens)
    say(f"decode edge lengths {lens.tolist()} path={path} slices={slices}")
    got = gpu_decode(inp, B.make_plan(path, 128, id_slices=slices))
    ref = oracle_decode(inp)
    assert np.all(got[0] == 0)
    assert_close(got, ref, "bf16", "edge lengths")


def test_many_head_groups_and_dc512(gpu):
    wl = W.WORKLOADS[4].replace(batch=3, seq_len_range=(50, 700), seed=41)
    inp = W.generate(wl)
    for path in (B.PATH_VALU, B.PATH_MFMA):
        say(f"decode h128 dc512 ragged paged path={path}")
        assert_close(gpu_decode(inp, B.make_plan(path, 256)), oracle_decode(inp), "bf16", f"path {path}")


@pytest.mark.parametrize("heads,split", [(256, 32), (256, 2048), (64, 256)])
def test_head_blocks_dc512(gpu, heads, split):
    # the head-split kernel takes heads in blocks of 64: 256 heads run four
    # blocks per token range, 64 heads a single one
    wl = W.WORKLOADS[4].replace(name=f"h{heads}_dc512", heads=heads, batch=2, seq_len_range=(40, 300), seed=43)
    inp = W.generate(wl)
    say(f"decode h{heads} dc512 ragged paged split={split}")
    assert_close(gpu_decode(inp, B.make_plan(B.PATH_MFMA, split)), oracle_decode(inp), "bf16", f"h{heads} split {split}")


def test_edge_lengths_dc512(gpu):
    wl = W.WORKLOADS[4].replace(name="edge_dc512", batch=7, paged=False, seq_len_range=(1, 64), seed=44)
    # empty, one token, a partial tile, one tile, one past a tile, two tiles plus one, full capacity
    lens = np.array([0, 1, 15, 16, 17, 33, 64])
    inp = W.generate(wl, seq_lens=lens)
    say(f"decode dc512 edge lengths {lens.tolist()}")
    got = gpu_decode(inp, B.make_plan(B.PATH_MFMA, 32))
    assert np.all(got[0] == 0)
    assert_close(got, oracle_decode(inp), "bf16", "dc512 edge lengths")


@pytest.mark.parametrize("case", ["mixed", "short", "one_long"])
def test_balanced_schedule_dc512(gpu, case):
    # The 128-head kernel splits the batch's tokens evenly over its work-groups:
    # ranges that start mid-sequence, span many short or empty sequences, or
    # hold less than a token each (fewer tokens than work-groups).
    wl = W.WORKLOADS[4].replace(name=f"sched_{case}_dc512", paged=True, seed=45)
    if case == "mixed":
        lens = np.array([0, 1, 2100, 0, 17, 4097, 5, 0, 3, 1500, 2, 0])
    elif case == "short":
        lens = np.array([1, 0, 2, 3, 0, 1, 5, 4, 1, 0, 2, 7] * 4)
    else:
        lens = np.array([0, 6000, 0])
    wl = wl.replace(batch=len(lens), seq_len_range=(1, int(max(lens.max(), 64))))
    inp = W.generate(wl, seq_lens=lens)
    say(f"decode dc512 balanced schedule {case}: {int(lens.sum())} tokens, {len(lens)} sequences")
    got = gpu_decode(inp)
    assert np.all(got[lens == 0] == 0)
    assert_close(got, oracle_decode(inp), "bf16", f"balanced {case}")


@pytest.mark.parametrize("batch", [300, 700])
def test_balanced_schedule_large_batch(gpu, batch):
    # More sequences than the schedule's work-group has threads (256): its
    # prefix sums over the lengths run in several passes; 64 heads (one head
    # block), lengths 0 .. 40 with a quarter of the sequences empty.
    wl = W.WORKLOADS[4].replace(name=f"sched_b{batch}_h64_dc512", heads=64, paged=True, seed=49, batch=batch,
                                seq_len_range=(1, 40))
    lens = np.random.default_rng(batch).integers(0, 41, size=batch)
    lens[::4] = 0
    inp = W.generate(wl, seq_lens=lens)
    say(f"decode dc512 balanced schedule, {batch} sequences: {int(lens.sum())} tokens")
    got = gpu_decode(inp)
    assert np.all(got[lens == 0] == 0)
    assert_close(got, oracle_decode(inp), "bf16", f"balanced batch {batch}")


@pytest.mark.parametrize("total", [393310, 395300])
def test_list_chunk_edges_dc512(gpu, total):
    # Token ranges just past one token list (3072 tokens) per work-group at
    # 128 heads (128 ranges on a 256-CU device): the second list of a range
    # holds a lone unit (393310 tokens: 3072 or 3073 per range) or one to two
    # units (395300: 3088 or 3089), the ends of the value product's pairs.
    lens = np.array([total - 5, 5])
    wl = W.WORKLOADS[4].replace(name=f"chunk_edges_{total}_dc512", batch=2, paged=True, seed=48,
                                seq_len_range=(1, int(lens.max())))
    inp = W.generate(wl, seq_lens=lens)
    say(f"decode dc512 list-chunk edges: {total} tokens over 2 sequences")
    assert_close(gpu_decode(inp), oracle_decode(inp), "bf16", f"chunk edges {total}")


def test_peaked_logits_dc512(gpu):
    # query x 8: logits of standard deviation about 8, so the softmax is sharp
    # and a score error of 2^-9 relative (one bf16 rounding of either operand)
    # moves the output by more than the bar; the 128-head kernel's fp16
    # operands (2^-12) stay within it.  Running maxima also grow by more than
    # 2^8 between the tiles of a range, so the kernel rescales its accumulators.
    wl = W.WORKLOADS[4].replace(name="peaked_dc512", batch=4, seq_len_range=(2500, 3500), seed=46)
    inp = W.generate(wl)
    inp.q[:] = W.f32_to_bf16_bits(W.bf16_bits_to_f32(inp.q) * np.float32(8.0))
    say("decode dc512 peaked logits (q x 8)")
    got = gpu_decode(inp, B.make_plan(B.PATH_MFMA, 256))
    assert_close(got, oracle_decode(inp), "bf16", "peaked dc512")


def test_peaked_logits(gpu):
    inp = W.generate(SMALL.replace(seed=22), seq_lens=np.array([64, 500, 129, 7]))
    inp.q[:] = W.f32_to_bf16_bits(W.bf16_bits_to_f32(inp.q) * np.float32(8.0))
    say("decode peaked logits (q x 8)")
    got = gpu_decode(inp, B.make_plan(B.PATH_MFMA, 64))
    ref = oracle_decode(inp)
    assert_close(got, ref, "bf16", "peaked")


def test_paged_equals_contiguous_bitwise(gpu):
    wl = SMALL.replace(paged=False, batch=3, seed=23, seq_len_range=(100, 700))
    inp = W.generate(wl)
    P = wl.page_size
    rng = np.random.default_rng(0)
    perm = rng.permutation(3 * inp.max_pages).astype(np.int32)
    pt = perm.reshape(3, inp.max_pages)
    paged = W.generate(wl)
    for b in range(3):
        for j in range(int(inp.seq_lens[b])):
            src = inp.slot(b, j)
            dst = pt[b, j // P] * P + j % P
            paged.latent_cache[dst] = inp.latent_cache[src]
            paged.token_ids[dst] = inp.token_ids[src]
    paged.page_table = pt
    for path, slices in PATHS:
        say(f"decode paged vs contiguous path={path} slices={slices}")
        a = gpu_decode(inp, B.make_plan(path, 96, id_slices=slices))
        b = gpu_decode(paged, B.make_plan(path, 96, id_slices=slices))
        assert np.array_equal(a, b)


def test_repeatable_bitwise(gpu):
    inp = full_inputs(1)
    dd = B.stage_decode(inp)
    say("decode layer1b x3 repeatability")
    outs = []
    for _ in range(3):
        B.run_decode(dd)
        outs.append(B.out_to_f64(dd.out).copy())
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


@pytest.mark.parametrize("lens", [(1500, 700, 3, 4096), (512, 513, 0, 1)])
def test_fused_absorption_fallback_same_bits(gpu, monkeypatch, lens):
    """On the d_c 128 path the split kernel absorbs the query itself: each
    non-empty split of a sequence absorbs a share of its heads and publishes a
    stamp; a work-group that does not see every stamp within its poll limit
    absorbs all 16 heads itself.  Forcing that path from the host (a limit of
    0 polls) must give the same bits as the shared absorption, and both the
    oracle's result.  The lengths give 3, 2, 1 and 8 non-empty splits of 512
    tokens, one sequence of a single token and an empty one."""
    wl = W.WORKLOADS[1].replace(batch=len(lens), seq_len=4096)
    inp = W.generate(wl, seq_lens=np.array(lens, dtype=np.int32))
    dd = B.stage_decode(inp)
    say(f"decode fused absorption shared, lens={lens}")
    B.run_decode(dd)
    shared = B.out_to_f64(dd.out).copy()
    monkeypatch.setenv("EGMLA_SPIN_LIMIT", "0")
    say(f"decode fused absorption local, lens={lens}")
    B.run_decode(dd)
    local = B.out_to_f64(dd.out).copy()
    assert np.array_equal(shared, local)
    assert_close(shared, oracle_decode(inp), "bf16", "fused absorption")


def test_split_choice_changes_result_within_tolerance(gpu):
    inp = full_inputs(2)
    ref = full_ref(2)
    for split, slices in ((256, 1), (1024, 1), (2048, 1), (256, 8), (1024, 8), (4096, 8)):
        say(f"decode longctx split={split} slices={slices}")
        assert_close(gpu_decode(inp, B.make_plan(B.PATH_MFMA, split, id_slices=slices)), ref, "bf16",
                     f"split {split} slices {slices}")
    say("decode longctx VALU path")
    assert_close(gpu_decode(inp, B.make_plan(B.PATH_VALU, 0)), ref, "bf16", "valu")


@pytest.mark.parametrize("path,slices", PATHS)
def test_out_of_range_ids_and_lengths_are_clamped(gpu, path, slices):
    # lengths beyond the capacity clamp to the capacity; cached ids below 0 or
    # at or past V clamp into [0, V): the oracle is fed the clamped values
    inp = W.generate(SMALL.replace(seed=24, paged=False), seq_lens=np.array([10, 20, 30, 40]))
    V = inp.wl.vocab
    cap = inp.max_pages * inp.wl.page_size
    inp.seq_lens[:] = [10, 20, 30, 10 ** 6]
    used = np.concatenate([b * cap + np.arange(min(int(L), cap)) for b, L in enumerate(inp.seq_lens)])
    bad = np.random.default_rng(7).choice(used, size=64, replace=False)
    inp.token_ids[bad[:32]] = -3
    inp.token_ids[bad[32:]] = V + 7
    say(f"decode clamped ids and lengths path={path} slices={slices}")
    got = gpu_decode(inp, B.make_plan(path, 64, id_slices=slices))
    inp.seq_lens[:] = [10, 20, 30, cap]
    inp.token_ids[:] = np.clip(inp.token_ids, 0, V - 1)
    assert_close(got, oracle_decode(inp), "bf16", "clamped")


def test_out_of_range_ids_dc512(gpu):
    wl = W.WORKLOADS[4].replace(name="clamp_dc512", batch=3, seq_len_range=(40, 300), seed=47)
    inp = W.generate(wl)
    V = wl.vocab
    P = wl.page_size
    used = np.concatenate([inp.page_table[b, np.arange(L) // P].astype(np.int64) * P + np.arange(L) % P
                           for b, L in enumerate(inp.seq_lens)])
    bad = np.random.default_rng(8).choice(used, size=200, replace=False)
    inp.token_ids[bad[:100]] = -1
    inp.token_ids[bad[100:]] = V
    say("decode dc512 clamped ids")
    got = gpu_decode(inp)
    inp.token_ids[:] = np.clip(inp.token_ids, 0, V - 1)
    assert_close(got, oracle_decode(inp), "bf16", "clamped dc512")
