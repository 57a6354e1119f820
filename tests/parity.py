"""Shared helpers of the GPU parity tests: run the oracle and the HIP path on
the same seeded inputs and compare at the stated tolerances."""
import sys

import numpy as np

from oracle import eg_mla_oracle as orc

# Tolerances against the fp64 oracle.
BF16_MAX_ABS = 1e-2
BF16_REL_L2 = 5e-3
FP32_MAX_ABS = 1e-5


def say(msg: str) -> None:
    """Names the case about to run on the GPU (flushed before the launch)."""
    print(msg, file=sys.stderr, flush=True)


def oracle_decode(inp, **over):
    wl = inp.wl
    args = dict(latent_dim=wl.latent_dim, head_dim=wl.head_dim, rope_dim=wl.rope_dim, storage=wl.dtype,
                page_table=inp.page_table, page_size=wl.page_size, max_pages=inp.max_pages)
    args.update(over)
    return orc.decode(inp.q, inp.latent_cache, inp.token_ids, inp.gate_table, inp.w_uk, inp.w_uv, inp.seq_lens,
                      **args)


def errors(got: np.ndarray, ref: np.ndarray):
    d = got - ref
    max_abs = float(np.abs(d).max()) if d.size else 0.0
    nrm = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(d) / nrm) if nrm > 0 else float(np.linalg.norm(d))
    return max_abs, rel


def bf16_elementwise_bound(ref: np.ndarray) -> np.ndarray:
    """Per-element bf16 bound: the stated absolute bound plus the rounding of a
    bf16 output of that size (half an ulp is at most 2^-8 |out| for the
    ulp spacing 2^-7 |out| of the binade)."""
    return BF16_MAX_ABS + 2.0 ** -8 * np.abs(ref)


def assert_close(got: np.ndarray, ref: np.ndarray, storage: str, what: str = ""):
    """Element-wise parity at the stated tolerances.

    fp32 storage: |got - ref| <= 1e-5 everywhere.  bf16 storage: relative L2
    error <= 5e-3, and every element within 1e-2 + 2^-8 |ref| (the output is
    itself rounded to bf16, which alone moves an element by up to 2^-8 |ref|;
    for outputs below 1 in size the bound is the plain 1e-2 plus at most
    4e-3).
    """
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    max_abs, rel = errors(got, ref)
    if storage == "fp32":
        say(f"  {what}: max_abs={max_abs:.3e} rel_l2={rel:.3e}")
        assert max_abs <= FP32_MAX_ABS, f"{what}: fp32 max abs err {max_abs:.3e} > {FP32_MAX_ABS}"
    else:
        ratio = float(np.max(np.abs(got - ref) / bf16_elementwise_bound(ref))) if ref.size else 0.0
        say(f"  {what}: max_abs={max_abs:.3e} rel_l2={rel:.3e} max|ref|={float(np.abs(ref).max()):.3g} "
            f"worst err/bound={ratio:.3f}")
        assert ratio <= 1.0, f"{what}: an element exceeds 1e-2 + 2^-8|ref| (worst err/bound {ratio:.3f})"
        assert rel <= BF16_REL_L2, f"{what}: bf16 rel L2 err {rel:.3e} > {BF16_REL_L2}"
    return max_abs, rel
