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


def assert_close(got: np.ndarray, ref: np.ndarray, storage: str, what: str = "", scaled: bool = False):
    """Element-wise parity at the stated tolerances.

    ``scaled=True`` (stress cases with outputs far above unit size: a few
    tokens, peaked logits) multiplies the bf16 max-abs bound by
    max(1, max|ref|): a bf16 output alone is rounded by up to 2^-9 |out|,
    and a bf16 probability or key error moves the output in proportion to
    the value vectors' size, so the absolute error scales with |out|.
    """
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    max_abs, rel = errors(got, ref)
    say(f"  {what}: max_abs={max_abs:.3e} rel_l2={rel:.3e} max|ref|={float(np.abs(ref).max()):.3g}")
    if storage == "fp32":
        assert max_abs <= FP32_MAX_ABS, f"{what}: fp32 max abs err {max_abs:.3e} > {FP32_MAX_ABS}"
    else:
        bound = BF16_MAX_ABS * (max(1.0, float(np.abs(ref).max())) if scaled else 1.0)
        assert max_abs <= bound, f"{what}: bf16 max abs err {max_abs:.3e} > {bound:.3e}"
        assert rel <= BF16_REL_L2, f"{what}: bf16 rel L2 err {rel:.3e} > {BF16_REL_L2}"
    return max_abs, rel
