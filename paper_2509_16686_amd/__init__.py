"""EG-MLA decode for MI355X (gfx950): a C-ABI HIP library and its thin Python binding.

Submodules:
  binding    -- ctypes binding of libegmla.so (append, decode, prefill_ref)
  workloads  -- seeded synthetic inputs (no method arithmetic)
  accounting -- algorithmic bytes / flops of a decode call
  build      -- compiles the HIP library for gfx950
"""
__all__ = ["binding", "workloads", "accounting", "build"]
