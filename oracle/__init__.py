"""fp64 CPU oracle for EG-MLA (test infrastructure only; see eg_mla_oracle)."""
