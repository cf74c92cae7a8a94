"""fp64 CPU oracle for the LazyAttention hot path (test infrastructure only; see lazy_oracle)."""
