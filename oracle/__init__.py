"""fp64 CPU oracle (test infrastructure only; see segpa_oracle)."""
