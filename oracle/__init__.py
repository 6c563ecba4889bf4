"""CPU oracle (test infrastructure only; see cosa_oracle module docstring)."""
