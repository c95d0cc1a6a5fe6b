"""CPU oracle of the KV-cache splice (test infrastructure only; see splice_oracle)."""
