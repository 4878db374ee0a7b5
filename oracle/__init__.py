"""CPU oracle for the OASIS hot path: test infrastructure only (see oasis_oracle)."""
