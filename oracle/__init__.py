"""CPU oracle (test infrastructure only; see decoder_stage)."""
