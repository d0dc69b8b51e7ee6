"""CPU oracle of the HiLo-Token compressed DiT block -- test infrastructure only (see hilo_oracle)."""
