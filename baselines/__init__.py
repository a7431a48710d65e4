"""Host-side comparison baselines of the benchmark (not part of the library, not the oracle)."""
