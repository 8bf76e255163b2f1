"""CPU reference decoder: test infrastructure only (tests, smoke check, CPU-baseline leg)."""
