"""Plain CPU oracle for batched TFHE PBS (test infrastructure only)."""
