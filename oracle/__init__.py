"""fp64 CPU oracle for the HERMES streaming step (test infrastructure only)."""
