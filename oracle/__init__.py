"""fp64 CPU oracle for the convolution passes (test infrastructure only)."""
