"""CPU oracle of the WpAq bipolar-INT GEMM: test infrastructure only."""
