"""CPU oracle (test infrastructure only): plain definitions the GPU path is checked against."""
