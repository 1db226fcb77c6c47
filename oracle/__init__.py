"""CPU oracle for the UFP4 hot path. Test infrastructure only: used by the tests, the smoke check and
the CPU-baseline leg of the benchmark, never by the product path."""
