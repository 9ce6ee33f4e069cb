"""CPU oracle for the EQB routing path.  Test infrastructure only: the test
suite, the smoke check and the benchmark's CPU-baseline leg use it; the
product library never does."""
