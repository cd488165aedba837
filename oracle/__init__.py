"""CPU oracle of ProxyAttn's prefill path.  Test infrastructure only: used by
the tests, the package smoke check and the benchmark's CPU-baseline leg."""
