"""fp64 CPU oracle of the WeDLM decode step.  Test infrastructure only: the
tests, the package smoke check and the benchmark's CPU-baseline leg use it;
the HIP library never does."""
