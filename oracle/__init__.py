"""fp64 CPU oracle of the batched kernel-latency model.

Test infrastructure: only the tests, the smoke check and the CPU-baseline leg
of the benchmark may import it.  It shares no code with the HIP library."""
