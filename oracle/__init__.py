"""Oracle package: test infrastructure (plain CPU code written from the paper).
Only tests, the smoke check and the benchmark's CPU-baseline leg import it."""
