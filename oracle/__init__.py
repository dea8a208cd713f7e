"""CPU oracle for the DynaSpec dynamic draft head.  Test infrastructure only:
imported by the tests, the smoke check and the benchmark's CPU-baseline leg,
never by the library."""
