"""CPU oracle for the AVTP pruning-layer operator (test infrastructure only).

Imported only by the tests, the smoke check and the CPU-baseline leg of the
benchmark; never by the library or its binding.
"""
