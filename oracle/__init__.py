"""CPU oracle for the FOCUS scale-learning step -- TEST INFRASTRUCTURE ONLY.

Used by the tests, the smoke check and the benchmark's CPU-baseline leg; never by the HIP library
or its binding, with which it shares no code.
"""
