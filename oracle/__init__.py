"""CPU oracle for RcLLM's selective prefill of one attention layer.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
benchmark's CPU-baseline leg, never by the GPU path.
"""
