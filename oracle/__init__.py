"""CPU oracle for the W4A4G4 triple-branch linear layer.

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the
benchmark's CPU-baseline leg, never by the GPU library or its binding.
"""
