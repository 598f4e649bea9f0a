"""MI355X-native subspace-network (SSN) stage-boundary codec.

The compute lives in a HIP/C-ABI shared library (``libssn.so``, declared in
``include/ssn.h``); ``paper_2607_13332_amd.ssn`` is a thin ctypes binding over
it that marshals torch device tensors and the current HIP stream.
``paper_2607_13332_amd.inputs`` holds the seeded synthetic input generators.
"""
__all__ = ["inputs", "ssn"]
