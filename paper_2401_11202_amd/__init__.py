"""MI355X-native execution of PartIR:Core loops (#tile / #sum) on one GPU.

``paper_2401_11202_amd.partir`` is the Python binding of the HIP library
``libpartir.so`` (C ABI in ``include/partir.h``); ``inputs`` and
``workloads`` describe seeded synthetic workloads.
"""
__all__ = ["partir", "inputs", "workloads"]
