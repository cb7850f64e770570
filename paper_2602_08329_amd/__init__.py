"""MI355X-native decode hot path of Pre-hoc Sparsity (PrHS).

The compute path is the C-ABI library ``libprhs.so`` (HIP kernels for gfx950);
``paper_2602_08329_amd.binding`` marshals torch tensors into it.  Importing
this package does not load the library; ``binding.lib()`` does, and fails
loudly when it has not been built.
"""

__all__ = ["binding", "synth", "schedule"]
