"""MI355X-native interface-adjoint scan of LBI (latent bounded interfaces).

The compute path lives in the HIP library ``_lib/liblbi.so`` (C-ABI declared
in ``include/lbi.h``); ``paper_2605_09204_amd.binding`` marshals torch tensors
into it.  The library is loaded on first use and a missing build raises an
error: there is no CPU fallback.  ``paper_2605_09204_amd.synth`` draws seeded
synthetic operands.
"""
