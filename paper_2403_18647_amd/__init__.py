"""SDSAT two-step-draft-then-verify block decoding on MI355X (gfx950).

The compute path is the HIP library ``libsdsat.so`` (C-ABI declared in
``include/sdsat.h``); ``binding`` marshals arguments to it through ctypes
with PyTorch device tensors as the memory and stream provider.  ``synth``
makes seeded synthetic inputs.
"""
