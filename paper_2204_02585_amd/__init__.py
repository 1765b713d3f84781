"""MI355X-native cached renderer for SqueezeNeRF (factorized FastNeRF).

The renderer itself is the C-ABI library ``libsqn.so`` built from ``csrc/``
(hand-written HIP for gfx950); ``binding`` marshals torch device tensors to
it and ``scenes`` makes seeded synthetic inputs.  Importing the package does
not load the library; ``binding`` does, and raises if it is missing.
"""
__version__ = "0.1.0"
