"""HIGGS quantized linear layers on MI355X (gfx950).

``higgs`` binds the C ABI of libhiggs.so (see include/higgs.h); ``synth`` draws
the seeded synthetic weights and activations used by the tests and benchmark.
"""
__all__ = ["higgs", "synth"]
