"""MI355X-native gradient dropping (Aji & Heafield, EMNLP 2017).

``gd`` binds the HIP library (``libgd.so``, C ABI declared in
``include/gd.h``); ``workloads`` draws the seeded synthetic gradients.
Importing the package does not load the library; the first call does, and
fails loudly if it has not been built.
"""
__all__ = ["gd", "workloads"]
