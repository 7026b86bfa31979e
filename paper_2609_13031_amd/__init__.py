"""MI355X-native FP8 in-context-learning attention for tabular foundation models.

The compute path is the HIP library ``libtfm.so`` built from ``csrc/`` (see
``include/tfm.h`` for the C ABI); ``tfm`` is its thin Python binding and
``workloads`` draws seeded synthetic inputs.  Importing the package loads
nothing; ``tfm.lib()`` loads the library and raises if it has not been built.
"""
