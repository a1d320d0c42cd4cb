"""MI355X-native DeepReduce sparse-gradient codec (arXiv 2102.03112).

The codec itself is the C-ABI library ``libdeepreduce.so`` built from the HIP
sources in ``csrc/`` for gfx950; ``binding`` wraps its entry points for
Python callers that hold torch device tensors.  Importing this package does
not load the library; ``binding.lib()`` does, and raises if it is missing.
"""
