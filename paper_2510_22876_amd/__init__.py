"""Greedy verify + KV realign for batch speculative decoding (EqSpec,
arXiv 2510.22876) on AMD MI355X.

The compute path is the HIP library ``libspecdec.so`` (C ABI declared in
``include/specdec.h``); ``paper_2510_22876_amd.specdec`` is its ctypes
binding.  Importing this package loads nothing native.
"""
