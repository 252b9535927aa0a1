"""Entropic-time decode step on MI355X: a HIP library (libent.so) and its binding.

The library computes, per sequence of a decode batch, the exact entropy of
the next-token distribution, entropic time and the temperature law, the
entropy-driven kept set of paged KV blocks, decode attention over the kept
blocks, and the sampled token (arXiv 2603.03310).  `ent` is the ctypes
binding with the C ABI's names; `build` compiles the library in-tree.
"""
from . import ent  # noqa: F401
