"""VaSE-AttnV eviction round for AMD Instinct MI355X (gfx950).

``vase`` is the binding of the HIP library ``libvase.so`` (built in-tree by
``paper_2606_03928_amd.build``); ``synth`` draws the synthetic Qwen3-shaped
caches.  The library is loaded on first use, so importing the package does not
need a GPU.
"""
from . import synth, vase  # noqa: F401

__all__ = ["synth", "vase"]
