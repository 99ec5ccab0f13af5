"""MI355X (gfx950) simulator of the memory-constrained LLM-inference schedulers
A_max, A_min and H-SF of arXiv 2508.14544.

The simulation runs in hand-written HIP kernels behind the C ABI declared in
``include/schedsim.h`` (``libschedsim.so``); ``binding`` is its ctypes front
end and ``workloads`` draws seeded synthetic instances.  Importing the package
does not load the library; ``binding.load_library()`` does, and raises if it
has not been built.
"""
__all__ = ["binding", "workloads", "build"]
__version__ = "0.1.0"
