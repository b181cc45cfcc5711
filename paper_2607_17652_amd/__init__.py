"""MI355X-native (gfx950) packed wavefront denoising step of FlowBlock.

The compute path is the C-ABI library ``libflowblock.so`` built from
``csrc/`` (hand-written HIP kernels); ``binding`` is a thin ctypes layer over
it, and ``synth`` draws seeded synthetic workloads.  Importing the package
loads nothing: the library is opened on first use of ``binding``.
"""
__version__ = "0.1.0"
