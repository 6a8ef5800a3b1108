"""MI355X-native QCFuse fusion step: HIP kernels for gfx950 behind a C ABI.

Importing the package loads nothing native; ``paper_2606_05875_amd.qcf``
loads ``libqcf.so`` and fails loudly if it has not been built.
"""
__version__ = "0.1.0"
