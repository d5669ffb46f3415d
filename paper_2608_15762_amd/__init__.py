"""MI355X-native GMG what-if simulator (SliceScheduler, arXiv 2608.15762).

Importing the package loads nothing: the HIP binding lives in
``paper_2608_15762_amd.ss`` and the seeded input generator in
``paper_2608_15762_amd.synth``.
"""
__version__ = "0.1.0"
