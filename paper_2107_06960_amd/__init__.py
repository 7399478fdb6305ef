"""MI355X-native fused tile partitioning (MAFAT, arXiv 2107.06960).

The compute path is the HIP library ``libmafat.so`` (built from ``csrc/``);
``mafat`` is its thin ctypes binding.  Importing this package loads nothing;
import ``paper_2107_06960_amd.mafat`` to use the library.
"""
