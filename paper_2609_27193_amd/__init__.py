"""MI355X-native LayerCheck decision-step library (score, select, pack, restore).

The compute path is the HIP shared library built from ``csrc/``; the Python
module :mod:`paper_2609_27193_amd.layercheck` is a thin ctypes binding over its
C interface.  Importing this package loads nothing: the library is opened on
first use and a missing build raises immediately.
"""
