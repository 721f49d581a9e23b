"""PISA (pyramid Top-K block selection + block-sparse attention) for MI355X.

The compute path is the HIP library ``libpisa.so`` built from ``csrc/``; the
Python module :mod:`paper_2609_31093_amd.pisa` is a thin ctypes binding with
the same entry-point names as the C ABI in ``include/pisa.h``.
"""
