"""MI355X-native paged GQA prefill/decode attention on split compute units.

The HIP library is loaded lazily by :mod:`paper_2504_14489_amd.mw`; importing
the package itself touches no GPU and loads no native code.
"""
__all__ = ["workloads", "accounting", "mw"]
