"""WISE hot path on MI355X (gfx950): dense attention with block-mass pooling,
support selection to CSR, and block-sparse attention, behind the C ABI in
include/wise.h.

The compiled library is loaded lazily by `paper_2609_27373_amd.wise`; importing
this package alone touches no GPU and needs no built library.
"""

__all__ = ["workloads", "wise"]
