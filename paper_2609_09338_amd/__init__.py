"""Osprey speculative draft-and-verify step on AMD MI355X (gfx950).

`binding` exposes the C ABI of libosprey (include/osprey.h) to Python;
`workload` drives it on the seeded synthetic workloads.  The library must be
built (`python -m paper_2609_09338_amd.build`); nothing here falls back to a
CPU implementation.
"""
from ._lib import LIB_PATH  # noqa: F401
