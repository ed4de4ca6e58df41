"""Measurement tooling beside the library: the write-ceiling probe
(ceilings.hip, built by build()) and digests of rocprofv3 output."""
