"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle.

Holds none of the quantiser's arithmetic: only corpus / query / tenant /
allowlist generation.  See synth.workloads for the recipes.
"""
from .workloads import (CHUNK, isotropic_mixture, isotropic_queries, shifted_mixture,
                        powerlaw_mixture_rows, workload, zipf_tenants,
                        allowlists, allowlist_bitmap, uniform_partition_tenants)

__all__ = ["CHUNK", "isotropic_mixture", "isotropic_queries", "shifted_mixture",
           "powerlaw_mixture_rows", "workload", "zipf_tenants", "allowlists",
           "allowlist_bitmap", "uniform_partition_tenants"]
