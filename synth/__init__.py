"""Seeded synthetic inputs shared by the oracle tests and the GPU path (random draws only)."""
from .gmm import (WORKLOADS, WORKLOAD_ORDER, Workload, cluster_sizes, gaussian_mixture,
                  make_workload, standard_normal_factor)

__all__ = ["WORKLOADS", "WORKLOAD_ORDER", "Workload", "cluster_sizes", "gaussian_mixture",
           "make_workload", "standard_normal_factor"]
