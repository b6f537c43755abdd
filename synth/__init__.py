"""Seeded synthetic inputs shared by the oracle tests and the GPU path (random draws only)."""
from .gmm import (TABLE2, WORKLOADS, WORKLOAD_ORDER, Workload, cluster_sizes, cnr_bar, gaussian_mixture,
                  make_workload, standard_normal_factor)

__all__ = ["TABLE2", "WORKLOADS", "WORKLOAD_ORDER", "Workload", "cluster_sizes", "cnr_bar",
           "gaussian_mixture", "make_workload", "standard_normal_factor"]
