"""Seeded synthetic inputs for log-linear attention, shared by the tests, the smoke check
and the benchmark.  This module holds no arithmetic of the method itself: it draws
standard normals in a fixed order, applies the input transforms of each workload
(scaling, softplus, sigmoid, L2-normalisation of keys) and rounds to the storage dtype.
Both the float64 oracle and the GPU library receive exactly the arrays returned here.
"""

from .gen import (WORKLOADS, Workload, generate, level_weight_matrices, shared_qk, to_storage,  # noqa: F401
                  upstream_grad)
