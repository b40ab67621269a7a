"""Seeded synthetic inputs for the PSS hashed-embedding layer.

Shared by the tests, the benchmark and the CPU oracle checks.  Holds none of
the layer's arithmetic (no hashing, gathering, pooling or updates): it only
draws table cardinalities, bag lengths, token indices, initial weights and
upstream gradients with the shapes of DLRM/criteo-tb style workloads.  The
hash seed of a workload is carried as a plain integer; each side derives
(a, b) from it with its own SplitMix64.
"""
from .configs import CONFIGS, Workload, get  # noqa: F401
from .gen import make_inputs, make_grad, make_weights, Inputs  # noqa: F401
