"""The five workload shapes of the PSS hashed-embedding layer.

Each workload is a DLRM-style batch of T categorical features ("tables"),
B samples, one bag of token indices per (table, sample), embedding width d,
chunk size Z and a flat shared array of M weights.  Shapes follow the
criteo-tb setting of the paper's experiments (26 categorical features,
d = 128, at most 40M rows per table; the 10 MB compressed embedding of the
10^4x point); the datasets themselves are not used: every value is drawn
from a seeded generator.
"""
from __future__ import annotations

from dataclasses import dataclass, replace


@dataclass(frozen=True)
class Workload:
    key: str            # short id, c1 .. c5
    name: str           # what the workload is
    T: int              # tables (categorical features)
    B: int              # samples per batch
    d: int              # embedding width
    Z: int              # chunk size (consecutive weights per hashed chunk)
    M: int              # weights in the shared array
    weight_dtype: str   # "f32" or "bf16" storage of the shared array
    cardinality: str    # "fixed:<n>" or "loguniform:<lo>:<hi>"
    bag: str            # "one" or "poisson:<mean>:<lo>:<hi>"
    index_dist: str     # "uniform" or "zipf:<s>"
    optimizer: str      # "sgd" or "adagrad"
    lr: float
    eps: float          # Adagrad epsilon
    hash_seed: int      # seed of the universal hash parameters (a, b)
    data_seed: int      # seed of every drawn input

    @property
    def C(self) -> int:
        return self.d // self.Z

    def scaled(self, **kw) -> "Workload":
        """Same workload with some sizes overridden (e.g. B, M for tests)."""
        return replace(self, **kw)


CONFIGS = {
    "c1": Workload("c1", "tiny-4x1000-d16-z4", T=4, B=256, d=16, Z=4, M=4096,
                   weight_dtype="f32", cardinality="fixed:1000", bag="one",
                   index_dist="uniform", optimizer="sgd", lr=0.1, eps=1e-10,
                   hash_seed=1, data_seed=1001),
    "c2": Workload("c2", "criteo-tb-1hot-26t-d128-z32-10MB", T=26, B=65536, d=128, Z=32,
                   M=2_500_000, weight_dtype="f32", cardinality="loguniform:3:40000000",
                   bag="one", index_dist="zipf:1.1", optimizer="sgd", lr=0.1, eps=1e-10,
                   hash_seed=2, data_seed=1002),
    "c3": Workload("c3", "multihot-26t-pois20-d64-z16-64MB-adagrad", T=26, B=32768, d=64, Z=16,
                   M=16_000_000, weight_dtype="f32", cardinality="fixed:10000000",
                   bag="poisson:20:1:64", index_dist="zipf:1.05", optimizer="adagrad",
                   lr=0.01, eps=1e-10, hash_seed=3, data_seed=1003),
    "c4": Workload("c4", "hbm-hashing-trick-26t-d128-z1-4GB", T=26, B=65536, d=128, Z=1,
                   M=1_000_000_000, weight_dtype="f32", cardinality="fixed:40000000",
                   bag="one", index_dist="uniform", optimizer="sgd", lr=0.1, eps=1e-10,
                   hash_seed=4, data_seed=1004),
    "c5": Workload("c5", "rowhash-bf16-26t-d128-z128-adagrad", T=26, B=262144, d=128, Z=128,
                   M=64_000_000, weight_dtype="bf16", cardinality="fixed:40000000",
                   bag="one", index_dist="zipf:1.2", optimizer="adagrad", lr=0.01,
                   eps=1e-10, hash_seed=5, data_seed=1005),
}


def get(key: str) -> Workload:
    return CONFIGS[key]
