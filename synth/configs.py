"""The five recommendation-shaped workloads, as data.

Each names the size of one PS shard's step: K gradient contributions per
global batch (the gradient-buffer capacity, written M in the paper's Sec. 3.1),
local batch B with L embedding IDs per sample drawn from a Zipf law over R
table rows of width D, P dense parameters, the staleness law of the
contributions, the tolerance threshold iota of Eq. 1 and the optimiser.

Where a workload leaves a hyper-parameter open the value used here is marked
``assumed`` and follows the paper's Table 1 (Criteo uses iota = 3, the other
two tasks iota = 4; Adam learning rates there range from 6e-4 to 1.5e-3).
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace

SEED_BASE = 2205110480      # seed of workload c is SEED_BASE + c
STEP = 1000                 # global step k of the update being applied


@dataclass(frozen=True)
class Workload:
    name: str
    K: int                  # contributions per global batch
    B: int                  # local batch size (samples per contribution)
    L: int                  # IDs per sample (multi-hot) or number of one-hot fields
    one_hot_fields: bool    # True: L fields of floor(R/L) rows, one ID per field
    zipf_s: float
    R: int                  # embedding rows on this shard
    D: int                  # embedding width
    P: int                  # dense parameters on this shard
    grad_sigma: float       # standard deviation of the synthetic gradients
    staleness: tuple        # ("uniform", hi) -> {0..hi}; ("geometric", p) -> P(s) = p (1-p)^s
    iota: int               # tolerance threshold of Eq. 1
    optimizer: str          # "adagrad" | "adam"
    lr: float
    eps: float = 1e-8
    beta1: float = 0.9
    beta2: float = 0.999
    notes: tuple = field(default_factory=tuple)

    @property
    def n_per_contribution(self) -> int:
        return self.B * self.L

    @property
    def N(self) -> int:
        return self.K * self.n_per_contribution

    @property
    def adam_t(self) -> int:
        return STEP + 1

    def scaled(self, **kw) -> "Workload":
        return replace(self, **kw)


CONFIGS = [
    Workload("c0", K=4, B=256, L=20, one_hot_fields=False, zipf_s=1.1, R=100_000, D=16,
             P=65_536, grad_sigma=1e-2, staleness=("uniform", 3), iota=2,
             optimizer="adagrad", lr=0.01, eps=1e-8),
    Workload("c1", K=32, B=1024, L=26, one_hot_fields=True, zipf_s=1.05, R=10_000_000, D=64,
             P=2_000_000, grad_sigma=1e-2, staleness=("geometric", 0.5), iota=3,
             optimizer="adagrad", lr=0.01, eps=1e-8,
             notes=("iota assumed (Criteo-like, Table 1)", "lr, eps, sigma assumed")),
    Workload("c2", K=100, B=512, L=200, one_hot_fields=False, zipf_s=1.2, R=100_000_000, D=16,
             P=8_000_000, grad_sigma=1e-2, staleness=("geometric", 0.4), iota=4,
             optimizer="adam", lr=1e-3, eps=1e-8,
             notes=("lr, eps, sigma assumed",)),
    Workload("c3", K=64, B=2048, L=50, one_hot_fields=False, zipf_s=1.05, R=20_000_000, D=32,
             P=200_000_000, grad_sigma=1e-3, staleness=("uniform", 5), iota=4,
             optimizer="adam", lr=1e-3, eps=1e-8,
             notes=("iota assumed (Table 1, Alimama/Private)", "lr, eps assumed")),
    Workload("c4", K=256, B=256, L=1000, one_hot_fields=False, zipf_s=1.1, R=500_000_000, D=32,
             P=16_000_000, grad_sigma=1e-2, staleness=("geometric", 0.3), iota=8,
             optimizer="adagrad", lr=0.01, eps=1e-8,
             notes=("lr, eps, sigma assumed (as c0)",)),
]

BY_NAME = {c.name: c for c in CONFIGS}


def seed_of(name: str) -> int:
    return SEED_BASE + int(name.lstrip("c").split("_")[0])
