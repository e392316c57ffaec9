"""Workload descriptions for the sparse-dense training step.

Five workloads, from a tiny fp32 correctness case up to a 33 GB embedding
configuration, describe one training step of the Lattice Network's
sparse-dense core: the categorical feature processor (embedding tables,
Section 3.3.1), the dense feature processor (bottom MLP), the pairwise
interaction (dot-product Gram, or the factorization-machine block of the
DHEN/Wukong fusion block, Section 3.3.2), the task modules (top MLP with one
logit per objective, Section 3.3.3) and a masked multi-objective loss
(impressions train only their routed heads, Section 3.2.1).

A ``Config`` is pure data: shapes, distributions and seeds.  Nothing here
computes any part of the method.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Optional, Tuple


@dataclass(frozen=True)
class Config:
    name: str
    B: int                       # batch size
    F: int                       # number of sparse (categorical) features
    rows: int                    # rows per embedding table
    d: int                       # embedding dim (uniform across features)
    dtype: str                   # storage dtype: "f32" or "bf16"
    index_dist: Tuple            # ("uniform",) or ("zipf", alpha)
    bag_dist: Tuple              # ("uniform", lo, hi) or ("poisson", mean, lo, hi)
    dense_in: int                # number of dense inputs (0: no dense path)
    bottom: Tuple[int, ...]      # bottom-MLP output widths; last == d
    interact: str                # "dot" | "fm" | "stack"
    top: Tuple[int, ...]         # top-MLP output widths; last == T (with towers: [..., T*towers, T])
    fm_rank: int = 0             # k of the FM block (fm / stack)
    stack_layers: int = 0        # number of FM-stack layers
    stack_n: int = 0             # vectors kept per stack layer
    lcb_n: int = 0               # of those, vectors from the linear compression block (0: FM block only)
    label_p: Tuple = ("fixed", 0.3)          # or ("uniform", lo, hi) per objective
    mask: Tuple = ("none",)                  # ("none",) | ("iid", keep) | ("domain",)
    domains: Optional[Tuple] = None          # (proportions, active features, labelled heads)
    pool: str = "sum"
    lr_tables: float = 0.0                   # row-sparse SGD step on the tables (0: none)
    seed: int = 0
    ln_eps: float = 1e-5
    towers: int = 0                          # per-objective towers: hidden units per tower (0: none);
                                             # the last top layer then reads only its tower's units
    untie: int = 0                           # parameter untying: leading top layers with one
                                             # parameter set per domain (batches then arrive
                                             # grouped by domain)
    top_act: str = "relu"                    # hidden top layers: "relu" | "swishrn" | "hardswishrn"
    norm_block: int = 128                    # SwishRN groups: 128 (BlockNorm) or 0 (the whole row)
    norm_eps: float = 1e-6
    stack_fp8: Optional[str] = None          # STACK: the FM projection in FP8 ("precise" / "fast")

    # ---- derived shapes -------------------------------------------------
    @property
    def has_dense(self) -> bool:
        return self.dense_in > 0

    @property
    def n_slots(self) -> int:
        """Stacked vectors per sample: dense vector (slot 0) then one per feature."""
        return self.F + (1 if self.has_dense else 0)

    @property
    def first_emb_slot(self) -> int:
        return 1 if self.has_dense else 0

    @property
    def T(self) -> int:
        return self.top[-1]

    @property
    def n_pairs(self) -> int:
        n = self.n_slots
        return n * (n - 1) // 2

    @property
    def inter_width(self) -> int:
        if self.interact == "dot":
            return self.n_pairs
        if self.interact == "fm":
            return self.n_slots * self.fm_rank
        if self.interact == "stack":
            return self.stack_n * self.d
        raise ValueError(self.interact)

    @property
    def top_in(self) -> int:
        if self.interact == "stack":
            return self.inter_width
        return (self.d if self.has_dense else 0) + self.inter_width

    @property
    def total_rows(self) -> int:
        return self.F * self.rows

    def scaled(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


SEED_BASE = 2512092000


TINY = Config(
    name="tiny-dot-f32", B=128, F=8, rows=4096, d=32, dtype="f32",
    index_dist=("uniform",), bag_dist=("uniform", 1, 8),
    dense_in=13, bottom=(64, 32), interact="dot", top=(64, 4),
    label_p=("fixed", 0.3), mask=("none",), seed=SEED_BASE + 1)

MID = Config(
    name="mid-dot-bf16", B=2048, F=26, rows=100_000, d=64, dtype="bf16",
    index_dist=("zipf", 1.1), bag_dist=("poisson", 10.0, 1, 64),
    dense_in=13, bottom=(256, 64), interact="dot", top=(512, 256, 8),
    label_p=("uniform", 0.01, 0.3), mask=("iid", 0.5), seed=SEED_BASE + 2)

LARGE_FM = Config(
    name="large-emb-fm", B=8192, F=64, rows=2_000_000, d=128, dtype="bf16",
    index_dist=("zipf", 1.05), bag_dist=("poisson", 20.0, 1, 128),
    dense_in=64, bottom=(512, 128), interact="fm", fm_rank=32,
    top=(1024, 512, 16), label_p=("uniform", 0.01, 0.3), mask=("iid", 0.5),
    lr_tables=0.01, seed=SEED_BASE + 3)

MULTIDOMAIN = Config(
    name="multidomain-dot", B=8192, F=96, rows=1_000_000, d=128, dtype="bf16",
    index_dist=("zipf", 1.1), bag_dist=("poisson", 15.0, 1, 128),
    dense_in=64, bottom=(512, 128), interact="dot", top=(1024, 512, 32),
    label_p=("uniform", 0.01, 0.3), mask=("domain",),
    domains=((0.4, 0.3, 0.2, 0.1), 40, 8), seed=SEED_BASE + 4)

DEEP_STACK = Config(
    name="deep-stack", B=16384, F=256, rows=500_000, d=128, dtype="bf16",
    index_dist=("zipf", 1.05), bag_dist=("poisson", 8.0, 1, 64),
    dense_in=0, bottom=(), interact="stack", fm_rank=64, stack_layers=3,
    stack_n=64, top=(2048, 512, 64), label_p=("uniform", 0.01, 0.3),
    mask=("iid", 0.5), seed=SEED_BASE + 5)

WORKLOADS = {c.name: c for c in (TINY, MID, LARGE_FM, MULTIDOMAIN, DEEP_STACK)}


def small(cfg: Config, B: int, rows: int, **kw) -> Config:
    """Same structure as ``cfg`` with a smaller batch and tables (parity sizes)."""
    return cfg.scaled(B=B, rows=rows, **kw)
