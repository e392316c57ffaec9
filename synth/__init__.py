"""Seeded synthetic workloads (inputs only; none of the method's arithmetic)."""
from .configs import Config, WORKLOADS, TINY, MID, LARGE_FM, MULTIDOMAIN, DEEP_STACK, SEED_BASE, small  # noqa: F401
from .gen import (make_batch, make_dense_params, make_tables, randn, zipf_cdf,  # noqa: F401
                  zipf_ranks, rank_permutation, domain_counts, to_storage, torch_dtype,
                  sub_batch)
