"""MI355X-native routing + Exact Quantile Balancing statistics for one MoE layer.

The kernels live in libeqb.so (C ABI declared in include/eqb.h); ``eqb`` is its
thin Python binding.
"""
from . import eqb
from .eqb import Layer, run_layer, eqb_rank, qb_loop, rank_averaged_qb, histogram_qb

__all__ = ["eqb", "Layer", "run_layer", "eqb_rank", "qb_loop", "rank_averaged_qb", "histogram_qb"]
