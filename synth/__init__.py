"""Seeded synthetic inputs for the text-encoder prefill workloads.

This package is shared by the oracle and by the HIP path. It holds no part of
the encoder's arithmetic: it only draws weights, embeddings and sequence
layouts from fixed seeds, rounded to the storage type of the workload.
"""
from .workloads import (  # noqa: F401
    Dims, Workload, SeqLayout, DIMS_TINY, DIMS_FULL, WORKLOADS, workload,
    layer_weights, final_norm_gain, embeddings, seq_lens, round_to_bf16,
    mixed_layouts, grid_for_length,
)
