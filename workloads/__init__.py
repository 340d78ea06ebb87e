"""Seeded synthetic workloads for the AR-DiT chunk-denoise block.

This package draws inputs only: shapes, seeds, normal draws and the
fp32 -> bf16 rounding both sides consume. It contains none of the block's
arithmetic, so the oracle and the HIP path can both use it without sharing
any of the computation they are compared on.
"""
from .gen import (  # noqa: F401
    BlockShape, Workload, WORKLOADS, workload, make_rng,
    bf16_bits, bits_to_f32, bf16_round, normal_bf16,
    draw_time_weights, draw_block_weights, BLOCK_WEIGHT_ORDER,
    TIME_WEIGHT_ORDER, draw_ragged_streams, ring_page_ids, stream_page_ids,
)
