"""Seeded synthetic workloads shared by the tests, the oracle checks and the benchmark.

This package only draws random numbers and encodes them as bfloat16; it holds no
step of the retrieval method itself.
"""
from .gen import (CONFIGS, Config, StreamSpec, bf16_bits, planted_frames, make_queries,
                  frame_block_keys, make_stream, stream_specs)

__all__ = ["CONFIGS", "Config", "StreamSpec", "bf16_bits", "planted_frames", "make_queries",
           "frame_block_keys", "make_stream", "stream_specs"]
