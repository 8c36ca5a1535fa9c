"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke check.

This package holds no collective arithmetic: it draws random numbers, builds count and
displacement tables, and returns host arrays. Both the GPU library's callers and the CPU
oracle's callers take their inputs from here, so neither side depends on the other.
"""
from .generators import (  # noqa: F401
    alltoallv_layout,
    bf16_bits_from_f32,
    device_normal_bf16,
    device_uniform_f32,
    normal_bf16,
    normal_f32,
    row_ids_int32,
    uniform_f32,
    zipf_counts,
    small_int_valued,
)
