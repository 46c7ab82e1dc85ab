"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This package only draws random data in the storage formats the hot path
consumes (packed int4 codes, fp16 scales / zeros / LoRA factors / router
weights, fp32 token draws).  It contains none of the method's arithmetic:
no dequantization, routing, expert or combine math.
"""

from .gen import *  # noqa: F401,F403
