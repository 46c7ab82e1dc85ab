"""CPU oracle for the streaming-MoE decode hot path (TEST INFRASTRUCTURE ONLY).

This package is the plain, slow, obviously-correct reference that the HIP
path is checked against.  Only the test-suite, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import it.  The product path
(``paper_2609_18063_amd``) never imports, links or executes anything here,
and this package imports nothing from the product path.

Precision: every floating-point step is carried out in float64 unless the
method stores a value in a narrower type (fp16 weights, scales, zeros and
activations, int4 codes, fp32 router logits).  Where a floating-point value
decides an integer (an int4 code, a top-k index, an fp16 rounding of an
activation), the decision is taken in the precision the kernels use, and the
module that does it says so.

Modules
-------
quant    int4 affine group-64 format: quantize, dequantize, byte sizes.
routing  RMSNorm input, router / prerouter logits, softmax-top-k,
         sigmoid-group routing.
expert   SwiGLU expert with the unmerged LoRA delta, combine, one layer.
slots    slot table and the host-tier slot policy.
stack    40-layer decode chain with prediction-as-routing and the
         residual-mixing stand-in for attention.
batched  multi-token (prefill / batched decode) layer.
"""

from . import quant, routing, expert, slots, stack, batched  # noqa: F401
