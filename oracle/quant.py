"""Oracle: the int4 affine group-64 weight format (TEST INFRASTRUCTURE ONLY).

The paper stores every expert projection as int4 codes plus one scale and one
bias ("zero") per group of 64 weights ("int4 affine group-64", §2
Quantization; Tab. 1 "Quantization"; §3.1 Executor paths, the nine stacked
tensors: gate, up and down, each with its scales and biases).  A weight is
reconstructed as ``w_hat = s * q + z`` with ``q`` in ``[0, 15]``.

Readings (the paper is silent on these):

* Groups run along the input (reduction) dimension of each row.
* Packed storage: two codes per byte, the even input index in the low
  nibble.
* Scale and zero are stored as fp16.
* Quantizer: ``lo = min``, ``hi = max`` of the group in fp32;
  ``s = fp16((hi - lo) / 15)`` and ``z = fp16(lo)``, both round-to-nearest-
  even; ``q = clamp(rint((w - z) / s), 0, 15)`` evaluated in fp32 with the
  fp16 ``s`` and ``z`` (half-to-even), and ``q = 0`` when ``s == 0``.
  The code is an integer decided by floating point, so it is decided in
  fp32, the precision the GPU quantizer uses.
* Dequantization is exact here: it is done in float64, where ``s * q + z``
  of fp16 ``s``, ``z`` and a 4-bit ``q`` is exact.

The byte counts follow from the format: 4 bits per weight plus 4 bytes of
(scale, zero) per 64 weights, i.e. 0.5625 B per weight.  §3.1 (Problem)
prints the resulting sizes for the 35B tier: 1.77 MB per expert, 453 MB per
layer of 256 experts, 16.9 GiB over 40 layers.
"""

import numpy as np

GROUP = 64


def quantize_g64(w):
    """Quantize fp32 weights ``w [rows, cols]`` to (q uint8, s fp16, z fp16).

    ``q`` has one code per weight (values 0..15, unpacked), ``s`` and ``z``
    have shape ``[rows, cols // 64]``.  Follows the quantizer reading in the
    module docstring.
    """
    w = np.asarray(w, dtype=np.float32)
    rows, cols = w.shape
    if cols % GROUP:
        raise ValueError("cols must be a multiple of 64")
    g = w.reshape(rows, cols // GROUP, GROUP)
    lo = g.min(axis=-1)
    hi = g.max(axis=-1)
    # fp32 subtract, fp32 divide, then round to fp16 (round-to-nearest-even).
    s = ((hi - lo) / np.float32(15.0)).astype(np.float16)
    z = lo.astype(np.float16)
    s32 = s.astype(np.float32)[..., None]
    z32 = z.astype(np.float32)[..., None]
    with np.errstate(divide="ignore", invalid="ignore"):
        t = (g - z32) / s32                     # fp32
    q = np.clip(np.rint(t), 0, 15)              # rint = round half to even
    q = np.where(s32 == 0, 0, q)
    return q.astype(np.uint8).reshape(rows, cols), s, z


def unpack_nibbles(packed):
    """Codes from the packed storage: byte ``j`` of a row holds the codes of
    inputs ``2j`` (low nibble) and ``2j + 1`` (high nibble)."""
    packed = np.asarray(packed, dtype=np.uint8)
    rows, half = packed.shape
    q = np.empty((rows, 2 * half), dtype=np.uint8)
    q[:, 0::2] = packed & 0x0F
    q[:, 1::2] = packed >> 4
    return q


def pack_nibbles(q):
    """Inverse of :func:`unpack_nibbles` for codes ``q [rows, cols]`` in 0..15."""
    q = np.asarray(q, dtype=np.uint8)
    return (q[:, 0::2] | (q[:, 1::2] << 4)).astype(np.uint8)


def dequantize_g64(q, s, z):
    """Reconstruct ``w_hat = s * q + z`` (float64, exact) for every weight."""
    q = np.asarray(q, dtype=np.float64)
    rows, cols = q.shape
    s64 = np.asarray(s, dtype=np.float64)
    z64 = np.asarray(z, dtype=np.float64)
    assert s64.shape == (rows, cols // GROUP) and z64.shape == s64.shape
    # group g of a row holds inputs 64 g .. 64 g + 63
    w = s64[:, :, None] * q.reshape(rows, cols // GROUP, GROUP) + z64[:, :, None]
    return w.reshape(rows, cols)


def projection_bytes(out_dim, in_dim):
    """Stored bytes of one int4 g64 projection: codes + (fp16 s, fp16 z)."""
    return out_dim * in_dim // 2 + out_dim * (in_dim // GROUP) * 4


def expert_bytes(d, inter):
    """Stored bytes of one SwiGLU expert: gate [I x d], up [I x d], down [d x I]."""
    return 2 * projection_bytes(inter, d) + projection_bytes(d, inter)


def lora_bytes(d, inter, rank, projections=3):
    """fp16 LoRA factors A [r x in] and B [out x r] on gate, up and down."""
    per = {
        "gate": rank * d + inter * rank,
        "up": rank * d + inter * rank,
        "down": rank * inter + d * rank,
    }
    names = ["gate", "up", "down"][:projections]
    return 2 * sum(per[n] for n in names)
