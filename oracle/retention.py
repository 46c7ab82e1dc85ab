"""Oracle: merging the LoRA delta and re-quantizing, the rejected alternative (TEST INFRASTRUCTURE ONLY).

§3.3 (Recovery LoRA) keeps the adapter unmerged, ``y = W_int4 v + (alpha/r)
B (A v)``.  The alternative it rejects folds the delta into the dequantized
weight and quantizes the sum back to int4 g64.  Because a delta of RMS about
1e-3 is smaller than the group step, the re-quantization puts most weights
back on their old codes and the delta is largely lost.  The paper gives two
measures of what survives (§3.3, footnote on retention):

* weight level, per target: ``sum(actual * delta) / sum(delta^2)`` with
  ``delta = (alpha/r) B A`` and ``actual = requant(W + delta) - W``;
* output level: ``1 - ||U - M|| / ||U - B||`` for the outputs of the
  unmerged (U), merged (M) and base (B) models on the same inputs.

Readings (the paper is silent on these):

* ``W`` is the dequantized int4 weight ``s q + z``.  The merged weight
  ``W + delta`` is formed in float64 and rounded once to fp32, the
  quantizer's input precision, and re-quantized with the same g64
  quantizer as the base (:func:`oracle.quant.quantize_g64`: min/max per
  group, fp16 scale and zero).
* Output level is taken at the expert (and layer) output, the last point
  of the path built here; the paper measures it at the model's logits.
* Both measures are over all weights of a target (all outputs of all
  tokens) at once, not averaged per row or per token.

Arithmetic is float64 apart from the fp32 rounding of the merged weight.
"""

import numpy as np

from .quant import quantize_g64, dequantize_g64, unpack_nibbles, pack_nibbles
from .expert import expert_forward


def lora_delta(lora, lora_scale):
    """``delta = (alpha / r) B A`` in float64, ``[out, in]``."""
    a, b = lora
    return lora_scale * (np.asarray(b, dtype=np.float64) @ np.asarray(a, dtype=np.float64))


def requantize_with(qsz, delta):
    """Add ``delta [out, in]`` (float64) to the dequantized projection and
    re-quantize.  Returns ``(qsz_merged, actual)`` with
    ``actual = dequant(qsz_merged) - dequant(qsz)`` (float64)."""
    qp, s, z = qsz
    w = dequantize_g64(unpack_nibbles(qp), s, z)
    merged = (w + np.asarray(delta, dtype=np.float64)).astype(np.float32)
    q2, s2, z2 = quantize_g64(merged)
    actual = dequantize_g64(q2, s2, z2) - w
    return (pack_nibbles(q2), s2, z2), actual


def merge_requantize(qsz, lora, lora_scale):
    """Fold the adapter ``lora = (A, B)`` into one int4 g64 projection.

    Returns ``(qsz_merged, delta, actual)``: the merged projection in the
    storage format of ``qsz`` (packed codes, fp16 scale and zero), the
    intended change ``delta`` and the change that survives (float64).
    """
    delta = lora_delta(lora, lora_scale)
    merged, actual = requantize_with(qsz, delta)
    return merged, delta, actual


def weight_retention(actual, delta):
    """``sum(actual * delta) / sum(delta^2)``: the fraction of the intended
    weight change that survives, projected on the intended direction."""
    actual = np.asarray(actual, dtype=np.float64)
    delta = np.asarray(delta, dtype=np.float64)
    den = float(np.sum(delta * delta))
    if den == 0.0:
        raise ValueError("retention is undefined for a zero delta")
    return float(np.sum(actual * delta)) / den


def output_retention(u, m, b):
    """``1 - ||U - M|| / ||U - B||`` over all entries of the three outputs."""
    u = np.asarray(u, dtype=np.float64)
    m = np.asarray(m, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = float(np.linalg.norm(u - b))
    if den == 0.0:
        raise ValueError("retention is undefined when the adapter changes nothing")
    return 1.0 - float(np.linalg.norm(u - m)) / den


def merged_bundle(bundle, lora_scale):
    """The expert with every adapter merged and re-quantized (no adapters
    left), plus per-projection ``(delta, actual)`` for the weight measure."""
    out = {"lora": {"gate": None, "up": None, "down": None}}
    parts = {}
    lo = bundle.get("lora") or {}
    for p in ("gate", "up", "down"):
        if lo.get(p) is None:
            out[p] = bundle[p]
            continue
        out[p], delta, actual = merge_requantize(bundle[p], lo[p], lora_scale)
        parts[p] = (delta, actual)
    return out, parts


def base_bundle(bundle):
    """The expert with its adapters removed (the base model B)."""
    return {"gate": bundle["gate"], "up": bundle["up"], "down": bundle["down"],
            "lora": {"gate": None, "up": None, "down": None}}


def expert_retention(bundle, x16_rows, lora_scale):
    """Both measures for one adapted expert on tokens ``x16_rows [T, d]``.

    Returns a dict with the weight-level retention of every adapted
    projection, the output-level retention over the T expert outputs and the
    three output sets ``U``, ``M``, ``B`` (float64 ``[T, d]``).
    """
    merged, parts = merged_bundle(bundle, lora_scale)
    base = base_bundle(bundle)
    rows = np.asarray(x16_rows, dtype=np.float16)
    u = np.stack([expert_forward(bundle, x, lora_scale)[0] for x in rows])
    m = np.stack([expert_forward(merged, x, lora_scale)[0] for x in rows])
    b = np.stack([expert_forward(base, x, lora_scale)[0] for x in rows])
    return {
        "weight": {p: weight_retention(act, dl) for p, (dl, act) in parts.items()},
        "output": output_retention(u, m, b),
        "U": u, "M": m, "B": b, "merged": merged,
    }
