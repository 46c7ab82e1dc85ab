"""Oracle: SwiGLU experts, unmerged LoRA delta, combine, one MoE layer (TEST INFRASTRUCTURE ONLY).

Expert (§3.1, Math contract): ``y = down(silu(gate(x)) * up(x))`` where each
projection is an int4 g64 matrix dequantized as ``s * q + z``.

LoRA (§3.3 and Fig. 1): every adapted projection adds the unmerged parallel
delta ``(alpha / r) * B (A v)`` to ``W_int4 v``; the int4 bytes are never
touched.  The paper uses ``r = 16, alpha = 32`` (Tab. 1, "LoRA").

Combine (§2, MoE routing; Fig. 1 sum node): the layer output is the routing-
weighted sum of the selected experts' outputs plus the always-on shared
expert(s).

Readings (the paper is silent or the configurations differ):

* ``silu(z) = z / (1 + exp(-z))``.
* The shared expert enters the sum with weight 1.0 and no gate.
* LoRA factors are stored fp16, ``A`` as ``[r, in]`` and ``B`` as
  ``[out, r]``; a projection with no adapter has ``None``.  Each expert
  (routed or shared) may carry its own adapter.
* All arithmetic is float64.

A *bundle* is a dict ``{"gate": (q, s, z), "up": (q, s, z), "down": (q, s, z),
"lora": {"gate": (A, B) | None, "up": ..., "down": ...}}`` where ``q`` is the
packed storage ``[out, in / 2]`` (two codes per byte, even input in the low
nibble) and ``s``, ``z`` are fp16 ``[out, in / 64]``.
"""

import numpy as np

from .quant import dequantize_g64, unpack_nibbles
from .routing import route, preroute


def silu(z):
    z = np.asarray(z, dtype=np.float64)
    return z / (1.0 + np.exp(-z))


def project(qsz, lora, v, lora_scale):
    """``W_int4 v + lora_scale * B (A v)`` with the delta kept unmerged."""
    qp, s, z = qsz
    v = np.asarray(v, dtype=np.float64)
    out = dequantize_g64(unpack_nibbles(qp), s, z) @ v
    if lora is not None:
        a, b = lora
        av = np.asarray(a, dtype=np.float64) @ v
        out = out + lora_scale * (np.asarray(b, dtype=np.float64) @ av)
    return out


def expert_forward(bundle, x16, lora_scale):
    """One SwiGLU expert on one token; returns (y [d], h [I])."""
    lo = bundle.get("lora") or {}
    x = np.asarray(x16, dtype=np.float16).astype(np.float64)
    g = project(bundle["gate"], lo.get("gate"), x, lora_scale)
    u = project(bundle["up"], lo.get("up"), x, lora_scale)
    h = silu(g) * u
    y = project(bundle["down"], lo.get("down"), h, lora_scale)
    return y, h


def combine(weights, y_routed, y_shared=()):
    """``y = sum_i w_i y_i + sum_s y_shared_s``."""
    y = np.zeros_like(np.asarray(y_routed[0], dtype=np.float64))
    for wi, yi in zip(weights, y_routed):
        y = y + float(wi) * np.asarray(yi, dtype=np.float64)
    for ys in y_shared:
        y = y + np.asarray(ys, dtype=np.float64)
    return y


def moe_layer(x16, k, routed, shared, lora_scale, w_router16=None,
              w_head16=None, routing=None):
    """One MoE layer on one token.

    ``routed(e)`` returns expert ``e``'s bundle (so tests only build the
    experts they touch); ``shared`` is a list of bundles.  The routing is the
    layer's own router on ``x`` unless ``routing = (inds, w)`` is given (a
    prediction consumed as routing, §3.2).  When ``w_head16`` is given, the
    head's prediction for the next layer is returned too.
    """
    out = {}
    if routing is None:
        l, inds, w = route(w_router16, x16, k)
        out["logits"] = l
    else:
        inds, w = routing
    out["idx"], out["w"] = np.asarray(inds, dtype=np.int32), np.asarray(w)
    ys = [expert_forward(routed(int(e)), x16, lora_scale)[0] for e in inds]
    yshared = [expert_forward(b, x16, lora_scale)[0] for b in shared]
    out["y_experts"] = ys + yshared
    out["y"] = combine(w, ys, yshared)
    if w_head16 is not None:
        pl, pi, pw = preroute(w_head16, x16, k)
        out["pred_logits"], out["pred_idx"], out["pred_w"] = pl, pi, pw
    return out
