"""Oracle: one MoE layer over a batch of tokens (TEST INFRASTRUCTURE ONLY).

Batched decode and prefill compute, per token, exactly what the one-token
layer computes (§3.1, Executor paths: *whole-layer* loads every expert of a
layer for prefill, and the Math contract requires every path to produce the
same outputs).  Grouping tokens by expert is an execution strategy of the
kernels, so the oracle simply loops over tokens.

Readings:

* Routing is softmax-top-k (App. A) on given fp32 logits ``[T, E]``; the
  synthetic logits stand in for router outputs with a skewed popularity.
"""

import numpy as np

from .routing import softmax_topk
from .expert import expert_forward, combine


def batched_layer(x16, logits, k, routed, shared, lora_scale, tokens=None):
    """``x16 [T, d]`` fp16, ``logits [T, E]`` fp32 -> dict of idx, w, y [T, d].

    ``tokens`` restricts the expert computation to a subset of token indices
    (routing is still computed for all); rows not computed are NaN.
    """
    x16 = np.asarray(x16, dtype=np.float16)
    t_all = x16.shape[0]
    idx = np.zeros((t_all, k), dtype=np.int32)
    w = np.zeros((t_all, k))
    for t in range(t_all):
        idx[t], w[t] = softmax_topk(logits[t], k)
    y = np.full((t_all, x16.shape[1]), np.nan)
    cache = {}

    def bundle(e):
        if e not in cache:
            cache[e] = routed(e)
        return cache[e]

    for t in (range(t_all) if tokens is None else tokens):
        ys = [expert_forward(bundle(int(e)), x16[t], lora_scale)[0] for e in idx[t]]
        ysh = [expert_forward(b, x16[t], lora_scale)[0] for b in shared]
        y[t] = combine(w[t], ys, ysh)
    return {"idx": idx, "w": w, "y": y}
