"""Oracle: multi-layer decode chain with prediction-as-routing (TEST INFRASTRUCTURE ONLY).

§3.2 (Motivation): the head owned by layer N runs at token t on layer N's
input and predicts layer N+1's routing at token t+1; layer N+1 consumes that
prediction as its routing (Prediction-as-routing).  Layers without a
prediction (layer 0, every layer at the first token, layers outside the
consumer range) route with their own router.

Readings (the paper's decoder has attention; this chain has none):

* Attention is replaced by a fixed residual mixing.  With ``r`` the fp32
  residual of one token: ``r_0 = xi_t + rmsnorm(r_L of the previous token)``
  (zero before the first token, the normalization done in float64); every
  layer N does ``r <- r + D_N * r[perm_N]`` with fp16 ``D_N`` and a fixed
  permutation, then ``x_N = fp16(rmsnorm(r))``, then ``r <- r + y_N``.
* The oracle carries ``r`` in float64; the fp16 rounding of ``x_N`` is the
  layer-input rounding of :func:`oracle.routing.rms_norm_f16`.
* The consumer range defaults to every layer ``1 .. L-1``; the head of the
  last layer is not evaluated.
"""

import numpy as np

from .routing import route, preroute, RMS_EPS
from .expert import expert_forward, combine


def _rmsnorm64(v, eps=RMS_EPS):
    v = np.asarray(v, dtype=np.float64)
    return v / np.sqrt(np.mean(v * v) + eps)


def _x16(r):
    return _rmsnorm64(r).astype(np.float16)


def decode_chain(tokens_xi, layers, k, lora_scale, consumers=None):
    """Run the chain over ``tokens_xi [T, d]`` (fp32 draws).

    ``layers[N]`` is a dict with ``router`` (fp16 [E, d]), ``head`` (fp16
    [E, d] or None), ``mix_d`` (fp16 [d]), ``mix_perm`` (int [d]),
    ``routed(e)`` -> bundle and ``shared`` (list of bundles).
    Returns a per-token list of per-layer records (x16, idx, w, y, y_experts,
    source, and the head's prediction).
    """
    nl = len(layers)
    if consumers is None:
        consumers = set(range(1, nl))
    pred = {}                     # (t, N) -> (idx, w) predicted one token earlier
    r_prev = None
    out = []
    for t, xi in enumerate(np.asarray(tokens_xi, dtype=np.float32)):
        r = np.asarray(xi, dtype=np.float64)
        if r_prev is not None:
            r = r + _rmsnorm64(r_prev)
        recs = []
        for n, lay in enumerate(layers):
            r = r + np.asarray(lay["mix_d"], dtype=np.float64) * r[np.asarray(lay["mix_perm"])]
            x16 = _x16(r)
            if t > 0 and n in consumers and (t, n) in pred:
                idx, w = pred[(t, n)]
                src = "pred"
            else:
                _, idx, w = route(lay["router"], x16, k)
                src = "router"
            ys = [expert_forward(lay["routed"](int(e)), x16, lora_scale)[0] for e in idx]
            ysh = [expert_forward(b, x16, lora_scale)[0] for b in lay["shared"]]
            y = combine(w, ys, ysh)
            rec = {"x16": x16, "idx": np.asarray(idx), "w": np.asarray(w), "y": y, "src": src,
                   "y_experts": ys + ysh}
            if n + 1 < nl and lay.get("head") is not None:
                pl, pi, pw = preroute(lay["head"], x16, k)
                pred[(t + 1, n + 1)] = (pi, pw)
                rec["pred_idx"], rec["pred_w"], rec["pred_logits"] = pi, pw, pl
            recs.append(rec)
            r = r + y
        out.append(recs)
        r_prev = r
    return out
