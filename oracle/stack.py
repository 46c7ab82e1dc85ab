"""Oracle: multi-layer decode chain with prediction-as-routing (TEST INFRASTRUCTURE ONLY).

§3.2 (Motivation): the head owned by layer N runs at token t on layer N's
input and predicts layer N+1's routing at token t+1; layer N+1 consumes that
prediction as its routing (Prediction-as-routing).  Layers without a
prediction (layer 0, every layer at the first token, layers outside the
consumer range) route with their own router.

Readings (the paper's decoder has attention; this chain has none):

* Attention is replaced by a fixed residual mixing on the residual ``r`` of
  one token, which is stored in fp32 (the type the method keeps it in):

  - token start (:func:`token_start`): ``r = xi_t + rmsnorm(r_prev)``, where
    ``r_prev`` is the residual the previous token left after its last layer
    (nothing is added at the first token);
  - before layer N (:func:`mix`): ``r <- r + D_N * r[perm_N]`` with fp16
    ``D_N`` and a fixed permutation (element j takes element ``perm_N[j]``);
  - layer input: ``x_N = fp16(rmsnorm(r))`` (:func:`oracle.routing.rms_norm_f16`);
  - after layer N (:func:`add_output`): ``r <- r + y_N``.

  Each update is computed in float64 and rounded once to fp32.  (Where the
  float64 value is itself rounded, the fp32 result can differ from the
  correctly rounded one, with a chance of about 2^-29 per element; the GPU
  tests compare residuals within one fp32 ulp.)
* The consumer range defaults to every layer ``1 .. L-1``; the head of the
  last layer is not evaluated.
"""

import numpy as np

from .routing import route, preroute, rms_norm_f16, RMS_EPS
from .expert import expert_forward, combine


def token_start(xi, r_prev=None, eps=RMS_EPS):
    """Residual at the start of a token: ``fp32(xi + rmsnorm(r_prev))``
    (``xi`` alone at the first token, ``r_prev is None``).  The RMS norm has
    no learned scale and is computed in float64."""
    r = np.asarray(xi, dtype=np.float32).astype(np.float64)
    if r_prev is not None:
        p = np.asarray(r_prev, dtype=np.float32).astype(np.float64)
        r = r + p / np.sqrt(np.mean(p * p) + eps)
    return r.astype(np.float32)


def mix(r, mix_d, mix_perm):
    """Attention stand-in of one layer: ``fp32(r + D * r[perm])`` for the fp32
    residual ``r``, fp16 ``D`` and the permutation ``perm``."""
    r64 = np.asarray(r, dtype=np.float32).astype(np.float64)
    d64 = np.asarray(mix_d, dtype=np.float16).astype(np.float64)
    return (r64 + d64 * r64[np.asarray(mix_perm, dtype=np.int64)]).astype(np.float32)


def add_output(r, y):
    """Residual after a layer: ``fp32(r + y)``."""
    return (np.asarray(r, dtype=np.float32).astype(np.float64)
            + np.asarray(y, dtype=np.float64)).astype(np.float32)


def decode_chain(tokens_xi, layers, k, lora_scale, consumers=None):
    """Run the chain over ``tokens_xi [T, d]`` (fp32 draws).

    ``layers[N]`` is a dict with ``router`` (fp16 [E, d]), ``head`` (fp16
    [E, d] or None), ``mix_d`` (fp16 [d]), ``mix_perm`` (int [d]),
    ``routed(e)`` -> bundle and ``shared`` (list of bundles).
    Returns a per-token list of per-layer records (the mixed residual
    ``r_mixed``, x16, idx, w, y, y_experts, source, and the head's prediction).
    """
    nl = len(layers)
    if consumers is None:
        consumers = set(range(1, nl))
    pred = {}                     # (t, N) -> (idx, w) predicted one token earlier
    r_prev = None
    out = []
    for t, xi in enumerate(np.asarray(tokens_xi, dtype=np.float32)):
        r = token_start(xi, r_prev)
        recs = []
        for n, lay in enumerate(layers):
            r = mix(r, lay["mix_d"], lay["mix_perm"])
            x16 = rms_norm_f16(r)
            if t > 0 and n in consumers and (t, n) in pred:
                idx, w = pred[(t, n)]
                src = "pred"
            else:
                _, idx, w = route(lay["router"], x16, k)
                src = "router"
            ys = [expert_forward(lay["routed"](int(e)), x16, lora_scale)[0] for e in idx]
            ysh = [expert_forward(b, x16, lora_scale)[0] for b in lay["shared"]]
            y = combine(w, ys, ysh)
            rec = {"r_mixed": r, "x16": x16, "idx": np.asarray(idx), "w": np.asarray(w), "y": y,
                   "src": src, "y_experts": ys + ysh}
            if n + 1 < nl and lay.get("head") is not None:
                pl, pi, pw = preroute(lay["head"], x16, k)
                pred[(t + 1, n + 1)] = (pi, pw)
                rec["pred_idx"], rec["pred_w"], rec["pred_logits"] = pi, pw, pl
            recs.append(rec)
            r = add_output(r, y)
        out.append(recs)
        r_prev = r
    return out
