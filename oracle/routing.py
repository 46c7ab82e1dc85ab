"""Oracle: layer input, router / prerouter logits and routing (TEST INFRASTRUCTURE ONLY).

Softmax-top-k follows App. A (Softmax-topk): ``g = softmax(l)``,
``inds = top-k(g, K)``, ``w = g[inds] / sum(g[inds])``.  The same function
serves the layer's own router and the prerouter head, whose prediction is
consumed as the next layer's routing (§3.2, Prediction-as-routing).

Sigmoid-group routing follows App. A (Sigmoid-group): sigmoid scores, group
score = sum of the group's top two, the best ``G`` of ``n`` groups survive,
top-k among survivors, weights ``s * sigma[inds] / (sum sigma[inds] + 1e-20)``;
selection uses the biased score and the weights use the raw sigmoid.

Readings (the paper is silent on these):

* Layer input: ``x = fp16(xi / sqrt(mean(xi^2) + 1e-6))`` with no learned
  scale.  The normalized value is computed in float64 and rounded once to
  fp16 (round-to-nearest-even).  The fp16 code of ``x`` is decided by
  floating point, and float64 makes the decision independent of the order
  of the reduction.
* Router and head logits are fp32: the exact dot product of fp16 weights and
  fp16 activations (computed in float64, where every product is exact),
  rounded once to fp32.
* Top-k order: descending, ties to the lower expert index.  The softmax is
  strictly increasing in the logit, so the set equals the top-k of the logits
  except where two logits are closer than float64 can separate after the
  exponential.
* Sigmoid-group bias: an optional per-expert vector added to the sigmoid
  before selection (zero when absent); group membership is contiguous
  (group ``i`` holds experts ``i*E/n .. (i+1)*E/n - 1``).
"""

import numpy as np

RMS_EPS = 1e-6


def rms_norm_f16(xi, eps=RMS_EPS):
    """Layer input: RMS-normalize fp32 rows of ``xi`` and store as fp16."""
    xi = np.asarray(xi, dtype=np.float32)
    x64 = xi.astype(np.float64)
    ms = np.mean(x64 * x64, axis=-1, keepdims=True)
    r = 1.0 / np.sqrt(ms + eps)
    return (x64 * r).astype(np.float16)


def logits_fp32(w16, x16):
    """Router or head logits ``l = W x`` for fp16 ``W [E, d]`` and ``x [.., d]``.

    Every fp16 x fp16 product is exact in float64 and the float64 sum of at
    most a few thousand of them is within a few float64 ulps of exact; the
    result is rounded once to fp32.
    """
    w64 = np.asarray(w16, dtype=np.float16).astype(np.float64)
    x64 = np.asarray(x16, dtype=np.float16).astype(np.float64)
    return (x64 @ w64.T).astype(np.float32)


def softmax(l):
    l = np.asarray(l, dtype=np.float64)
    m = np.max(l)
    e = np.exp(l - m)
    return e / np.sum(e)


def topk_desc(values, k):
    """Indices of the ``k`` largest values, descending, ties to the lower index."""
    order = np.argsort(-np.asarray(values, dtype=np.float64), kind="stable")
    return order[:k].astype(np.int32)


def softmax_topk(l, k):
    """App. A softmax-top-k for one token's logits ``l [E]`` -> (inds int32 [k], w [k])."""
    g = softmax(l)
    inds = topk_desc(g, k)
    w = g[inds] / np.sum(g[inds])
    return inds, w


def route(w_router16, x16, k):
    """Router logits followed by softmax-top-k, for one token."""
    l = logits_fp32(w_router16, x16)
    inds, w = softmax_topk(l, k)
    return l, inds, w


def preroute(w_head16, x16, k):
    """Prerouter head (the linear path at these shapes) + the same routing math.

    The returned set and weights are the routing of the *next* layer at the
    *next* token (§3.2, Motivation and Prediction-as-routing).
    """
    return route(w_head16, x16, k)


def near_tie_gap(l, k):
    """Gap between the k-th and (k+1)-th largest logits (inf when k == E)."""
    l = np.sort(np.asarray(l, dtype=np.float64))[::-1]
    if k >= l.size:
        return np.inf
    return float(l[k - 1] - l[k])


def sigmoid_group_topk(l, k, n_groups, top_groups, scale, bias=None):
    """App. A sigmoid-group routing for one token's logits ``l [E]``."""
    l = np.asarray(l, dtype=np.float64)
    e = l.size
    if e % n_groups:
        raise ValueError("E must be a multiple of the group count")
    sig = 1.0 / (1.0 + np.exp(-l))
    sel = sig + (0.0 if bias is None else np.asarray(bias, dtype=np.float64))
    per = e // n_groups
    grp = sel.reshape(n_groups, per)
    gscore = np.array([np.sum(np.sort(row)[::-1][:2]) for row in grp])
    keep = topk_desc(gscore, top_groups)
    masked = np.full(e, -np.inf)
    for gi in keep:
        masked[gi * per:(gi + 1) * per] = sel[gi * per:(gi + 1) * per]
    inds = topk_desc(masked, k)
    w = scale * sig[inds] / (np.sum(sig[inds]) + 1e-20)
    return inds, w
