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

The full prerouter head follows §3.2 (Head): per layer
``fc1 -> erf-GELU -> fc2`` plus a linear residual path ``l`` on the hidden
state; the input feature is the hidden state concatenated with two top-k
one-hots, the experts this layer routed to at this token and those at the
previous token (``d + 2E`` features).  Readings for the head:

* Feature order: ``[x (d), onehot(routed at t) (E), onehot(routed at t-1) (E)]``;
  at the first token the previous-token one-hot is all zero.
* Both linear layers carry optional fp16 biases (zero when absent); ``l``
  acts on ``x`` alone (``W_l [E, d]``, the shape of the next layer's router,
  from which it is warm-started; absent means zero).
* Precision (the heads are fp16): fc1's pre-activation and GELU are exact
  (float64), the hidden activation is rounded once to fp16 (it is fc2's fp16
  input), and ``fc2(hidden) + b2 + l(x)`` is exact and rounded once to fp32.
* GELU is the erf form ``z * Phi(z) = z (1 + erf(z / sqrt 2)) / 2``.
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


def gelu_erf(z):
    """erf-GELU ``z Phi(z)`` in float64 (§3.2, Head)."""
    from scipy.special import erf
    z = np.asarray(z, dtype=np.float64)
    return 0.5 * z * (1.0 + erf(z / np.sqrt(2.0)))


def prerouter_feature(x16, routed_t, routed_tm1, n_experts):
    """The head's input: ``x`` followed by the one-hots of the set routed at
    this token and at the previous one (``None`` at the first token), as
    float64 ``[d + 2E]``."""
    x = np.asarray(x16, dtype=np.float16).astype(np.float64)
    oh = np.zeros(2 * n_experts, dtype=np.float64)
    oh[np.asarray(routed_t, dtype=np.int64)] = 1.0
    if routed_tm1 is not None:
        oh[n_experts + np.asarray(routed_tm1, dtype=np.int64)] = 1.0
    return np.concatenate([x, oh])


def prerouter_mlp_logits(head, x16, routed_t, routed_tm1):
    """Full prerouter head logits, fp32 ``[E]``.

    ``head``: dict with ``w1`` fp16 ``[H, d + 2E]``, ``w2`` fp16 ``[E, H]``,
    and optional ``b1`` fp16 ``[H]``, ``b2`` fp16 ``[E]``, ``wl`` fp16
    ``[E, d]`` (None or absent: zero).
    """
    w1 = np.asarray(head["w1"], dtype=np.float16).astype(np.float64)
    w2 = np.asarray(head["w2"], dtype=np.float16).astype(np.float64)
    n_e = w2.shape[0]
    f = prerouter_feature(x16, routed_t, routed_tm1, n_e)
    pre = w1 @ f
    if head.get("b1") is not None:
        pre = pre + np.asarray(head["b1"], dtype=np.float16).astype(np.float64)
    hid = gelu_erf(pre).astype(np.float16).astype(np.float64)
    out = w2 @ hid
    if head.get("b2") is not None:
        out = out + np.asarray(head["b2"], dtype=np.float16).astype(np.float64)
    if head.get("wl") is not None:
        wl = np.asarray(head["wl"], dtype=np.float16).astype(np.float64)
        out = out + wl @ np.asarray(x16, dtype=np.float16).astype(np.float64)
    return out.astype(np.float32)


def preroute_mlp(head, x16, routed_t, routed_tm1, k):
    """Full prerouter head + softmax-top-k: the next layer's routing at the
    next token (§3.2, Head and Prediction-as-routing)."""
    l = prerouter_mlp_logits(head, x16, routed_t, routed_tm1)
    inds, w = softmax_topk(l, k)
    return l, inds, w


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
