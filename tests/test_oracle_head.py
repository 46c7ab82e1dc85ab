"""Pins of the oracle's full prerouter head (§3.2, Head): fc1 -> erf-GELU ->
fc2 plus the linear residual path on the hidden state, over the feature
[x, onehot(routed at t), onehot(routed at t-1)].

* GELU: closed-form values of the standard normal distribution and the
  identity gelu(z) - gelu(-z) = z (the tanh approximation fails both).
* A hand case with small integer weights whose logits are worked out below
  (feature order, biases, the fp16 rounding of the hidden activation, the
  residual path and the selection).
* With fc1 and fc2 zero the head is its linear residual path: the logits are
  exactly the linear head's (routing.logits_fp32, pinned in
  test_oracle_routing.py).
* The first token has no previous set: equal to any previous set whose fc1
  columns are zero.
"""

import numpy as np
import pytest

from oracle import routing

PHI1 = 0.8413447460685429   # standard normal CDF at 1 (textbook value)
PHI3 = 0.9986501019683699   # ... at 3


def test_gelu_erf_closed_forms():
    g = routing.gelu_erf(np.array([0.0, 1.0, -1.0, 8.0, -8.0]))
    assert g[0] == 0.0
    assert abs(g[1] - PHI1) < 1e-15
    assert abs(g[2] - (-(1.0 - PHI1))) < 1e-15
    assert abs(g[3] - 8.0) < 1e-13
    assert abs(g[4]) < 1e-13
    z = np.random.default_rng(0).normal(size=1000) * 3.0
    assert np.max(np.abs(routing.gelu_erf(z) - routing.gelu_erf(-z) - z)) < 1e-13


def test_head_hand_case():
    # d = 2, E = 3, H = 2, K = 1; x = [1, 2], routed at t = {2}, at t-1 = {0}
    # feature f = [1, 2 | 0, 0, 1 | 1, 0, 0]
    # fc1 row 0 = [1, 0 | 0, 0, 1 | 1, 0, 0] -> 1 + 1 + 1 = 3
    # fc1 row 1 = [0, 1 | 1, 0, 0 | 0, 0, 0] -> 2, plus b1 = -2 -> 0
    # hidden = fp16(gelu([3, 0])) = fp16([3 Phi(3), 0]) = [2.99609375, 0]
    #   (3 Phi(3) = 2.99595..., fp16 spacing 2^-9 on [2, 4): 1534 / 512)
    # fc2 rows [1, 0], [0, 1], [2, -1] -> [2.99609375, 0, 5.9921875]
    # + b2 [0, 0.5, 0] + W_l x ([0, 0], [1, 0], [0, 1] on [1, 2] -> [0, 1, 2])
    # logits = [2.99609375, 1.5, 7.9921875]; top-1 = expert 2, weight 1
    assert abs(3.0 * PHI3 - 2.99595) < 1e-5
    head = {
        "w1": np.array([[1, 0, 0, 0, 1, 1, 0, 0],
                        [0, 1, 1, 0, 0, 0, 0, 0]], dtype=np.float16),
        "b1": np.array([0, -2], dtype=np.float16),
        "w2": np.array([[1, 0], [0, 1], [2, -1]], dtype=np.float16),
        "b2": np.array([0, 0.5, 0], dtype=np.float16),
        "wl": np.array([[0, 0], [1, 0], [0, 1]], dtype=np.float16),
    }
    x = np.array([1, 2], dtype=np.float16)
    l, inds, w = routing.preroute_mlp(head, x, [2], [0], 1)
    assert l.dtype == np.float32
    assert l.tolist() == [2.99609375, 1.5, 7.9921875]
    assert inds.tolist() == [2] and w.tolist() == [1.0]
    # the two one-hot blocks swapped give a different fc1 row 0 (1 instead of 3)
    l2 = routing.prerouter_mlp_logits(head, x, [0], [2])
    assert l2.tolist() != l.tolist()


def test_head_zero_mlp_is_linear_head():
    rng = np.random.default_rng(1)
    d, e, h = 64, 16, 32
    wl = (rng.normal(size=(e, d)) * 0.05).astype(np.float16)
    x = rng.normal(size=d).astype(np.float16)
    head = {"w1": np.zeros((h, d + 2 * e), dtype=np.float16),
            "w2": np.zeros((e, h), dtype=np.float16), "wl": wl}
    l = routing.prerouter_mlp_logits(head, x, [1, 5], [3, 4])
    assert np.array_equal(l, routing.logits_fp32(wl, x))


def test_head_first_token_has_no_previous_set():
    rng = np.random.default_rng(2)
    d, e, h = 32, 8, 16
    w1 = (rng.normal(size=(h, d + 2 * e)) * 0.1).astype(np.float16)
    head = {"w1": w1, "w2": (rng.normal(size=(e, h)) * 0.1).astype(np.float16),
            "b1": (rng.normal(size=h) * 0.1).astype(np.float16)}
    x = rng.normal(size=d).astype(np.float16)
    first = routing.prerouter_mlp_logits(head, x, [2, 6], None)
    cut = dict(head)
    cut["w1"] = w1.copy()
    cut["w1"][:, d + e:] = 0
    assert np.array_equal(first, routing.prerouter_mlp_logits(cut, x, [2, 6], [0, 7]))
    assert not np.array_equal(first, routing.prerouter_mlp_logits(head, x, [2, 6], [0, 7]))
