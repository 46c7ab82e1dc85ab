"""Pins for the oracle's layer input and routing math (CPU only).

Softmax-top-k (App. A) is fixed by brute force over every K-subset, by a
library softmax in the K = E case, by shift invariance and by K = 1.  The
logits are fixed by exact rational arithmetic, the layer input by a hand-
derived case.  Sigmoid-group routing (App. A) is fixed by its reductions to
plain top-k and by brute force over group choices.
"""

import itertools
import json
import os
from fractions import Fraction

import numpy as np
import pytest
from scipy.special import softmax as sp_softmax

from oracle import routing

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _fp32_ulp(v):
    v = np.float32(abs(v))
    return float(np.nextafter(v, np.float32(np.inf)) - v)


def test_rmsnorm_hand_case():
    g = json.load(open(os.path.join(GOLD, "closed_forms.json")))
    x = routing.rms_norm_f16(np.array([3.0, 4.0], dtype=np.float32))
    assert x.dtype == np.float16
    assert x.astype(np.float64).tolist() == g["rmsnorm_3_4"]["value"]


def test_rmsnorm_unit_rms():
    rs = np.random.default_rng(0)
    xi = rs.normal(0, 3.0, size=(4, 2048)).astype(np.float32)
    x = routing.rms_norm_f16(xi).astype(np.float64)
    rms = np.sqrt(np.mean(x * x, axis=-1))
    assert np.all(np.abs(rms - 1) < 2e-3)
    # row-wise: scaling a row scales nothing in the output (up to epsilon)
    x2 = routing.rms_norm_f16(xi * 8).astype(np.float64)
    assert np.mean(x2 == x) > 0.999


def test_logits_exact_rational():
    rs = np.random.default_rng(1)
    w = rs.normal(0, 0.02, size=(6, 96)).astype(np.float16)
    x = rs.normal(0, 1, size=96).astype(np.float16)
    got = routing.logits_fp32(w, x)
    assert got.dtype == np.float32
    for e in range(6):
        exact = sum(Fraction(float(w[e, j])) * Fraction(float(x[j])) for j in range(96))
        err = abs(Fraction(float(got[e])) - exact)
        assert err <= Fraction(_fp32_ulp(float(exact))) / 2 * Fraction(1001, 1000)


def test_softmax_topk_sum_and_k1():
    rs = np.random.default_rng(2)
    for _ in range(20):
        l = rs.normal(0, 1, size=16).astype(np.float32)
        for k in (1, 2, 5, 16):
            inds, w = routing.softmax_topk(l, k)
            assert abs(np.sum(w) - 1.0) < 1e-12
            assert len(set(inds.tolist())) == k
        inds, w = routing.softmax_topk(l, 1)
        assert w.tolist() == [1.0] and inds[0] == int(np.argmax(l))


def test_softmax_topk_k_equals_e_is_full_softmax():
    rs = np.random.default_rng(3)
    l = rs.normal(0, 2, size=32).astype(np.float32)
    inds, w = routing.softmax_topk(l, 32)
    ref = sp_softmax(l.astype(np.float64))
    assert np.allclose(w, ref[inds], rtol=1e-13, atol=0)


def test_softmax_topk_shift_invariant():
    rs = np.random.default_rng(4)
    # multiples of 2^-10 in [-4, 4]: adding 2.0 is exact in fp32
    l = (rs.integers(-4096, 4096, size=64) / 1024.0).astype(np.float32)
    i1, w1 = routing.softmax_topk(l, 8)
    i2, w2 = routing.softmax_topk(l + np.float32(2.0), 8)
    assert i1.tolist() == i2.tolist()
    assert np.allclose(w1, w2, rtol=1e-14, atol=0)


def test_topk_brute_force_all_subsets():
    rs = np.random.default_rng(5)
    for trial in range(40):
        e = int(rs.integers(2, 9))
        k = int(rs.integers(1, e + 1))
        l = rs.normal(0, 1, size=e).astype(np.float32)
        inds, w = routing.softmax_topk(l, k)
        g = sp_softmax(l.astype(np.float64))
        best = max(itertools.combinations(range(e), k), key=lambda c: sum(g[i] for i in c))
        assert sorted(inds.tolist()) == sorted(best)
        # descending order of the selected values
        assert all(l[inds[i]] >= l[inds[i + 1]] for i in range(k - 1))
        # weights: the renormalized softmax restricted to the set
        assert np.allclose(w, g[inds] / sum(g[i] for i in best), rtol=1e-13)


def test_topk_ties_go_to_lower_index():
    l = np.array([1.0, 3.0, 3.0, 2.0, 3.0], dtype=np.float32)
    assert routing.softmax_topk(l, 1)[0].tolist() == [1]
    assert routing.softmax_topk(l, 2)[0].tolist() == [1, 2]
    assert routing.softmax_topk(l, 4)[0].tolist() == [1, 2, 4, 3]


def test_topk_matches_argsort_of_logits():
    rs = np.random.default_rng(6)
    l = rs.normal(0, 1, size=(50, 256)).astype(np.float32)
    for row in l:
        inds, _ = routing.softmax_topk(row, 8)
        assert inds.tolist() == np.argsort(-row, kind="stable")[:8].tolist()


def test_near_tie_gap():
    l = np.array([0.5, 0.1, 0.3, 0.2], dtype=np.float32)
    assert routing.near_tie_gap(l, 2) == pytest.approx(0.1, abs=1e-7)
    assert routing.near_tie_gap(l, 4) == np.inf


def test_sigmoid_group_single_group_is_plain_topk():
    rs = np.random.default_rng(7)
    l = rs.normal(0, 1, size=16)
    inds, w = routing.sigmoid_group_topk(l, 4, n_groups=1, top_groups=1, scale=2.5)
    sig = 1 / (1 + np.exp(-l))
    assert inds.tolist() == np.argsort(-l, kind="stable")[:4].tolist()
    assert np.allclose(w, 2.5 * sig[inds] / sig[inds].sum(), rtol=1e-14)
    assert abs(w.sum() - 2.5) < 1e-12
    # all groups surviving is the same as no grouping
    inds2, w2 = routing.sigmoid_group_topk(l, 4, n_groups=4, top_groups=4, scale=2.5)
    assert inds2.tolist() == inds.tolist() and np.allclose(w, w2)


def test_sigmoid_group_brute_force():
    rs = np.random.default_rng(8)
    for trial in range(30):
        l = rs.normal(0, 1, size=8)
        bias = rs.normal(0, 0.3, size=8)
        inds, w = routing.sigmoid_group_topk(l, 2, n_groups=4, top_groups=2, scale=1.0, bias=bias)
        sig = 1 / (1 + np.exp(-l))
        sel = sig + bias
        # groups of 2: group score = the sum of both members (its top 2)
        gs = [sel[2 * i] + sel[2 * i + 1] for i in range(4)]
        keep = max(itertools.combinations(range(4), 2), key=lambda c: sum(gs[i] for i in c))
        members = [e for gi in keep for e in (2 * gi, 2 * gi + 1)]
        best = max(itertools.combinations(members, 2), key=lambda c: sum(sel[i] for i in c))
        assert sorted(inds.tolist()) == sorted(best)
        # weights use the raw sigmoid, not the biased score
        assert np.allclose(w, sig[inds] / sig[inds].sum(), rtol=1e-13)


def test_sigmoid_group_hand_case():
    # 8 experts, 4 groups of 2, keep 2 groups, K = 2.
    # group scores (sum of the pair): g0 = s(2)+s(-1) = 1.150, g1 = s(0)+s(0) = 1,
    # g2 = s(3)+s(1) = 1.684, g3 = s(-1)+s(-3) = 0.316 -> g2 and g0 survive;
    # the top two sigmoids among experts 0, 1, 4, 5 are s(3) (4) and s(2) (0).
    l = np.array([2.0, -1.0, 0.0, 0.0, 3.0, 1.0, -1.0, -3.0])
    inds, w = routing.sigmoid_group_topk(l, 2, n_groups=4, top_groups=2, scale=2.5)
    assert inds.tolist() == [4, 0]
    s3, s2 = 1 / (1 + np.exp(-3.0)), 1 / (1 + np.exp(-2.0))
    assert np.allclose(w, [2.5 * s3 / (s3 + s2), 2.5 * s2 / (s3 + s2)], rtol=1e-14)


def test_rmsnorm_single_rounding_against_high_precision():
    """The layer input is the fp16 nearest (ties to even) to the exact
    normalized value: checked with 40-digit decimal arithmetic."""
    from decimal import Decimal, getcontext
    getcontext().prec = 40
    rs = np.random.default_rng(9)
    xi = rs.normal(0, 2.0, size=(8, 2048)).astype(np.float32)
    got = routing.rms_norm_f16(xi)
    for t in range(xi.shape[0]):
        ds = [Decimal(float(v)) for v in xi[t]]
        ms = sum(v * v for v in ds) / Decimal(xi.shape[1])
        r = Decimal(1) / (ms + Decimal("1e-6")).sqrt()
        for j in range(xi.shape[1]):
            v = ds[j] * r
            c = np.float16(float(v))
            cands = [np.nextafter(c, np.float16(-np.inf)), c, np.nextafter(c, np.float16(np.inf))]
            dist = [abs(Decimal(float(cc)) - v) for cc in cands]
            best = min(dist)
            near = [cc for cc, dd in zip(cands, dist) if dd == best]
            if len(near) > 1:
                near = [cc for cc in near if int(cc.view(np.uint16)) % 2 == 0]
            assert got[t, j].view(np.uint16) == near[0].view(np.uint16), (t, j)
