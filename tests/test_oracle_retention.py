"""Pins of the merge-and-requantize oracle (§3.3, Recovery LoRA: the merged
alternative and its two retention measures).

Each pin fixes the result by a property of the int4 g64 grid rather than by
re-running the oracle's own formula:

* a zero change re-quantizes to the same bytes wherever a group's codes span
  0..15 (its min and max sit on the grid ends, so scale and zero reproduce);
* a change of whole grid steps at interior codes survives exactly
  (retention 1) and a change under half a step is erased exactly
  (retention 0), at the weight and at the expert-output level;
* a change far above the step survives up to the re-quantization error,
  which is at most half of the new step per weight, so the retention is
  within the Cauchy-Schwarz bound ||e|| / ||delta|| of 1;
* in the paper's regime (delta RMS 1e-3 against the int4 step of the
  synthetic weights) most of the change is lost, which is the paper's claim.
"""

import numpy as np
import pytest

from oracle import quant as Q, retention as RT, expert as EX


def _proj(rows, cols, seed, std=0.02):
    w = np.random.default_rng(seed).normal(0.0, std, size=(rows, cols)).astype(np.float32)
    q, s, z = Q.quantize_g64(w)
    return (Q.pack_nibbles(q), s, z), q


def _spanning_groups(q):
    g = q.reshape(q.shape[0], -1, Q.GROUP)
    return (g.min(axis=-1) == 0) & (g.max(axis=-1) == 15)


def test_zero_change_requantizes_to_same_bytes():
    qsz, q = _proj(32, 256, 1)
    span = _spanning_groups(q)
    assert span.mean() > 0.9
    (qp2, s2, z2), actual = RT.requantize_with(qsz, np.zeros((32, 256)))
    q2 = Q.unpack_nibbles(qp2).reshape(32, 4, Q.GROUP)
    q1 = q.reshape(32, 4, Q.GROUP)
    assert np.array_equal(q2[span], q1[span])
    assert np.array_equal(s2[span], qsz[1][span]) and np.array_equal(z2[span], qsz[2][span])
    assert np.all(actual.reshape(32, 4, Q.GROUP)[span] == 0.0)


def _interior_delta(q, s, rng, kind):
    """A change at interior codes only (1..14), zero at every code 0 / 15."""
    rows, cols = q.shape
    step = np.repeat(s.astype(np.float64), Q.GROUP, axis=1)
    interior = (q >= 1) & (q <= 14)
    if kind == "steps":   # whole steps, codes stay in 1..14
        k = rng.integers(-3, 4, size=q.shape)
        k = np.clip(q.astype(np.int64) + k, 1, 14) - q
        return np.where(interior, k * step, 0.0)
    frac = rng.uniform(-0.45, 0.45, size=q.shape)   # under half a step
    return np.where(interior, frac * step, 0.0)


def test_whole_steps_survive_exactly():
    rng = np.random.default_rng(2)
    qsz, q = _proj(16, 128, 2)
    span = np.repeat(_spanning_groups(q), Q.GROUP, axis=1)
    delta = np.where(span, _interior_delta(q, qsz[1], rng, "steps"), 0.0)
    assert np.any(delta != 0)
    _, actual = RT.requantize_with(qsz, delta)
    assert np.array_equal(actual, delta)
    assert RT.weight_retention(actual, delta) == 1.0


def test_sub_half_step_is_erased_exactly():
    rng = np.random.default_rng(3)
    qsz, q = _proj(16, 128, 3)
    span = np.repeat(_spanning_groups(q), Q.GROUP, axis=1)
    delta = np.where(span, _interior_delta(q, qsz[1], rng, "frac"), 0.0)
    (qp2, s2, z2), actual = RT.requantize_with(qsz, delta)
    assert np.all(actual[span] == 0.0)
    assert RT.weight_retention(actual[span], delta[span]) == 0.0


def test_large_change_within_requantization_bound():
    qsz, q = _proj(16, 256, 4)
    delta = np.random.default_rng(5).normal(0.0, 0.5, size=(16, 256))
    (qp2, s2, z2), actual = RT.requantize_with(qsz, delta)
    e = actual - delta
    # per weight: half the new step, plus the fp32 rounding of the merged value
    w = Q.dequantize_g64(q, qsz[1], qsz[2])
    half = np.repeat(s2.astype(np.float64), Q.GROUP, axis=1) / 2
    assert np.all(np.abs(e) <= half * (1 + 1e-3) + 2.0 ** -23 * np.abs(w + delta) + 1e-7)
    rho = RT.weight_retention(actual, delta)
    assert abs(rho - 1.0) <= np.linalg.norm(e) / np.linalg.norm(delta)
    assert abs(rho - 1.0) < 0.05


def _tiny_expert(seed, d=128, inter=64, r=4):
    rng = np.random.default_rng(seed)
    out = {"lora": {}}
    for p, (o, i) in {"gate": (inter, d), "up": (inter, d), "down": (d, inter)}.items():
        out[p] = _proj(o, i, seed * 7 + len(p))[0]
        out["lora"][p] = (rng.normal(0, 1.0 / r, size=(r, i)).astype(np.float16),
                          rng.normal(0, 1.0, size=(o, r)).astype(np.float16))
    return out


def test_output_level_erased_and_exact_cases():
    b = _tiny_expert(6)
    x = np.random.default_rng(7).normal(0, 1, size=(5, 128)).astype(np.float16)
    # scale 1e-9: every change is far under half a step (and moves no group's
    # min or max by half an fp16 ulp), so the merged expert is the base expert
    tiny = RT.expert_retention(b, x, 1e-9)
    for p in ("gate", "up", "down"):
        m, base = tiny["merged"][p], b[p]
        assert all(np.array_equal(u, v) for u, v in zip(m, base))
        assert tiny["weight"][p] == 0.0
    assert np.array_equal(tiny["M"], tiny["B"])
    assert tiny["output"] == 0.0
    # the unmerged expert with B = 0 is the base expert, bit for bit
    zb = {**b, "lora": {p: (a, np.zeros_like(bb)) for p, (a, bb) in b["lora"].items()}}
    assert np.array_equal(EX.expert_forward(zb, x[0], 2.0)[0], EX.expert_forward(b, x[0], 0.0)[0])


def test_output_level_whole_steps_merge_to_the_unmerged_expert():
    """Replace the adapters' delta by whole steps at interior codes: the merged
    expert then computes exactly W + delta, the unmerged expert's weight, so
    U == M up to float64 summation order and the retention is 1."""
    rng = np.random.default_rng(8)
    b = _tiny_expert(9)
    merged, unmerged = {"lora": {}}, {}
    for p in ("gate", "up", "down"):
        qsz = b[p]
        q = Q.unpack_nibbles(qsz[0])
        span = np.repeat(_spanning_groups(q), Q.GROUP, axis=1)
        delta = np.where(span, _interior_delta(q, qsz[1], rng, "steps"), 0.0)
        merged[p], actual = RT.requantize_with(qsz, delta)
        merged["lora"][p] = None
        assert np.array_equal(actual, delta)
        unmerged[p] = Q.dequantize_g64(q, qsz[1], qsz[2]) + delta
    x = np.random.default_rng(10).normal(0, 1, size=128).astype(np.float16).astype(np.float64)
    ym = EX.expert_forward(merged, x, 0.0)[0]
    h = EX.silu(unmerged["gate"] @ x) * (unmerged["up"] @ x)
    yu = unmerged["down"] @ h
    yb = EX.expert_forward(RT.base_bundle(b), x, 0.0)[0]
    assert np.allclose(ym, yu, rtol=1e-12, atol=1e-15)
    assert abs(RT.output_retention(yu, ym, yb) - 1.0) < 1e-9


def test_paper_regime_loses_most_of_the_change():
    """delta RMS about 1e-3 against N(0, 0.02) weights (group step about
    6e-3): the re-quantized merge keeps well under half of the change."""
    b = _tiny_expert(11, r=4)
    for p in b["lora"]:
        a, bb = b["lora"][p]
        # rescale B so that 2 B A has RMS 1e-3
        d = RT.lora_delta((a, bb), 2.0)
        b["lora"][p] = (a, (bb.astype(np.float64) * (1e-3 / np.sqrt(np.mean(d * d)))).astype(np.float16))
    x = np.random.default_rng(12).normal(0, 1, size=(8, 128)).astype(np.float16)
    res = RT.expert_retention(b, x, 2.0)
    for p in ("gate", "up", "down"):
        assert 0.0 < res["weight"][p] < 0.5, (p, res["weight"][p])
    assert res["output"] < 0.5


def test_undefined_cases_raise():
    with pytest.raises(ValueError):
        RT.weight_retention(np.zeros(4), np.zeros(4))
    with pytest.raises(ValueError):
        RT.output_retention(np.ones(3), np.ones(3), np.ones(3))
