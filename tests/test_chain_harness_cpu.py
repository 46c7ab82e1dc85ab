"""CPU checks of the teacher-forced chain comparison used by the GPU chain
tests: it accepts the oracle chain's own records, and it rejects records
with a planted mistake (a wrong residual, a layer input off by one fp16 ulp,
a routing swap away from a near-tie, a prediction not used as routing, a
layer output off by more than the bar)."""

import numpy as np
import pytest

import synth
from oracle import stack as o_stack
from tests.gpu_harness import teacher_forced_chain, free_running_divergence, sample_layers


def _layers(wl, L):
    out = []
    for n in range(L):
        d, perm = synth.mixing(wl, n)
        out.append({"router": synth.router_weights(wl, n, 0),
                    "head": synth.router_weights(wl, n, 1) if n + 1 < L else None,
                    "mix_d": d, "mix_perm": perm,
                    "routed": (lambda e, n=n: synth.bundle(wl, n, e)),
                    "shared": [synth.bundle(wl, n, wl.E + s) for s in range(wl.S)]})
    return out


@pytest.fixture(scope="module")
def chain():
    wl = synth.WORKLOADS["tiny"]
    L, T = 4, 3
    layers = _layers(wl, L)
    xi = synth.token_draws(wl, 0, T)
    ref = o_stack.decode_chain(xi, layers, wl.K, wl.lora_scale)
    rec = {"r": np.zeros((T, L, wl.d), np.float32), "x": np.zeros((T, L, wl.d), np.float16),
           "idx": np.zeros((T, L, wl.K), np.int32), "w": np.zeros((T, L, wl.K), np.float32),
           "pidx": np.full((T, L, wl.K), -1, np.int32), "pw": np.zeros((T, L, wl.K), np.float32),
           "y": np.zeros((T, L, wl.d), np.float32)}
    for t in range(T):
        for n in range(L):
            r = ref[t][n]
            rec["r"][t, n], rec["x"][t, n] = r["r_mixed"], r["x16"]
            rec["idx"][t, n], rec["w"][t, n], rec["y"][t, n] = r["idx"], r["w"], r["y"]
            if "pred_idx" in r:
                rec["pidx"][t, n], rec["pw"][t, n] = r["pred_idx"], r["pred_w"]
    return wl, L, T, layers, xi, rec


def _copy(rec):
    return {k: v.copy() for k, v in rec.items()}


def test_accepts_the_oracle_chain(chain):
    wl, L, T, layers, xi, rec = chain
    stats = teacher_forced_chain(rec, xi, layers, wl, L)
    assert stats["steps"] == L * T and stats["y_checked"] == L * T
    assert stats["pred_routing"] == (T - 1) * (L - 1)
    assert free_running_divergence(rec, xi, layers, wl, L) is None


def test_rejects_planted_mistakes(chain):
    wl, L, T, layers, xi, rec = chain
    bad = _copy(rec)
    bad["r"][1, 2, 5] *= 1.0 + 1e-5                       # residual off
    with pytest.raises(AssertionError, match="stand-in"):
        teacher_forced_chain(bad, xi, layers, wl, L)
    bad = _copy(rec)
    bad["x"][2, 1, 7] = np.nextafter(bad["x"][2, 1, 7], np.float16(np.inf))   # one fp16 ulp
    with pytest.raises(AssertionError, match="layer input"):
        teacher_forced_chain(bad, xi, layers, wl, L)
    bad = _copy(rec)
    bad["idx"][0, 1, [0, 1]] = bad["idx"][0, 1, [1, 0]]      # order swap, not a near-tie
    with pytest.raises(AssertionError):
        teacher_forced_chain(bad, xi, layers, wl, L)
    bad = _copy(rec)
    bad["idx"][2, 3, 0] = (bad["idx"][2, 3, 0] + 1) % wl.E   # not the prediction made for it
    with pytest.raises(AssertionError, match="prediction not used"):
        teacher_forced_chain(bad, xi, layers, wl, L)
    bad = _copy(rec)
    bad["y"][1, 1] *= 1.01                                   # output beyond the bar
    with pytest.raises(AssertionError):
        teacher_forced_chain(bad, xi, layers, wl, L)


def test_sample_layers_covers_first_tokens():
    f = sample_layers(5, 10, full_tokens=2, per_token=3)
    assert all(f(t, n) for t in range(2) for n in range(10))
    assert all(sum(f(t, n) for n in range(10)) == 3 for t in range(2, 5))
