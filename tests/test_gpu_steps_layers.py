"""GPU parity of the independent-step schedules in the configuration the
benchmark launches them: a slot table of several layers whose experts,
routers and heads all differ, and steps whose table layer rotates over them
(``step_layer``), with the workspace sized for the whole table.

Each step is compared with the oracle layer of its own table layer: routing
and prediction bit-exact except at counted near-ties (oracle K-th / (K+1)-th
logit gap within 1e-5), layer output within 2e-3.  The last table layer has
no head: its steps must leave the prediction records untouched.  Workloads:
the tiny layer over its 1000 seeded tokens, and the 35B-class layer over 128
tokens; the near-tie counts are printed.
"""

import numpy as np
import pytest

import synth
from oracle import expert as o_expert, routing as o_routing
from tests.gpu_harness import TOL_REL_INF, build_chain, check_routing, rel_inf

pytestmark = pytest.mark.gpu

N_LAYERS = 4          # table layers; the last one has no head


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    from paper_2609_18063_amd import binding
    binding.lib()
    return torch


def _stack(wl, torch):
    from paper_2609_18063_amd import binding as B
    chain, np_layers = build_chain(wl, N_LAYERS, torch)
    arr = B.engine_layer_array(chain.layers)
    return chain, np_layers, arr


def _run(fn, chain, arr, steps, xi, torch, ws=None):
    from paper_2609_18063_amd import binding as B
    spec = chain.spec
    d, K = spec.d_model, spec.top_k
    T = xi.shape[0]
    if ws is None:
        ws = torch.zeros(B.engine_workspace_bytes(spec, N_LAYERS), dtype=torch.uint8, device="cuda")
    out = {
        "y": torch.full((T, d), float("nan"), dtype=torch.float32, device="cuda"),
        "idx": torch.full((T, K), -7, dtype=torch.int32, device="cuda"),
        "w": torch.zeros(T, K, dtype=torch.float32, device="cuda"),
        "pidx": torch.full((T, K), -7, dtype=torch.int32, device="cuda"),
        "pw": torch.zeros(T, K, dtype=torch.float32, device="cuda"),
        "status": torch.zeros(1, dtype=torch.int32, device="cuda"),
    }
    steps_t = torch.from_numpy(np.ascontiguousarray(steps, dtype=np.int32)).cuda()
    xi_t = torch.from_numpy(np.ascontiguousarray(xi)).cuda()
    print("launch %s: T=%d d=%d layers %s" % (fn, T, d, np.bincount(steps).tolist()), flush=True)
    getattr(B, fn)(spec, chain.table, arr, steps_t, xi_t, out["y"], ws, idx=out["idx"], w=out["w"],
                   pidx=out["pidx"], pw=out["pw"], status=out["status"])
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}, ws


def _check(wl, np_layers, steps, xi, out, what, y_tokens=None):
    K = wl.K
    assert int(out["status"][0]) == 0, (what, out["status"])
    stats = {"routing": {}, "prediction": {}, "y_checked": 0, "max_err": 0.0, "headless": 0}
    for t in range(xi.shape[0]):
        lay = np_layers[int(steps[t])]
        x16 = o_routing.rms_norm_f16(xi[t])
        logits = o_routing.logits_fp32(lay["router"], x16)
        check_routing(out["idx"][t], out["w"][t], logits, K, (what, t), stats["routing"])
        if lay["head"] is not None:
            pl = o_routing.logits_fp32(lay["head"], x16)
            check_routing(out["pidx"][t], out["pw"][t], pl, K, (what, t, "pred"), stats["prediction"])
        else:
            assert (out["pidx"][t] == -7).all(), (what, t, "a step without a head wrote a prediction")
            stats["headless"] += 1
        if y_tokens is not None and t not in y_tokens:
            continue
        # the device's routing (equal to the oracle's, or a counted near-tie
        # swap: then the oracle reruns with the device's set)
        idx, w = out["idx"][t], out["w"][t]
        ys = [o_expert.expert_forward(lay["routed"](int(e)), x16, wl.lora_scale)[0] for e in idx]
        ysh = [o_expert.expert_forward(b, x16, wl.lora_scale)[0] for b in lay["shared"]]
        err = rel_inf(out["y"][t], o_expert.combine(w, ys, ysh))
        assert err <= TOL_REL_INF, (what, t, err)
        stats["max_err"] = max(stats["max_err"], err)
        stats["y_checked"] += 1
    return stats


def _steps(T, seed):
    """Rotating table layers (as the benchmark launches them), with a seeded
    shuffle in every round so that consecutive steps meet every pair."""
    rs = np.random.default_rng(seed)
    return np.concatenate([rs.permutation(N_LAYERS) for _ in range((T + N_LAYERS - 1) // N_LAYERS)])[:T]


@pytest.fixture(scope="module")
def tiny_stack(torch_cuda):
    return _stack(synth.WORKLOADS["tiny"], torch_cuda)


@pytest.fixture(scope="module")
def big_stack(torch_cuda):
    return _stack(synth.WORKLOADS["moe35b"], torch_cuda)


@pytest.mark.parametrize("fn", ["engine_tokens", "engine_layers"])
def test_tiny_1000_tokens_rotating_layers(tiny_stack, torch_cuda, fn):
    chain, np_layers, arr = tiny_stack
    wl = synth.WORKLOADS["tiny"]
    T = 1000
    xi = synth.token_draws(wl, 0, T)
    steps = _steps(T, 1)
    out, _ = _run(fn, chain, arr, steps, xi, torch_cuda)
    stats = _check(wl, np_layers, steps, xi, out, fn + " tiny")
    print("%s tiny, 1000 tokens over %d layers:" % (fn, N_LAYERS), stats)
    assert stats["y_checked"] == T


def test_moe35b_128_tokens_rotating_layers(big_stack, torch_cuda):
    """The throughput schedule against the oracle on 128 tokens; the latency
    schedule on the same steps: identical routing and predictions (the same
    router arithmetic), outputs within the layer bar of the oracle on a
    quarter of them."""
    chain, np_layers, arr = big_stack
    wl = synth.WORKLOADS["moe35b"]
    T = 128
    xi = synth.token_draws(wl, 0, T)
    steps = np.arange(T, dtype=np.int32) % N_LAYERS          # the benchmark's rotation
    out, ws = _run("engine_tokens", chain, arr, steps, xi, torch_cuda)
    stats = _check(wl, np_layers, steps, xi, out, "engine_tokens moe35b")
    print("engine_tokens moe35b, 128 tokens over %d layers:" % N_LAYERS, stats)
    lat, _ = _run("engine_layers", chain, arr, steps, xi, torch_cuda, ws=ws)
    for k in ("idx", "w", "pidx", "pw"):
        assert np.array_equal(out[k], lat[k]), k
    lstats = _check(wl, np_layers, steps, xi, lat, "engine_layers moe35b", y_tokens=set(range(0, T, 4)))
    print("engine_layers moe35b:", lstats)
    assert stats["y_checked"] == T and lstats["y_checked"] == T // 4
