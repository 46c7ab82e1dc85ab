"""GPU parity of the persistent decode engine against the CPU oracle.

Independent single-token steps are compared token by token, like the
per-call layer tests. The engine's decode chain is compared with the
oracle's chain, like the per-call chain. Also checked: state carried across
launches (the residual and the head predictions in the workspace), repeated
launches on one workspace, and the status word.
"""

import numpy as np
import pytest

import synth
from tests.gpu_harness import (TOL_REL_INF, DeviceLayer, build_chain, check_routing,
                               check_sigmoid_routing, free_running_divergence, oracle_token, rel_inf, sample_layers,
                               teacher_forced_chain)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    from paper_2609_18063_amd import binding
    binding.lib()
    return torch


def _engine_steps(dl, xi, torch, ws=None):
    from paper_2609_18063_amd import binding as B
    wl = dl.wl
    T = xi.shape[0]
    assert B.engine_supported(dl.spec)
    arr = B.engine_layer_array([{"router": dl.router_t, "head": dl.head_t}])
    if ws is None:
        ws = torch.zeros(B.engine_workspace_bytes(dl.spec, 0), dtype=torch.uint8, device="cuda")
    out = {
        "y": torch.full((T, wl.d), float("nan"), dtype=torch.float32, device="cuda"),
        "idx": torch.full((T, wl.K), -7, dtype=torch.int32, device="cuda"),
        "w": torch.zeros(T, wl.K, dtype=torch.float32, device="cuda"),
        "pidx": torch.full((T, wl.K), -7, dtype=torch.int32, device="cuda"),
        "pw": torch.zeros(T, wl.K, dtype=torch.float32, device="cuda"),
        "status": torch.zeros(1, dtype=torch.int32, device="cuda"),
    }
    steps = torch.zeros(T, dtype=torch.int32, device="cuda")
    xi_t = torch.from_numpy(np.ascontiguousarray(xi)).cuda()
    B.engine_layers(dl.spec, dl.table, arr, steps, xi_t, out["y"], ws, idx=out["idx"], w=out["w"],
                    pidx=out["pidx"], pw=out["pw"], status=out["status"])
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}, ws


def _check_steps(dl, xi, out, what):
    wl = dl.wl
    stats = {}
    assert int(out["status"][0]) == 0, out["status"]
    for t in range(xi.shape[0]):
        ref = oracle_token(dl, xi[t])
        exact = check_routing(out["idx"][t], out["w"][t], ref["logits"], wl.K, what, stats)
        check_routing(out["pidx"][t], out["pw"][t], ref["pred_logits"], wl.K, what + " pred", stats)
        if exact:
            err = rel_inf(out["y"][t], ref["y"])
            assert err <= TOL_REL_INF, (what, t, err)
            stats["max_err"] = max(stats.get("max_err", 0.0), err)
    return stats


def test_engine_steps_tiny(torch_cuda):
    dl = DeviceLayer(synth.WORKLOADS["tiny"])
    xi = synth.token_draws(dl.wl, 0, 24)
    out, _ = _engine_steps(dl, xi, torch_cuda)
    stats = _check_steps(dl, xi, out, "engine tiny")
    print("engine tiny steps:", stats)


def test_engine_steps_moe35b_and_repeat(torch_cuda):
    """Full-size 35B-class layer; a second launch on the same workspace
    (tags continue from the device counter) gives identical outputs."""
    dl = DeviceLayer(synth.WORKLOADS["moe35b"])
    xi = synth.token_draws(dl.wl, 0, 6)
    out, ws = _engine_steps(dl, xi, torch_cuda)
    stats = _check_steps(dl, xi, out, "engine moe35b")
    print("engine moe35b steps:", stats)
    again, _ = _engine_steps(dl, xi, torch_cuda, ws=ws)
    for k in ("y", "idx", "w", "pidx", "pw"):
        assert np.array_equal(out[k], again[k]), k


def _engine_chain(chain, xi, L, torch, first_token=0, ws=None, r_state=None, record=True):
    from paper_2609_18063_amd import binding as B
    spec = chain.spec
    wl_d, K = spec.d_model, spec.top_k
    T = xi.shape[0]
    arr = getattr(chain, "engine_arr", None)
    if arr is None:
        arr = B.engine_layer_array(chain.layers)
        chain.engine_arr = arr
    if ws is None:
        ws = torch.zeros(B.engine_workspace_bytes(spec, L), dtype=torch.uint8, device="cuda")
    if r_state is None:
        r_state = torch.zeros(wl_d, dtype=torch.float32, device="cuda")
    n = T * L
    rec = None
    if record:
        rec = {
            "x": torch.zeros(n, wl_d, dtype=torch.float16, device="cuda"),
            "r": torch.zeros(n, wl_d, dtype=torch.float32, device="cuda"),
            "idx": torch.full((n, K), -7, dtype=torch.int32, device="cuda"),
            "w": torch.zeros(n, K, dtype=torch.float32, device="cuda"),
            "pidx": torch.full((n, K), -1, dtype=torch.int32, device="cuda"),
            "pw": torch.zeros(n, K, dtype=torch.float32, device="cuda"),
            "y": torch.zeros(n, wl_d, dtype=torch.float32, device="cuda"),
        }
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    xi_t = torch.from_numpy(np.ascontiguousarray(xi)).cuda()
    g = (lambda k: None) if rec is None else (lambda k: rec[k])
    print("engine chain: L=%d T=%d first_token=%d" % (L, T, first_token), flush=True)
    B.engine_chain(spec, chain.table, arr, L, first_token, xi_t, r_state, ws, x_rec=g("x"),
                   r_rec=g("r"), idx=g("idx"), w=g("w"), pidx=g("pidx"), pw=g("pw"),
                   y_rec=g("y"), status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0, int(status.item())
    if rec is not None:
        rec = {k: v.view(T, L, *v.shape[1:]) for k, v in rec.items()}
    return rec, ws, r_state


def test_engine_chain_tiny_40_layers_256_tokens(torch_cuda):
    """The tiny 40-layer chain over 256 tokens, teacher-forced at every
    (token, layer): stand-in, layer input, routing and predictions (near-ties
    counted); layer outputs at every layer of the first 8 tokens and 8 seeded
    layers of each later token."""
    wl = synth.WORKLOADS["tiny"]
    L, T = 40, 256
    chain, np_layers = build_chain(wl, L, torch_cuda)
    xi = synth.token_draws(wl, 0, T)
    rec, _, _ = _engine_chain(chain, xi, L, torch_cuda)
    rec = {k: v.cpu().numpy() for k, v in rec.items()}
    stats = teacher_forced_chain(rec, xi, np_layers, wl, L,
                                 y_at=sample_layers(T, L, full_tokens=8, per_token=8),
                                 what="engine tiny")
    stats["free_running_divergence"] = free_running_divergence(rec, xi[:16], np_layers, wl, L)
    print("engine tiny chain:", stats)
    assert stats["steps"] == L * T and stats["pred_routing"] == (T - 1) * (L - 1)


def test_engine_chain_split_launches_match(torch_cuda):
    """Six tokens in one launch equal three + three launches: the residual
    and the head predictions carry over in r_state and the workspace."""
    torch = torch_cuda
    wl = synth.WORKLOADS["tiny"]
    L, T = 8, 6
    chain, _ = build_chain(wl, L, torch)
    xi = synth.token_draws(wl, 0, T)
    one, _, r1 = _engine_chain(chain, xi, L, torch)
    a, ws, r2 = _engine_chain(chain, xi[:3], L, torch)
    b, _, r2 = _engine_chain(chain, xi[3:], L, torch, first_token=3, ws=ws, r_state=r2)
    assert torch.equal(r1, r2)
    for k in ("y", "idx", "pidx", "x", "r"):
        joined = torch.cat([a[k], b[k]], dim=0)
        assert torch.equal(one[k], joined), k


def test_engine_chain_moe35b_40_layers(torch_cuda):
    """The 35B-class 40-layer stack over 16 tokens, teacher-forced at every
    (token, layer); layer outputs at every layer of the first two tokens and
    three seeded layers of each later token; the free-running divergence of
    the first two tokens is reported."""
    wl = synth.WORKLOADS["moe35b"]
    L, T = 40, 16
    chain, np_layers = build_chain(wl, L, torch_cuda)
    xi = synth.token_draws(wl, 0, T)
    rec, _, _ = _engine_chain(chain, xi, L, torch_cuda)
    rec = {k: v.cpu().numpy() for k, v in rec.items()}
    stats = teacher_forced_chain(rec, xi, np_layers, wl, L, y_at=sample_layers(T, L),
                                 what="engine moe35b")
    stats["free_running_divergence"] = free_running_divergence(rec, xi[:2], np_layers, wl, L)
    print("engine moe35b chain:", stats)
    assert stats["steps"] == L * T and stats["pred_routing"] == (T - 1) * (L - 1)


def test_engine_rejects_unsupported_shape(torch_cuda):
    from paper_2609_18063_amd import binding as B
    assert not B.engine_supported(B.make_spec(512, 16, 16, 0, 256, 8, 2.0))   # 16*256/8 rows
    assert not B.engine_supported(B.spec_from_workload(synth.WORKLOADS["tier8b"]))
    assert B.engine_supported(B.spec_from_workload(synth.WORKLOADS["moe35b"]))


def test_engine_chain_8b_tier_shape(torch_cuda):
    """The 8B-tier layer (d 4096, 64 experts top-4, I 1024, r 16) through the
    two-half chain: 4 layers x 4 tokens in one launch, teacher-forced at every
    (token, layer); expert outputs at every layer of the first token and one
    seeded layer of each later token."""
    wl = synth.WORKLOADS["tier8b"]
    L, T = 4, 4
    chain, np_layers = build_chain(wl, L, torch_cuda)
    xi = synth.token_draws(wl, 0, T)
    rec, _, _ = _engine_chain(chain, xi, L, torch_cuda)
    rec = {k: v.cpu().numpy() for k, v in rec.items()}
    stats = teacher_forced_chain(rec, xi, np_layers, wl, L,
                                 y_at=sample_layers(T, L, full_tokens=1, per_token=1),
                                 what="engine 8B tier")
    print("engine 8B-tier chain:", stats)
    assert stats["steps"] == L * T and stats["pred_routing"] == (T - 1) * (L - 1)


@pytest.mark.parametrize("name,L,T,groups", [
    ("tiny", 8, 24, (4, 2, 1.0)),
    ("tier8b", 4, 4, (8, 4, 2.5)),
])
def test_engine_chain_sigmoid_group(torch_cuda, name, L, T, groups):
    """The two-half chain with sigmoid-group selection (App. A) for both the
    own router and the head's predictions: teacher-forced at every (token,
    layer) against the oracle's sigmoid_group_topk, near-ties within SG_TIE
    counted; expert outputs at every layer of the first token and one seeded
    layer of each later token."""
    from paper_2609_18063_amd import binding as B
    wl = synth.WORKLOADS[name]
    n, G, s = groups
    spec = B.make_spec(wl.d, wl.E, wl.K, wl.S, wl.I, wl.r, wl.lora_scale, sigmoid_group=groups)
    assert B.engine_chain_supported(spec)
    chain, np_layers = build_chain(wl, L, torch_cuda, spec=spec)
    xi = synth.token_draws(wl, 0, T)
    rec, _, _ = _engine_chain(chain, xi, L, torch_cuda)
    rec = {k: v.cpu().numpy() for k, v in rec.items()}

    def route_check(idx, w, logits, tag, st):
        return check_sigmoid_routing(idx, w, logits, wl.K, n, G, s, None, st, tag)

    stats = teacher_forced_chain(rec, xi, np_layers, wl, L,
                                 y_at=sample_layers(T, L, full_tokens=1, per_token=1),
                                 what="engine sigmoid-group " + name, route_check=route_check)
    print("engine sigmoid-group chain %s:" % name, stats)
    assert stats["steps"] == L * T and stats["pred_routing"] == (T - 1) * (L - 1)
    assert stats["predictions"] == T * (L - 1)
    ties = stats["routing_near_ties"].get("near_tie", 0) + stats["prediction_near_ties"].get("near_tie", 0)
    assert ties <= 2, stats
