"""GPU parity of the throughput schedule of the decode engine
(moe_engine_tokens: one independent single-token step per team of 16
workgroups in flight, 16 at once)
against the CPU oracle, token by token.

Also checked: routing and predictions bit-identical to the latency schedule
(moe_engine_layers, same router arithmetic), outputs within the layer bar of
it, repeated launches on one workspace bit-identical, step counts that leave
teams idle, a workspace shared with the other schedule, and the status word
for a non-resident expert and a bad layer index.
"""

import numpy as np
import pytest

import synth
from tests.gpu_harness import TOL_REL_INF, DeviceLayer, check_routing, oracle_token, rel_inf

pytestmark = pytest.mark.gpu

TEAMS = 16   # steps in flight: team t runs the steps t, t + 16, ...


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    from paper_2609_18063_amd import binding
    binding.lib()
    return torch


@pytest.fixture(scope="module")
def tiny(torch_cuda):
    return DeviceLayer(synth.WORKLOADS["tiny"])


@pytest.fixture(scope="module")
def big(torch_cuda):
    return DeviceLayer(synth.WORKLOADS["moe35b"])


def _run(dl, xi, torch, fn="engine_tokens", ws=None, table=None, steps=None):
    from paper_2609_18063_amd import binding as B
    wl = dl.wl
    T = xi.shape[0]
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
    if steps is None:
        steps = torch.zeros(T, dtype=torch.int32, device="cuda")
    xi_t = torch.from_numpy(np.ascontiguousarray(xi)).cuda()
    print("launch %s: T=%d d=%d K=%d" % (fn, T, wl.d, wl.K), flush=True)
    getattr(B, fn)(dl.spec, table or dl.table, arr, steps, xi_t, out["y"], ws, idx=out["idx"],
                   w=out["w"], pidx=out["pidx"], pw=out["pw"], status=out["status"])
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy() for k, v in out.items()}
    res["ctl"] = ws[:32].view(torch.int32).cpu().numpy()   # control words (abort cause in 4..7)
    return res, ws


def _check(dl, xi, out, what, tokens=None):
    wl = dl.wl
    stats = {}
    assert int(out["status"][0]) == 0, (out["status"], "control words", out["ctl"][:8].tolist())
    for t in (range(xi.shape[0]) if tokens is None else tokens):
        ref = oracle_token(dl, xi[t])
        exact = check_routing(out["idx"][t], out["w"][t], ref["logits"], wl.K, what, stats)
        check_routing(out["pidx"][t], out["pw"][t], ref["pred_logits"], wl.K, what + " pred", stats)
        if exact:
            err = rel_inf(out["y"][t], ref["y"])
            assert err <= TOL_REL_INF, (what, t, err)
            stats["max_err"] = max(stats.get("max_err", 0.0), err)
            stats["tokens"] = stats.get("tokens", 0) + 1
    return stats


def test_tokens_supported(torch_cuda):
    from paper_2609_18063_amd import binding as B
    assert B.engine_tokens_supported(B.spec_from_workload(synth.WORKLOADS["moe35b"]))
    assert B.engine_tokens_supported(B.spec_from_workload(synth.WORKLOADS["tiny"]))
    assert not B.engine_tokens_supported(B.spec_from_workload(synth.WORKLOADS["tier8b"]))


def test_tokens_tiny_all_steps(tiny, torch_cuda):
    xi = synth.token_draws(tiny.wl, 0, 40)   # every team two or three steps
    out, _ = _run(tiny, xi, torch_cuda)
    stats = _check(tiny, xi, out, "tokens tiny")
    print("tokens tiny:", stats)
    assert stats["tokens"] >= 36


@pytest.mark.parametrize("T", [1, 3, 9, 17])
def test_tokens_tiny_idle_teams(tiny, torch_cuda, T):
    """Fewer steps than teams (and one step past a multiple of the team count)."""
    xi = synth.token_draws(tiny.wl, 40 + T, T)
    out, _ = _run(tiny, xi, torch_cuda)
    _check(tiny, xi, out, "tokens tiny T=%d" % T)


def test_tokens_moe35b_against_oracle_and_latency_schedule(big, torch_cuda):
    xi = synth.token_draws(big.wl, 0, 20)
    out, ws = _run(big, xi, torch_cuda)
    stats = _check(big, xi, out, "tokens moe35b")
    print("tokens moe35b:", stats)
    assert stats["tokens"] >= 18
    # a second launch on the same workspace: bit-identical
    again, ws = _run(big, xi, torch_cuda, ws=ws)
    for k in ("y", "idx", "w", "pidx", "pw"):
        assert np.array_equal(out[k], again[k]), k
    # the latency schedule on the same workspace: same router arithmetic, so
    # the same routing and predictions; outputs within the layer bar
    lat, ws = _run(big, xi, torch_cuda, fn="engine_layers", ws=ws)
    for k in ("idx", "w", "pidx", "pw"):
        assert np.array_equal(out[k], lat[k]), k
    for t in range(xi.shape[0]):
        assert rel_inf(out["y"][t], lat["y"][t]) <= TOL_REL_INF
    # and the throughput schedule once more after it (tags carry on)
    third, _ = _run(big, xi, torch_cuda, ws=ws)
    assert np.array_equal(out["y"], third["y"])


def test_tokens_status_slot_miss_and_bad_layer(tiny, torch_cuda):
    torch = torch_cuda
    from paper_2609_18063_amd import binding as B
    wl = tiny.wl
    table = B.SlotTable(1, tiny.n_ids, tiny.n_ids)
    for e in range(tiny.n_ids):
        table.bind(0, e, int(tiny.perm[e]), tiny.mbundles[e], keep=tiny.dev)
    table.unbind(0, 4)
    table.sync()
    xi = synth.token_draws(wl, 77, 16)
    out, _ = _run(tiny, xi, torch, table=table)
    routed4 = [t for t in range(16) if 4 in out["idx"][t].tolist()]
    assert (int(out["status"][0]) == B.MOE_STATUS_SLOT_MISS) == bool(routed4)
    others = [t for t in range(16) if t not in routed4]
    out["status"][0] = 0
    _check(tiny, xi, out, "tokens tiny miss", tokens=others)
    table.close()
    # a step whose layer is outside the table: BAD_INDEX, nothing hangs
    steps = torch.zeros(16, dtype=torch.int32, device="cuda")
    steps[5] = 3
    out2, _ = _run(tiny, xi, torch, steps=steps)
    assert int(out2["status"][0]) & B.MOE_STATUS_BAD_INDEX
    assert not (int(out2["status"][0]) & B.MOE_STATUS_ENGINE_ABORT)
    # the teams that never met the bad step finished their steps
    for t in range(16):
        if t % TEAMS != 5:
            ref = oracle_token(tiny, xi[t])
            if out2["idx"][t].tolist() == out["idx"][t].tolist() and t in others:
                assert rel_inf(out2["y"][t], ref["y"]) <= TOL_REL_INF
