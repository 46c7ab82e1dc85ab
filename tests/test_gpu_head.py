"""GPU parity of the full prerouter head (moe_preroute_mlp; §3.2, Head)
against the oracle (routing.preroute_mlp), through the C ABI.

The logits are compared within LOGIT_TOL of the largest oracle logit: the
kernel accumulates in fp32 where the oracle is exact, and a hidden unit whose
fp32 and exact values fall on either side of an fp16 rounding boundary moves
by one fp16 ulp. The predicted set must be the oracle's except where the
oracle's K-th and (K+1)-th logits are within that tolerance (counted).
Also: a head whose MLP is zero gives the linear head's routing (moe_preroute),
the first token's missing previous set (NULL and negative ids), and the
workspace and shape checks.
"""

import numpy as np
import pytest

import synth
from oracle import routing as o_routing

pytestmark = pytest.mark.gpu

LOGIT_TOL = 1e-4


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    from paper_2609_18063_amd import binding
    binding.lib()
    return torch


def _dev_head(torch, head):
    d_plus = head["w1"].shape[1]
    E = head["w2"].shape[0]
    d = d_plus - 2 * E
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    dev = {
        "w1_x": t(head["w1"][:, :d]), "w1_r": t(head["w1"][:, d:].T),
        "w2": t(head["w2"]),
        "b1": t(head["b1"]) if head.get("b1") is not None else None,
        "b2": t(head["b2"]) if head.get("b2") is not None else None,
        "w_l": t(head["wl"]) if head.get("wl") is not None else None,
    }
    return dev


def _run(torch, wl, head, x16, rt, rtm1, tm1_null=False):
    from paper_2609_18063_amd import binding as B
    spec = B.spec_from_workload(wl)
    T, K, E = x16.shape[0], wl.K, wl.E
    dev = _dev_head(torch, head)
    H = head["w1"].shape[0]
    hm = B.head_mlp(H, dev["w1_x"], dev["w1_r"], dev["w2"], dev["b1"], dev["b2"], dev["w_l"])
    ws = torch.zeros(B.preroute_mlp_workspace_bytes(spec, H, T), dtype=torch.uint8, device="cuda")
    x_t = torch.from_numpy(np.ascontiguousarray(x16)).cuda()
    rt_t = torch.from_numpy(np.ascontiguousarray(rt, dtype=np.int32)).cuda()
    rtm1_t = None if tm1_null else torch.from_numpy(np.ascontiguousarray(rtm1, dtype=np.int32)).cuda()
    logits = torch.full((T, E), float("nan"), dtype=torch.float32, device="cuda")
    idx = torch.full((T, K), -7, dtype=torch.int32, device="cuda")
    w = torch.zeros(T, K, dtype=torch.float32, device="cuda")
    print("launch moe_preroute_mlp: T=%d d=%d E=%d K=%d H=%d" % (T, wl.d, E, K, H), flush=True)
    B.preroute_mlp(spec, hm, x_t, rt_t, rtm1_t, idx, w, ws, logits=logits)
    torch.cuda.synchronize()
    return logits.cpu().numpy(), idx.cpu().numpy(), w.cpu().numpy()


def _check(wl, head, x16, rt, rtm1, got, what):
    logits, idx, w = got
    stats = {"near_tie": 0, "tokens": 0}
    for t in range(x16.shape[0]):
        prev = None if rtm1 is None or int(rtm1[t][0]) < 0 else rtm1[t]
        ref_l, ref_i, ref_w = o_routing.preroute_mlp(head, x16[t], rt[t], prev, wl.K)
        scale = float(np.max(np.abs(ref_l)))
        err = float(np.max(np.abs(logits[t].astype(np.float64) - ref_l)))
        assert err <= LOGIT_TOL * scale, (what, t, err, scale)
        if idx[t].tolist() == ref_i.tolist():
            assert np.allclose(w[t], ref_w, rtol=1e-4, atol=1e-6), (what, t, w[t], ref_w)
        else:
            assert sorted(set(idx[t].tolist())) == sorted(idx[t].tolist()), (what, t)
            l = ref_l.astype(np.float64)
            for pos in range(wl.K):
                if idx[t][pos] != ref_i[pos]:
                    assert abs(l[idx[t][pos]] - l[ref_i[pos]]) <= LOGIT_TOL * scale, (what, t, pos)
            stats["near_tie"] += 1
        stats["tokens"] += 1
        stats["max_logit_err"] = max(stats.get("max_logit_err", 0.0), err / scale)
    return stats


def _sets(wl, T, seed):
    g = np.random.default_rng(seed)
    rt = np.stack([g.choice(wl.E, wl.K, replace=False) for _ in range(T)]).astype(np.int32)
    rtm1 = np.stack([g.choice(wl.E, wl.K, replace=False) for _ in range(T)]).astype(np.int32)
    return rt, rtm1


@pytest.mark.parametrize("name,hidden,T", [("tiny", 64, 7), ("moe35b", 512, 12)])
def test_head_mlp_against_oracle(torch_cuda, name, hidden, T):
    wl = synth.WORKLOADS[name]
    head = synth.prerouter_mlp(wl, 3, hidden)
    from oracle.routing import rms_norm_f16
    x16 = rms_norm_f16(synth.token_draws(wl, 5, T))
    rt, rtm1 = _sets(wl, T, 11)
    rtm1[0, :] = -1                 # the first token has no previous set
    got = _run(torch_cuda, wl, head, x16, rt, rtm1)
    stats = _check(wl, head, x16, rt, rtm1, got, name)
    print("head", name, stats)
    assert stats["near_tie"] <= max(1, T // 4)


def test_head_mlp_no_previous_set(torch_cuda):
    wl = synth.WORKLOADS["tiny"]
    head = synth.prerouter_mlp(wl, 0, 64)
    from oracle.routing import rms_norm_f16
    x16 = rms_norm_f16(synth.token_draws(wl, 0, 4))
    rt, _ = _sets(wl, 4, 3)
    got = _run(torch_cuda, wl, head, x16, rt, None, tm1_null=True)
    _check(wl, head, x16, rt, None, got, "no previous")


def test_head_mlp_zero_mlp_is_linear_head(torch_cuda):
    """fc1 and fc2 zero: the prediction is the linear head's (moe_preroute)."""
    torch = torch_cuda
    from paper_2609_18063_amd import binding as B
    wl = synth.WORKLOADS["moe35b"]
    H, T = 64, 6
    wlin = synth.router_weights(wl, 2, 1)
    head = {"w1": np.zeros((H, wl.d + 2 * wl.E), np.float16), "w2": np.zeros((wl.E, H), np.float16),
            "wl": wlin}
    from oracle.routing import rms_norm_f16
    x16 = rms_norm_f16(synth.token_draws(wl, 9, T))
    rt, rtm1 = _sets(wl, T, 5)
    logits, idx, w = _run(torch, wl, head, x16, rt, rtm1)
    spec = B.spec_from_workload(wl)
    ws = torch.zeros(B.workspace_bytes(spec, T), dtype=torch.uint8, device="cuda")
    x_t = torch.from_numpy(x16).cuda()
    pi = torch.zeros(T, wl.K, dtype=torch.int32, device="cuda")
    pw = torch.zeros(T, wl.K, dtype=torch.float32, device="cuda")
    pl = torch.zeros(T, wl.E, dtype=torch.float32, device="cuda")
    B.preroute(spec, x_t, torch.from_numpy(wlin).cuda(), pi, pw, ws, logits=pl)
    torch.cuda.synchronize()
    assert np.array_equal(idx, pi.cpu().numpy())
    assert np.allclose(logits, pl.cpu().numpy(), rtol=0, atol=1e-5)


def test_head_mlp_rejects_bad_shapes(torch_cuda):
    torch = torch_cuda
    from paper_2609_18063_amd import binding as B
    wl = synth.WORKLOADS["tiny"]
    spec = B.spec_from_workload(wl)
    head = synth.prerouter_mlp(wl, 0, 64)
    dev = _dev_head(torch, head)
    x_t = torch.zeros(2, wl.d, dtype=torch.float16, device="cuda")
    rt = torch.zeros(2, wl.K, dtype=torch.int32, device="cuda")
    idx = torch.zeros(2, wl.K, dtype=torch.int32, device="cuda")
    w = torch.zeros(2, wl.K, dtype=torch.float32, device="cuda")
    ws = torch.zeros(B.preroute_mlp_workspace_bytes(spec, 64, 2), dtype=torch.uint8, device="cuda")
    bad = B.head_mlp(60, dev["w1_x"], dev["w1_r"], dev["w2"])   # hidden not a multiple of 8
    with pytest.raises(B.MoeError) as err:
        B.preroute_mlp(spec, bad, x_t, rt, None, idx, w, ws)
    assert err.value.code == B.MOE_EINVAL
    good = B.head_mlp(64, dev["w1_x"], dev["w1_r"], dev["w2"])
    small = torch.zeros(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(B.MoeError) as err:
        B.preroute_mlp(spec, good, x_t, rt, None, idx, w, small)
    assert err.value.code == B.MOE_ENOMEM
