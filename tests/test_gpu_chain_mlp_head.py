"""GPU parity of the decode chain whose predictions come from the full
prerouter head (fc1 -> erf-GELU -> fc2 + linear path; §3.2 Head), consumed
as routing (§3.2 Prediction-as-routing).

The head of layer N at token t sees layer N's x and the experts layer N
routed to at tokens t and t-1. At decode those sets are themselves the
predictions of the head before it, so the head is fed its own chain's
predictions (the paper's feature drift). Teacher-forced per-layer parity:
on the device's own x and its own recorded routing, each prediction must
equal the oracle head's, except where the oracle's logits are within 1e-4
of their largest magnitude (the full head rounds its hidden activation to
fp16 after an fp32 pre-activation, the oracle after an exact one; counted).
A layer that routes by a prediction must use exactly the prediction made
for it one token earlier; routing by the own router, the layer input and
the layer output are held to the chain's usual bars.
"""

import numpy as np
import pytest

import synth
from oracle import routing as o_routing
from tests.gpu_harness import build_chain, sample_layers, teacher_forced_chain

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


def _heads(wl, L, hidden, torch):
    from paper_2609_18063_amd import binding as B
    heads_np, structs, keep = [], [], []
    for n in range(L):
        if n + 1 == L:
            heads_np.append(None)
            structs.append(None)
            continue
        h = synth.prerouter_mlp(wl, n, hidden)
        d = wl.d

        def t(a):
            return torch.from_numpy(np.ascontiguousarray(a)).cuda()

        dev = {"w1_x": t(h["w1"][:, :d]), "w1_r": t(h["w1"][:, d:].T), "w2": t(h["w2"]),
               "b1": t(h["b1"]), "b2": t(h["b2"]), "w_l": t(h["wl"])}
        keep.append(dev)
        heads_np.append(h)
        structs.append(B.head_mlp(hidden, dev["w1_x"], dev["w1_r"], dev["w2"], dev["b1"], dev["b2"],
                                  dev["w_l"]))
    return heads_np, structs, keep


def _run(wl, L, T, hidden, torch):
    from paper_2609_18063_amd import chain as C
    base, np_layers = build_chain(wl, L, torch)
    heads_np, structs, keep = _heads(wl, L, hidden, torch)
    chain = C.DeviceChain(base.spec, base.table, base.layers, heads_mlp=structs)
    xi = synth.token_draws(wl, 0, T)
    print("per-call chain with the full head %s: L=%d T=%d H=%d" % (wl.name, L, T, hidden), flush=True)
    rec = chain.run_recorded(torch.from_numpy(xi).cuda())
    assert int(chain.status.item()) == 0
    rec = {k: v.cpu().numpy() for k, v in rec.items()}

    def pred_oracle(t, n, x):
        prev = rec["idx"][t - 1, n] if t > 0 else None
        l = o_routing.prerouter_mlp_logits(heads_np[n], x, rec["idx"][t, n], prev)
        return l, LOGIT_TOL * float(np.max(np.abs(l))), LOGIT_TOL

    del keep  # the device heads are no longer read
    return rec, xi, np_layers, pred_oracle, base


def test_chain_full_head_tiny(torch_cuda):
    wl = synth.WORKLOADS["tiny"]
    L, T = 8, 48
    rec, xi, np_layers, pred_oracle, base = _run(wl, L, T, 64, torch_cuda)
    stats = teacher_forced_chain(rec, xi, np_layers, wl, L,
                                 y_at=sample_layers(T, L, full_tokens=4, per_token=3),
                                 what="full-head tiny", pred_oracle=pred_oracle)
    print("full-head tiny chain:", stats)
    assert stats["steps"] == L * T
    assert stats["pred_routing"] == (T - 1) * (L - 1) and stats["predictions"] == T * (L - 1)
    base.table.close()


def test_chain_full_head_moe35b(torch_cuda):
    wl = synth.WORKLOADS["moe35b"]
    L, T = 4, 10
    rec, xi, np_layers, pred_oracle, base = _run(wl, L, T, 512, torch_cuda)
    stats = teacher_forced_chain(rec, xi, np_layers, wl, L,
                                 y_at=sample_layers(T, L, full_tokens=1, per_token=1),
                                 what="full-head 35B", pred_oracle=pred_oracle)
    print("full-head 35B chain:", stats)
    assert stats["pred_routing"] == (T - 1) * (L - 1) and stats["predictions"] == T * (L - 1)
    base.table.close()


def test_chain_full_head_graph_replay_matches_eager(torch_cuda):
    """The captured token graphs of the full-head chain reproduce its eager
    run bit for bit, replayed over several tokens twice."""
    torch = torch_cuda
    from paper_2609_18063_amd import chain as C
    wl = synth.WORKLOADS["tiny"]
    L, T = 6, 7
    base, _ = build_chain(wl, L, torch)
    _, structs, keep = _heads(wl, L, 64, torch)
    chain = C.DeviceChain(base.spec, base.table, base.layers, heads_mlp=structs)
    xi = torch.from_numpy(synth.token_draws(wl, 0, T)).cuda()
    chain.run_recorded(xi)
    r_eager = chain.r.clone()
    chain.capture()
    for rep in range(2):
        chain.reset()
        for t in range(T):
            chain.xi.copy_(xi[t:t + 1])
            chain.replay_token(t)
            torch.cuda.synchronize()
        assert torch.equal(chain.r, r_eager), rep
    del keep
    base.table.close()
