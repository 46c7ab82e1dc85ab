"""GPU parity of the per-call multi-layer decode chain (prediction-as-routing).

Teacher-forced per-layer parity (§3.2, Prediction-as-routing): every layer of
every token is checked against the oracle run on the device's own inputs of
that layer (the residual it mixed, the layer input it formed, the routing it
used).  Routing and predictions are bit-exact except at counted near-ties
(oracle K-th / (K+1)-th logit gap within 1e-5); a layer that routes by a
prediction must use exactly the prediction the device made one token
earlier.  The first point where the free-running device chain leaves the
free-running oracle chain is reported, not asserted: one rounding difference
at a near-tie sends the two chains down different experts from there on.
"""

import pytest

import synth
from tests.gpu_harness import (build_chain, free_running_divergence, sample_layers,
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


def _run(wl, L, T, torch):
    chain, np_layers = build_chain(wl, L, torch)
    xi = synth.token_draws(wl, 0, T)
    print("per-call chain %s: L=%d T=%d" % (wl.name, L, T), flush=True)
    rec = chain.run_recorded(torch.from_numpy(xi).cuda())
    assert int(chain.status.item()) == 0
    rec = {k: v.cpu().numpy() for k, v in rec.items()}
    return chain, rec, xi, np_layers


def test_chain_tiny_40_layers(torch_cuda):
    wl = synth.WORKLOADS["tiny"]
    L, T = 40, 64
    chain, rec, xi, np_layers = _run(wl, L, T, torch_cuda)
    stats = teacher_forced_chain(rec, xi, np_layers, wl, L,
                                 y_at=sample_layers(T, L, full_tokens=8, per_token=8),
                                 what="per-call tiny")
    stats["free_running_divergence"] = free_running_divergence(rec, xi[:16], np_layers, wl, L)
    print("tiny chain:", stats)
    assert stats["steps"] == L * T and stats["pred_routing"] == (T - 1) * (L - 1)


def test_chain_graph_replay_matches_eager(torch_cuda):
    """The three captured token graphs reproduce the eager chain bit for bit,
    replayed over several tokens twice."""
    torch = torch_cuda
    wl = synth.WORKLOADS["tiny"]
    L, T = 8, 6
    chain, np_layers = build_chain(wl, L, torch)
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


def test_chain_moe35b_40_layers(torch_cuda):
    """Full-size 40-layer stack of the 35B-class layer, 16 tokens: routing,
    predictions and the stand-in at every (token, layer); expert outputs at
    every layer of the first two tokens and three seeded layers of each
    later token."""
    wl = synth.WORKLOADS["moe35b"]
    L, T = 40, 16
    chain, rec, xi, np_layers = _run(wl, L, T, torch_cuda)
    stats = teacher_forced_chain(rec, xi, np_layers, wl, L, y_at=sample_layers(T, L),
                                 what="per-call moe35b")
    print("moe35b chain:", stats)
    assert stats["steps"] == L * T and stats["pred_routing"] == (T - 1) * (L - 1)
